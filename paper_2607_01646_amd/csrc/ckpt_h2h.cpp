// ckpt_h2h.cpp -- host-to-host replication to ring peers (paper Sec. V-B,
// "Host-to-host"; Sec. V-C, replication to k distinct peers against
// concurrent failures): the sending side.  After each local commit, one
// worker per peer streams the selected classes' chunks, their stored sums
// and the envelope to its peer (wire format in ckpt_wire.h) and waits for
// the verdict; the k streams run at once.  The receiving side is
// ckpt_peer.cpp.
#include "ckpt_host.h"

namespace ckpt {

// H2H worker thread of one peer (see Replicator).
void rep_worker(ckpt_ctx* c, Replicator* R)
{
    using clock = std::chrono::steady_clock;
    for (;;) {
        RepJob j;
        bool broken;
        {
            std::unique_lock<std::mutex> l(R->m);
            R->cv.wait(l, [&] { return R->stop || !R->q.empty(); });
            if (R->q.empty()) return;
            j = std::move(R->q.front());
            R->q.pop_front();
            broken = R->broken;
        }
        RepStatus st;
        st.state = REP_FAILED;
        // 1. The local offload has to commit first (bounded wait).
        const auto t_wait = clock::now();
        bool committed = false;
        while (!broken) {
            if (res_done(j.res, j.groups_copied, j.bounce)) {
                committed = !j.res->failed.load(std::memory_order_acquire);
                break;
            }
            if (clock::now() - t_wait > std::chrono::seconds(120)) break;
            {
                std::lock_guard<std::mutex> l(R->m);
                if (R->stop) break;
            }
            std::this_thread::sleep_for(std::chrono::microseconds(100));
        }
        if (broken) st.err = "the connection to the peer failed earlier: " + R->err;
        else if (!committed) st.err = "the local snapshot did not commit";
        const auto t_commit = clock::now();
        int fault = 0;
        uint64_t fa = 0, fb = 0;
        if (committed) {
            {
                std::lock_guard<std::mutex> l(R->m);
                fault = R->fault_kind;
                fa = R->fault_a;
                fb = R->fault_b;
                R->fault_kind = 0;
            }
            // 2. Send head, ids, sums, envelope and the chunks (the deadline
            // moves on while bytes flow: only a stalled connection fails).
            auto deadline = t_commit + std::chrono::seconds(120);
            const uint64_t m = R->ids.size();
            const uint64_t* sums_all = c->h_sums[j.buf];
            std::vector<uint64_t> sums(m);
            for (uint64_t k = 0; k < m; ++k) sums[k] = sums_all[R->ids[k]];
            const std::vector<uint8_t> env = build_envelope(c, j.step, j.meta, sums_all);
            WireHead h;
            std::memcpy(h.magic, kWireMagic, 8);
            h.snap_id = j.id;
            h.step = j.step;
            h.chunk_bytes = c->C;
            h.image_bytes = c->I;
            h.m = m;
            h.replica_bytes = R->bytes;
            h.env_len = env.size();
            bool ok = send_all(R->fd, &h, sizeof h, deadline) == 0 &&
                      send_all(R->fd, R->ids.data(), 8 * m, deadline) == 0 &&
                      send_all(R->fd, sums.data(), 8 * m, deadline) == 0 &&
                      send_all(R->fd, env.data(), env.size(), deadline) == 0;
            const uint8_t* img = c->h_img[j.buf];
            uint64_t sent = 0; // replica bytes sent so far
            for (uint64_t k = 0; ok && k < m;) {
                // one run of consecutive chunk ids is contiguous in the image
                uint64_t e = k + 1;
                while (e < m && R->ids[e] == R->ids[e - 1] + 1) ++e;
                const uint64_t lo = R->ids[k] * c->C, hi = std::min(R->ids[e - 1] * c->C + c->C, c->I);
                uint64_t n = hi - lo;
                if (fault == 2 && sent + n >= fa) { // debug: cut the stream after fa replica bytes
                    (void)send_all(R->fd, img + lo, fa - sent, deadline);
                    ok = false;
                    break;
                }
                if (fault == 1 && fa >= sent && fa < sent + n) { // debug: flip bit fb of replica byte fa
                    const uint64_t at = fa - sent;
                    uint8_t b = img[lo + at] ^ (uint8_t)(1u << (fb & 7));
                    ok = send_all(R->fd, img + lo, at, deadline) == 0 && send_all(R->fd, &b, 1, deadline) == 0 &&
                         send_all(R->fd, img + lo + at + 1, n - at - 1, deadline) == 0;
                } else {
                    ok = send_all(R->fd, img + lo, n, deadline) == 0;
                }
                sent += n;
                k = e;
            }
            const auto t1 = clock::now();
            // 3. The peer's verdict.
            WireAck a;
            if (ok) ok = recv_all(R->fd, &a, sizeof a, deadline) == 0 && std::memcmp(a.magic, kAckMagic, 8) == 0 &&
                         a.snap_id == j.id && a.n_bad <= m;
            if (ok && a.n_bad) {
                st.bad.resize(a.n_bad);
                ok = recv_all(R->fd, st.bad.data(), 8ull * a.n_bad, deadline) == 0;
            }
            const auto t2 = clock::now();
            if (ok) {
                st.state = a.status == CKPT_OK ? REP_OK : a.status == CKPT_ECORRUPT ? REP_CORRUPT : REP_FAILED;
                if (st.state == REP_FAILED) st.err = "the peer reported error " + std::to_string(a.status);
                std::lock_guard<std::mutex> l(R->m);
                R->last_send_ms = std::chrono::duration<double, std::milli>(t1 - t_commit).count();
                R->last_ack_ms = std::chrono::duration<double, std::milli>(t2 - t_commit).count();
            } else {
                st.err = fault == 2 ? "stream cut on request" : "sending to the peer failed";
                std::lock_guard<std::mutex> l(R->m);
                R->broken = true;
                R->err = st.err;
                ::shutdown(R->fd, SHUT_RDWR);
            }
        }
        std::lock_guard<std::mutex> l(R->m);
        R->status[j.id] = std::move(st);
        R->busy[j.buf] = false;
        R->cv.notify_all();
    }
}

// Stop one peer's worker (a job it is sending fails) and free it.
void rep_free(Replicator* R)
{
    {
        std::lock_guard<std::mutex> l(R->m);
        R->stop = true;
    }
    R->cv.notify_all();
    if (R->fd >= 0) ::shutdown(R->fd, SHUT_RDWR);
    if (R->worker.joinable()) R->worker.join();
    if (R->fd >= 0) ::close(R->fd);
    delete R;
}

void rep_stop(ckpt_ctx* c)
{
    for (Replicator* R : c->reps) { // interrupt every peer first, then join them one by one
        {
            std::lock_guard<std::mutex> l(R->m);
            R->stop = true;
        }
        R->cv.notify_all();
        if (R->fd >= 0) ::shutdown(R->fd, SHUT_RDWR);
    }
    for (Replicator* R : c->reps) rep_free(R);
    c->reps.clear();
}

bool rep_busy(ckpt_ctx* c, int b)
{
    for (Replicator* R : c->reps) {
        std::lock_guard<std::mutex> l(R->m);
        if (R->busy[b]) return true;
    }
    return false;
}

} // namespace ckpt

extern "C" {

ckpt_status ckpt_replicate_to(ckpt_ctx* c, const char* host, uint32_t port, uint64_t cls_mask)
{
    if (!c || !host || port == 0 || port > 65535 || cls_mask == 0) return fail(c, CKPT_EINVAL, "bad replication target");
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    if (c->reps.size() >= kMaxPeers) return fail(c, CKPT_EINVAL, "at most %zu replication peers", kMaxPeers);
    if (!c->reps.empty() && c->reps[0]->cls_mask != cls_mask)
        return fail(c, CKPT_EINVAL, "every peer receives the same classes");
    // Snapshots already issued are not sent to a peer added now: adding one
    // while a snapshot is in flight or being sent would leave it behind.
    for (Replicator* R : c->reps) {
        std::lock_guard<std::mutex> l(R->m);
        if (!R->q.empty() || R->busy[0] || R->busy[1])
            return fail(c, CKPT_EBUSY, "a replication is in progress");
    }
    // Chunks holding a byte of a fragment of a selected class.
    std::vector<uint8_t> pick(c->n_chunks, 0);
    for (const Frag& f : c->frags) {
        if (!f.nbytes || f.cls >= 64 || !((cls_mask >> f.cls) & 1)) continue;
        for (uint64_t k = f.off / c->C; k <= (f.off + f.nbytes - 1) / c->C; ++k) pick[k] = 1;
    }
    std::vector<uint64_t> ids;
    for (uint64_t k = 0; k < c->n_chunks; ++k)
        if (pick[k]) ids.push_back(k);
    if (ids.empty()) return fail(c, CKPT_EINVAL, "no registered fragment has a selected class");
    const int fd = dial(host, port);
    if (fd < 0) {
        if (errno == EINVAL) return fail(c, CKPT_EINVAL, "host must be a dotted IPv4 address");
        return fail(c, CKPT_EHIP, "connect to %s:%u: %s", host, port, strerror(errno));
    }
    Replicator* R = new Replicator();
    R->fd = fd;
    R->cls_mask = cls_mask;
    R->ids = std::move(ids);
    R->bytes = replica_bytes(R->ids.data(), R->ids.size(), c->C, c->I);
    R->first_id = c->next_id;
    c->reps.push_back(R);
    R->worker = std::thread(rep_worker, c, R);
    return CKPT_OK;
}

ckpt_status ckpt_replicate_remove(ckpt_ctx* c, uint32_t peer)
{
    if (!c) return CKPT_EINVAL;
    if (peer >= c->reps.size()) return fail(c, CKPT_ESTATE, "no replication peer %u", peer);
    Replicator* R = c->reps[peer];
    c->reps.erase(c->reps.begin() + peer);
    rep_free(R);
    return CKPT_OK;
}

ckpt_status ckpt_replica_chunks(ckpt_ctx* c, uint64_t* ids, uint64_t cap, uint64_t* n, uint64_t* replica_bytes_out)
{
    if (!c || !n) return CKPT_EINVAL;
    if (c->reps.empty()) return fail(c, CKPT_ESTATE, "no replication peer");
    const Replicator* R = c->reps[0]; // every peer receives the same chunks
    *n = R->ids.size();
    if (replica_bytes_out) *replica_bytes_out = R->bytes;
    if (ids) std::memcpy(ids, R->ids.data(), 8 * std::min<uint64_t>(cap, R->ids.size()));
    return CKPT_OK;
}

ckpt_status ckpt_replica_peer_result(ckpt_ctx* c, uint32_t peer, uint64_t snap_id, int32_t* state, uint64_t* bad,
                                     uint32_t cap, uint32_t* n_bad)
{
    if (!c || !state) return CKPT_EINVAL;
    if (peer >= c->reps.size()) return fail(c, CKPT_ESTATE, "no replication peer %u", peer);
    Replicator* R = c->reps[peer];
    std::lock_guard<std::mutex> l(R->m);
    auto s = R->status.find(snap_id);
    if (s == R->status.end())
        return fail(c, CKPT_ERANGE, "snapshot %llu is not being replicated", (unsigned long long)snap_id);
    *state = s->second.state;
    if (n_bad) *n_bad = (uint32_t)s->second.bad.size();
    if (bad) std::memcpy(bad, s->second.bad.data(), 8 * std::min<uint64_t>(cap, s->second.bad.size()));
    return CKPT_OK;
}

ckpt_status ckpt_replica_result(ckpt_ctx* c, uint64_t snap_id, int32_t* state, uint64_t* bad, uint32_t cap,
                                uint32_t* n_bad)
{
    if (!c || !state) return CKPT_EINVAL;
    if (c->reps.empty()) return fail(c, CKPT_ESTATE, "no replication peer");
    // Pending while any peer is; then failed, corrupt (the union of the bad
    // chunks) or OK.
    bool pending = false, failed = false;
    size_t asked = 0;
    std::vector<uint64_t> all;
    for (Replicator* R : c->reps) {
        if (snap_id < R->first_id) continue; // added after this snapshot
        ++asked;
        std::lock_guard<std::mutex> l(R->m);
        auto s = R->status.find(snap_id);
        if (s == R->status.end())
            return fail(c, CKPT_ERANGE, "snapshot %llu is not being replicated", (unsigned long long)snap_id);
        pending |= s->second.state == REP_PENDING;
        failed |= s->second.state == REP_FAILED;
        all.insert(all.end(), s->second.bad.begin(), s->second.bad.end());
    }
    if (!asked)
        return fail(c, CKPT_ERANGE, "snapshot %llu was not sent to any current peer", (unsigned long long)snap_id);
    std::sort(all.begin(), all.end());
    all.erase(std::unique(all.begin(), all.end()), all.end());
    *state = pending ? REP_PENDING : failed ? REP_FAILED : all.empty() ? REP_OK : REP_CORRUPT;
    if (n_bad) *n_bad = (uint32_t)all.size();
    if (bad) std::memcpy(bad, all.data(), 8 * std::min<uint64_t>(cap, all.size()));
    return CKPT_OK;
}

ckpt_status ckpt_replica_timing(ckpt_ctx* c, double* send_ms, double* ack_ms)
{
    if (!c || !send_ms || !ack_ms) return CKPT_EINVAL;
    if (c->reps.empty()) return fail(c, CKPT_ESTATE, "no replication peer");
    *send_ms = *ack_ms = 0;
    for (Replicator* R : c->reps) { // the slowest peer's
        std::lock_guard<std::mutex> l(R->m);
        *send_ms = std::max(*send_ms, R->last_send_ms);
        *ack_ms = std::max(*ack_ms, R->last_ack_ms);
    }
    return CKPT_OK;
}

ckpt_status ckpt_debug_h2h_fault_peer(ckpt_ctx* c, uint32_t peer, int32_t kind, uint64_t a, uint64_t b)
{
    if (!c || kind < 0 || kind > 2) return CKPT_EINVAL;
    if (peer >= c->reps.size()) return fail(c, CKPT_ESTATE, "no replication peer %u", peer);
    Replicator* R = c->reps[peer];
    std::lock_guard<std::mutex> l(R->m);
    if (kind && a >= R->bytes) return fail(c, CKPT_EINVAL, "fault position beyond the replica");
    R->fault_kind = kind;
    R->fault_a = a;
    R->fault_b = b;
    return CKPT_OK;
}

ckpt_status ckpt_debug_h2h_fault(ckpt_ctx* c, int32_t kind, uint64_t a, uint64_t b)
{
    return ckpt_debug_h2h_fault_peer(c, 0, kind, a, b);
}

ckpt_status ckpt_replica_peers(ckpt_ctx* c, uint32_t* n)
{
    if (!c || !n) return CKPT_EINVAL;
    *n = (uint32_t)c->reps.size();
    return CKPT_OK;
}

} // extern "C"
