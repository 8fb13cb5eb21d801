// ckpt_recover.cpp -- a replacement rank takes its optimizer state back
// from the ring peer (paper Sec. V-C, third recovery stage: the new rank
// pulls the optimizer shard from the in-memory replica its peer kept; the
// parameter shard comes from the ranks that share its logical partition).
//
// The replacement's context is registered with the failed rank's layout.
// It fetches the peer's newest committed replica on a connection of its
// own, checks that the replica's envelope describes exactly this layout,
// receives the replicated chunks into the host image that the next
// snapshot would fill (at their own image offsets), and runs the library's
// restore path on those chunks only: host -> device copies, the scatter
// kernel writing every fragment byte of the chunks back to the registered
// tensors, and the chunk sums recomputed and compared with the sums stored
// at pack time on the failed rank.  The restore of each run of chunks
// starts as soon as it has arrived, overlapping the rest of the transfer
// (the paper's recovery transport likewise overlaps communication with the
// work on the receiving node).
#include "ckpt_host.h"

namespace ckpt {
namespace {

constexpr uint64_t kMaxFetchEnvelope = 256ull << 20;

uint64_t word_sum(const uint8_t* p, uint64_t n)
{
    uint64_t s = 0;
    for (uint64_t k = 0; k + 8 <= n; k += 8) {
        uint64_t w;
        std::memcpy(&w, p + k, 8);
        s += w;
    }
    return s;
}

// The envelope's step, chunk sums and caller blob, once its framing and
// word-sum hold.  Field layout as written by build_envelope.
bool parse_envelope(const std::vector<uint8_t>& env, uint64_t* step, std::vector<uint64_t>* sums,
                    std::vector<uint8_t>* blob)
{
    if (env.size() < 64 || env.size() % 8) return false;
    if (std::memcmp(env.data(), "CKPTENV1", 8) != 0) return false;
    uint64_t n_chunks;
    uint32_t n_frag, meta_len;
    std::memcpy(step, env.data() + 16, 8);
    std::memcpy(&n_chunks, env.data() + 40, 8);
    std::memcpy(&n_frag, env.data() + 48, 4);
    std::memcpy(&meta_len, env.data() + 52, 4);
    const uint64_t table = 56, sums_at = table + 24ull * n_frag, blob_at = sums_at + 8 * n_chunks;
    if (n_chunks > env.size() / 8 || blob_at + round_up(meta_len, 8) + 8 != env.size()) return false;
    uint64_t stored;
    std::memcpy(&stored, env.data() + env.size() - 8, 8);
    if (word_sum(env.data(), env.size() - 8) != stored) return false;
    sums->resize(n_chunks);
    std::memcpy(sums->data(), env.data() + sums_at, 8 * n_chunks);
    blob->assign(env.data() + blob_at, env.data() + blob_at + meta_len);
    return true;
}

} // namespace
} // namespace ckpt

extern "C" {

ckpt_status ckpt_restore_from_peer(ckpt_ctx* c, const char* host, uint32_t port, void* stream, uint64_t* snap_id,
                                   uint64_t* step, uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad)
{
    using clock = std::chrono::steady_clock;
    if (!c || !host || !n_bad || (cap && !bad_chunks) || port == 0 || port > 65535)
        return fail(c, CKPT_EINVAL, "bad argument");
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    HIPCHK(c, hipSetDevice(c->device));
    *n_bad = 0;
    ckpt_status st = drain(c);
    if (st) return st;
    int b = 0;
    st = pick_target_image(c, &b);
    if (st) return st;

    const auto t0 = clock::now();
    auto deadline = t0 + std::chrono::seconds(300);
    const int fd = dial(host, port);
    if (fd < 0) {
        if (errno == EINVAL) return fail(c, CKPT_EINVAL, "host must be a dotted IPv4 address");
        return fail(c, CKPT_EHIP, "connect to %s:%u: %s", host, port, strerror(errno));
    }
    struct Closer {
        int fd;
        ~Closer() { ::close(fd); }
    } closer{fd};
    WireFetch f{};
    std::memcpy(f.magic, kFetchMagic, 8);
    WireAck a;
    if (send_all(fd, &f, sizeof f, deadline) || recv_all(fd, &a, sizeof a, deadline))
        return fail(c, CKPT_EHIP, "fetch from %s:%u: connection failed", host, port);
    if (std::memcmp(a.magic, kAckMagic, 8) != 0) return fail(c, CKPT_EINVAL, "malformed reply from the peer");
    if (a.status == CKPT_ENOSNAP) return fail(c, CKPT_ENOSNAP, "the peer holds no committed replica");
    if (a.status != CKPT_OK) return fail(c, CKPT_EHIP, "the peer refused the fetch (%d)", a.status);

    WireHead h;
    if (recv_all(fd, &h, sizeof h, deadline)) return fail(c, CKPT_EHIP, "fetch: connection broke");
    if (std::memcmp(h.magic, kWireMagic, 8) != 0 || h.m == 0 || h.m > c->n_chunks || h.env_len > kMaxFetchEnvelope)
        return fail(c, CKPT_EINVAL, "malformed replica header");
    if (h.chunk_bytes != c->C || h.image_bytes != c->I)
        return fail(c, CKPT_EINVAL, "the replica's chunk size or image size differs from this layout");
    std::vector<uint64_t> ids(h.m), sums(h.m);
    std::vector<uint8_t> env(h.env_len);
    if (recv_all(fd, ids.data(), 8 * h.m, deadline) || recv_all(fd, sums.data(), 8 * h.m, deadline) ||
        recv_all(fd, env.data(), h.env_len, deadline))
        return fail(c, CKPT_EHIP, "fetch: connection broke");
    for (uint64_t j = 0; j < h.m; ++j)
        if (ids[j] >= c->n_chunks || (j && ids[j] <= ids[j - 1]))
            return fail(c, CKPT_EINVAL, "malformed replica chunk list");
    if (replica_bytes(ids.data(), h.m, c->C, c->I) != h.replica_bytes)
        return fail(c, CKPT_EINVAL, "malformed replica size");

    // The envelope must describe this very layout: rebuilt from this
    // context's fragment table with the envelope's own step, sums and blob,
    // it has to come out byte for byte the same.
    uint64_t env_step = 0;
    std::vector<uint64_t> env_sums;
    std::vector<uint8_t> blob;
    if (!parse_envelope(env, &env_step, &env_sums, &blob) || env_step != h.step)
        return fail(c, CKPT_EINVAL, "the replica's envelope is malformed");
    if (env_sums.size() != c->n_chunks || build_envelope(c, env_step, blob, env_sums.data()) != env)
        return fail(c, CKPT_EINVAL, "the replica's envelope describes another layout");
    for (uint64_t j = 0; j < h.m; ++j)
        if (sums[j] != env_sums[ids[j]])
            return fail(c, CKPT_EINVAL, "the replica's sums disagree with its envelope");

    // Image b stops holding a restorable snapshot before its bytes change.
    c->holder[b] = 0;
    if (c->file_map) file_invalidate(c, b);
    for (uint64_t j = 0; j < h.m; ++j) c->h_sums[b][ids[j]] = sums[j];

    // The chunks arrive in id order; each span of consecutive chunks is
    // received just before its host -> device copy, so the network transfer
    // overlaps the copies and kernels of the spans before it.
    PeerRestore& pr = c->peer_restore;
    pr.valid = false;
    uint64_t got = 0;
    bool broke = false;
    auto t1 = t0;
    auto fill = [&](uint64_t lo, uint64_t hi) {
        if (recv_all(fd, c->h_img[b] + lo, hi - lo, deadline)) {
            broke = true;
            return false;
        }
        got += hi - lo;
        if (got == h.replica_bytes) t1 = clock::now();
        return true;
    };
    st = check_image(c, b, (hipStream_t)stream, true, &ids, bad_chunks, cap, n_bad, fill);
    if (broke)
        return fail(c, CKPT_EHIP, "fetch: connection broke after %llu of %llu replica bytes",
                    (unsigned long long)got, (unsigned long long)h.replica_bytes);
    if (st && st != CKPT_ECORRUPT) return st;
    const auto t2 = clock::now();
    pr.valid = true;
    pr.snap_id = h.snap_id;
    pr.step = h.step;
    pr.ids = std::move(ids);
    pr.envelope = std::move(env);
    pr.fetch_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
    pr.check_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
    if (snap_id) *snap_id = h.snap_id;
    if (step) *step = h.step;
    return st;
}

ckpt_status ckpt_peer_restore_info(ckpt_ctx* c, uint64_t* ids, uint64_t cap, uint64_t* n_ids, void* envelope,
                                   uint64_t env_cap, uint64_t* env_len, double* fetch_ms, double* check_ms)
{
    if (!c) return CKPT_EINVAL;
    const PeerRestore& pr = c->peer_restore;
    if (!pr.valid) return fail(c, CKPT_ESTATE, "no restore from a peer yet");
    if (envelope && env_cap < pr.envelope.size()) return fail(c, CKPT_EINVAL, "envelope buffer too small");
    if (n_ids) *n_ids = pr.ids.size();
    if (ids) std::memcpy(ids, pr.ids.data(), 8 * std::min<uint64_t>(cap, pr.ids.size()));
    if (env_len) *env_len = pr.envelope.size();
    if (envelope) std::memcpy(envelope, pr.envelope.data(), pr.envelope.size());
    if (fetch_ms) *fetch_ms = pr.fetch_ms;
    if (check_ms) *check_ms = pr.check_ms;
    return CKPT_OK;
}

} // extern "C"
