// ckpt_peer.cpp -- the receiving side of host-to-host replication (paper
// Sec. V-B, "Host-to-host": the optimizer-state part of each snapshot and
// its envelope go to the ring peer; Sec. VI-A: the buffer received from the
// ring predecessor is kept apart from the local snapshot and alternates
// between two host buffers the same way).
//
// One thread per peer accepts a sender and handles its snapshots in order:
// receive the replica into the pinned buffer that does not hold the newest
// committed replica, re-check every chunk sum on the GPU (host -> device
// copies through a two-slot device ring, then the library's checksum and
// chunk-reduce kernels over the replica laid out as an image of its own
// chunks; each unit is checked while the next one arrives), commit only if
// every sum matches, and answer the sender.  A
// stream that breaks mid-snapshot leaves the previous replica in place.
// A replacement rank (Sec. V-C, third recovery stage) fetches the newest
// committed replica on a connection of its own, also between two snapshots
// of a connected sender.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <new>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/ckpt.h"
#include "ckpt_internal.h"
#include "ckpt_wire.h"

using namespace ckpt;

namespace {
constexpr uint64_t kPeerDefaultGroup = 1ull << 30;
constexpr uint64_t kMaxEnvelope = 256ull << 20;
} // namespace

struct ckpt_peer {
    int device = 0;
    uint64_t group_cfg = kPeerDefaultGroup;
    uint32_t grid_cap = 0x7fffffff;
    int lfd = -1;
    uint32_t port = 0;
    std::thread th;
    std::atomic<bool> stop{false};

    std::mutex m; // guards everything below that the API reads
    std::condition_variable cv;
    int cfd = -1; // the connection being served
    int sfd = -1; // a fetch answered beside a connected sender

    // geometry, fixed by the first snapshot received
    bool ready = false;
    uint64_t C = 0, I = 0, n = 0, R = 0, G = 1;
    std::vector<uint64_t> ids;
    Geometry geo{};

    // the two replica buffers
    uint8_t* h_buf[2] = {nullptr, nullptr};
    uint64_t* h_sums[2] = {nullptr, nullptr};
    std::vector<uint8_t> env[2];
    uint64_t snap[2] = {0, 0}, step[2] = {0, 0};
    int committed = -1;

    // device side of the check
    uint8_t* d_ring = nullptr;
    unsigned long long *d_partials = nullptr, *d_expected = nullptr, *d_recomputed = nullptr;
    uint8_t* d_bad = nullptr;
    uint8_t* h_bad = nullptr;
    hipStream_t s_copy = nullptr, s_ker = nullptr;
    hipEvent_t ev_free[2] = {nullptr, nullptr}, ev_loaded[2] = {nullptr, nullptr};

    std::map<uint64_t, int32_t> results;
    std::vector<uint64_t> last_bad;
    double recv_ms = 0, check_ms = 0;
    std::string err;
};

namespace {

void set_err(ckpt_peer* p, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    std::lock_guard<std::mutex> l(p->m);
    p->err = buf;
}

void free_geometry(ckpt_peer* p)
{
    for (int b = 0; b < 2; ++b) {
        if (p->h_buf[b]) (void)hipHostFree(p->h_buf[b]);
        if (p->h_sums[b]) (void)hipHostFree(p->h_sums[b]);
        p->h_buf[b] = nullptr;
        p->h_sums[b] = nullptr;
        if (p->ev_free[b]) (void)hipEventDestroy(p->ev_free[b]);
        if (p->ev_loaded[b]) (void)hipEventDestroy(p->ev_loaded[b]);
        p->ev_free[b] = p->ev_loaded[b] = nullptr;
    }
    if (p->h_bad) (void)hipHostFree(p->h_bad);
    p->h_bad = nullptr;
    for (void* d : {(void*)p->d_ring, (void*)p->d_partials, (void*)p->d_expected, (void*)p->d_recomputed,
                    (void*)p->d_bad})
        if (d) (void)hipFree(d);
    p->d_ring = nullptr;
    p->d_partials = p->d_expected = p->d_recomputed = nullptr;
    p->d_bad = nullptr;
    for (hipStream_t s : {p->s_copy, p->s_ker})
        if (s) (void)hipStreamDestroy(s);
    p->s_copy = p->s_ker = nullptr;
}

// Allocate buffers for the sender's geometry (first snapshot only; the
// header and the ids have been checked).
bool setup_geometry(ckpt_peer* p, const WireHead& h, const std::vector<uint64_t>& ids)
{
    const uint64_t C = h.chunk_bytes;
    p->C = C;
    p->I = h.image_bytes;
    p->n = h.m;
    p->R = h.replica_bytes;
    p->ids = ids;
    uint32_t ts = 0;
    while (ts < kMaxTileShift && (C >> (ts + 1)) << (ts + 1) == C) ++ts; // largest power of two <= 8 KiB dividing C
    p->geo.image_bytes = p->R;
    p->geo.tile_shift = ts;
    p->geo.tiles_per_chunk = (uint32_t)(C >> ts);
    p->geo.n_tiles = (p->R + (1ull << ts) - 1) >> ts;
    p->geo.n_chunks = p->n;
    p->G = std::max<uint64_t>(1, p->group_cfg / C);
    const uint64_t unit = p->G * C;
    bool ok = hipSetDevice(p->device) == hipSuccess;
    for (int b = 0; ok && b < 2; ++b) {
        ok = hipHostMalloc((void**)&p->h_buf[b], p->R, hipHostMallocDefault) == hipSuccess &&
             hipHostMalloc((void**)&p->h_sums[b], 8 * p->n, hipHostMallocDefault) == hipSuccess;
        if (ok) std::memset(p->h_buf[b], 0, p->R);
    }
    ok = ok && hipHostMalloc((void**)&p->h_bad, p->n, hipHostMallocDefault) == hipSuccess &&
         hipMalloc((void**)&p->d_ring, 2 * std::min(unit, p->R)) == hipSuccess &&
         hipMalloc((void**)&p->d_partials, 8 * kTileParts * p->geo.n_tiles) == hipSuccess &&
         hipMalloc((void**)&p->d_expected, 8 * p->n) == hipSuccess &&
         hipMalloc((void**)&p->d_recomputed, 8 * p->n) == hipSuccess && hipMalloc((void**)&p->d_bad, p->n) == hipSuccess &&
         hipStreamCreateWithFlags(&p->s_copy, hipStreamNonBlocking) == hipSuccess &&
         hipStreamCreateWithFlags(&p->s_ker, hipStreamNonBlocking) == hipSuccess;
    for (int b = 0; ok && b < 2; ++b)
        ok = hipEventCreateWithFlags(&p->ev_free[b], hipEventDisableTiming) == hipSuccess &&
             hipEventCreateWithFlags(&p->ev_loaded[b], hipEventDisableTiming) == hipSuccess &&
             hipEventRecord(p->ev_free[b], p->s_ker) == hipSuccess;
    if (!ok) {
        free_geometry(p);
        return false;
    }
    p->ready = true;
    return true;
}

// Re-check every chunk sum of replica buffer b on the GPU; fills bad with
// the sender's ids of the chunks that differ.  fill(lo, hi) first puts
// replica bytes [lo, hi) in place (received from the sender while the
// earlier units are copied and checked).  Returns false when fill fails or
// on a HIP error, after the work already issued has finished.
template <class Fill>
bool check_on_gpu(ckpt_peer* p, int b, std::vector<uint64_t>& bad, Fill fill)
{
    const uint64_t unit = std::min(p->G * p->C, p->R);
    const uint64_t tile = 1ull << p->geo.tile_shift;
    bool ok = hipMemcpyAsync(p->d_expected, p->h_sums[b], 8 * p->n, hipMemcpyHostToDevice, p->s_copy) == hipSuccess;
    for (uint64_t lo = 0, u = 0; ok && lo < p->R; lo += unit, ++u) {
        const uint64_t hi = std::min(lo + unit, p->R);
        const int slot = (int)(u & 1);
        uint8_t* stage = p->d_ring + slot * unit;
        ok = fill(lo, hi) && hipStreamWaitEvent(p->s_copy, p->ev_free[slot], 0) == hipSuccess &&
             hipMemcpyAsync(stage, p->h_buf[b] + lo, hi - lo, hipMemcpyHostToDevice, p->s_copy) == hipSuccess &&
             hipEventRecord(p->ev_loaded[slot], p->s_copy) == hipSuccess &&
             hipStreamWaitEvent(p->s_ker, p->ev_loaded[slot], 0) == hipSuccess;
        const uint64_t t_lo = lo / tile, t_hi = (hi + tile - 1) / tile;
        ok = ok && launch_checksum(p->geo, t_lo, t_hi, stage, lo, p->d_partials, p->grid_cap, p->s_ker) == hipSuccess &&
             launch_chunk_reduce(p->geo, t_lo, t_hi, p->d_partials, p->d_recomputed, p->d_expected, p->d_bad,
                                 p->s_ker) == hipSuccess &&
             hipEventRecord(p->ev_free[slot], p->s_ker) == hipSuccess;
    }
    ok = ok && hipMemcpyAsync(p->h_bad, p->d_bad, p->n, hipMemcpyDeviceToHost, p->s_ker) == hipSuccess &&
         hipStreamSynchronize(p->s_ker) == hipSuccess;
    if (!ok) {
        (void)hipStreamSynchronize(p->s_copy);
        (void)hipStreamSynchronize(p->s_ker);
        return false;
    }
    bad.clear();
    for (uint64_t j = 0; j < p->n; ++j)
        if (p->h_bad[j]) bad.push_back(p->ids[j]);
    return true;
}

// Wait until the sender's fd or the listening socket is readable: 1 = the
// sender, 2 = a new connection, 0 = stopping or a poll error.
int wait_readable(ckpt_peer* p, int fd)
{
    while (!p->stop.load()) {
        pollfd q[2] = {{fd, POLLIN, 0}, {p->lfd, POLLIN, 0}};
        const int r = ::poll(q, 2, 200);
        if (r > 0) return (q[0].revents & (POLLIN | POLLHUP | POLLERR)) ? 1 : 2;
        if (r < 0 && errno != EINTR) return 0;
    }
    return 0;
}

// Answer a replacement rank's fetch (its magic already read): the newest
// committed replica in the sender's stream format.  Runs on the peer thread,
// so no snapshot can be received into that buffer meanwhile.
void serve_fetch(ckpt_peer* p, int fd)
{
    auto deadline = std::chrono::steady_clock::now() + std::chrono::seconds(120);
    WireFetch f;
    if (recv_all(fd, reinterpret_cast<char*>(&f) + 8, sizeof f - 8, deadline)) return;
    int b;
    {
        std::lock_guard<std::mutex> l(p->m);
        b = p->committed;
    }
    WireAck a;
    std::memcpy(a.magic, kAckMagic, 8);
    a.snap_id = b >= 0 ? p->snap[b] : 0;
    a.status = b >= 0 ? CKPT_OK : CKPT_ENOSNAP;
    a.n_bad = 0;
    a.reserved = 0;
    if (send_all(fd, &a, sizeof a, deadline) || b < 0) return;
    WireHead h;
    std::memcpy(h.magic, kWireMagic, 8);
    h.snap_id = p->snap[b];
    h.step = p->step[b];
    h.chunk_bytes = p->C;
    h.image_bytes = p->I;
    h.m = p->n;
    h.replica_bytes = p->R;
    h.env_len = p->env[b].size();
    const bool sent = send_all(fd, &h, sizeof h, deadline) == 0 &&
                      send_all(fd, p->ids.data(), 8 * p->n, deadline) == 0 &&
                      send_all(fd, p->h_sums[b], 8 * p->n, deadline) == 0 &&
                      send_all(fd, p->env[b].data(), p->env[b].size(), deadline) == 0 &&
                      send_all(fd, p->h_buf[b], p->R, deadline) == 0;
    if (!sent) set_err(p, "fetch of replica %llu: connection broke", (unsigned long long)h.snap_id);
}

// A connection accepted while a sender is being served: answer a fetch,
// refuse a second sender.
void side_connection(ckpt_peer* p)
{
    const int fd = ::accept(p->lfd, nullptr, nullptr);
    if (fd < 0) return;
    tune_socket(fd);
    {
        std::lock_guard<std::mutex> l(p->m);
        p->sfd = fd;
    }
    char magic[8];
    if (recv_all(fd, magic, 8, std::chrono::steady_clock::now() + std::chrono::seconds(10)) == 0) {
        if (std::memcmp(magic, kFetchMagic, 8) == 0) serve_fetch(p, fd);
        else set_err(p, "refused a connection while a sender is connected");
    }
    {
        std::lock_guard<std::mutex> l(p->m);
        p->sfd = -1;
    }
    ::close(fd);
}

void finish(ckpt_peer* p, uint64_t id, int32_t result)
{
    std::lock_guard<std::mutex> l(p->m);
    p->results[id] = result;
    while (p->results.size() > 256) p->results.erase(p->results.begin());
    p->cv.notify_all();
}

// Header fields that hold for any sender: chunk size a multiple of 256,
// an image of at most 2^48 bytes, 1 <= m <= the image's chunk count, and a
// replica of m chunks of which only the last may be short.  Checked before
// anything is allocated for the snapshot.
bool head_ok(const WireHead& h)
{
    const uint64_t C = h.chunk_bytes, I = h.image_bytes;
    if (std::memcmp(h.magic, kWireMagic, 8) != 0 || C == 0 || C % 256 || I == 0 || I % 16 || I > (1ull << 48) ||
        h.env_len > kMaxEnvelope)
        return false;
    const uint64_t img_chunks = I / C + (I % C != 0);
    return h.m != 0 && h.m <= img_chunks && h.replica_bytes > (h.m - 1) * C && h.replica_bytes <= h.m * C;
}

// Receive the header's m chunk ids in pieces, each checked as it arrives
// (increasing, inside the sender's image), so that memory grows only with
// valid ids actually received.  0 = received, -1 = the connection failed,
// -2 = an id out of order or out of range.
int recv_ids(int fd, const WireHead& h, std::vector<uint64_t>& ids, std::chrono::steady_clock::time_point& deadline)
{
    const uint64_t img_chunks = h.image_bytes / h.chunk_bytes + (h.image_bytes % h.chunk_bytes != 0);
    const uint64_t piece = 1ull << 17;
    ids.clear();
    while (ids.size() < h.m) {
        const uint64_t k0 = ids.size(), k = std::min<uint64_t>(piece, h.m - k0);
        ids.resize(k0 + k);
        if (recv_all(fd, ids.data() + k0, 8 * k, deadline)) return -1;
        for (uint64_t j = k0; j < k0 + k; ++j)
            if (ids[j] >= img_chunks || (j && ids[j] <= ids[j - 1])) return -2;
    }
    return 0;
}

// Handle one sender connection (the first snapshot's magic already read)
// until it closes or breaks; between snapshots, answer fetches on other
// connections.
void serve(ckpt_peer* p, int fd)
{
    using clock = std::chrono::steady_clock;
    for (bool first = true;; first = false) {
        if (!first) {
            const int w = wait_readable(p, fd);
            if (w == 0) return;
            if (w == 2) {
                side_connection(p);
                continue;
            }
        }
        const auto t0 = clock::now();
        auto deadline = t0 + std::chrono::seconds(120);
        WireHead h;
        if (!first && recv_all(fd, h.magic, 8, deadline)) return; // closed between snapshots
        if (first) std::memcpy(h.magic, kWireMagic, 8);
        if (recv_all(fd, reinterpret_cast<char*>(&h) + 8, sizeof h - 8, deadline)) return;
        if (!head_ok(h)) {
            set_err(p, "malformed replica header");
            return;
        }
        if (p->ready && (h.chunk_bytes != p->C || h.image_bytes != p->I || h.m != p->n || h.replica_bytes != p->R)) {
            set_err(p, "replica geometry changed");
            finish(p, h.snap_id, CKPT_EINVAL);
            return;
        }
        std::vector<uint64_t> ids;
        const int got_ids = recv_ids(fd, h, ids, deadline);
        if (got_ids == -1) {
            finish(p, h.snap_id, CKPT_EHIP);
            return;
        }
        const char* why = got_ids == -2 ? "malformed replica chunk list"
                          : p->ready    ? (ids != p->ids ? "replica geometry changed" : nullptr)
                          : replica_bytes(ids.data(), h.m, h.chunk_bytes, h.image_bytes) != h.replica_bytes
                              ? "malformed replica size"
                              : nullptr;
        if (why) {
            set_err(p, "%s", why);
            finish(p, h.snap_id, CKPT_EINVAL);
            return;
        }
        if (!p->ready && !setup_geometry(p, h, ids)) {
            set_err(p, "cannot take a replica of %llu bytes in %llu chunks", (unsigned long long)h.replica_bytes,
                    (unsigned long long)h.m);
            finish(p, h.snap_id, CKPT_ENOMEM);
            return;
        }
        int target;
        {
            std::lock_guard<std::mutex> l(p->m);
            target = p->committed == 0 ? 1 : 0;
        }
        std::vector<uint8_t> env(h.env_len);
        const bool got = recv_all(fd, p->h_sums[target], 8 * h.m, deadline) == 0 &&
                         recv_all(fd, env.data(), h.env_len, deadline) == 0;
        // The replica bytes arrive unit by unit, each checked on the GPU
        // while the next one is received.
        bool broke = !got;
        auto t1 = t0;
        auto fill = [&](uint64_t lo, uint64_t hi) {
            if (recv_all(fd, p->h_buf[target] + lo, hi - lo, deadline)) {
                broke = true;
                return false;
            }
            if (hi == h.replica_bytes) t1 = clock::now();
            return true;
        };
        std::vector<uint64_t> bad;
        const bool checked = got && check_on_gpu(p, target, bad, fill);
        if (broke) { // stream broken mid-snapshot: nothing committed
            set_err(p, "stream broke while receiving snapshot %llu", (unsigned long long)h.snap_id);
            finish(p, h.snap_id, CKPT_EHIP);
            return;
        }
        if (!checked) {
            set_err(p, "GPU check failed");
            finish(p, h.snap_id, CKPT_EHIP);
            return;
        }
        const auto t2 = clock::now();
        const int32_t result = bad.empty() ? CKPT_OK : CKPT_ECORRUPT;
        {
            std::lock_guard<std::mutex> l(p->m);
            if (bad.empty()) {
                p->env[target] = std::move(env);
                p->snap[target] = h.snap_id;
                p->step[target] = h.step;
                p->committed = target;
            } else {
                p->last_bad = bad;
            }
            p->recv_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
            p->check_ms = std::chrono::duration<double, std::milli>(t2 - t1).count();
        }
        WireAck a;
        std::memcpy(a.magic, kAckMagic, 8);
        a.snap_id = h.snap_id;
        a.status = result;
        a.n_bad = (uint32_t)bad.size();
        a.reserved = 0;
        const bool sent = send_all(fd, &a, sizeof a, deadline) == 0 &&
                          (bad.empty() || send_all(fd, bad.data(), 8 * bad.size(), deadline) == 0);
        finish(p, h.snap_id, result);
        if (!sent) return;
    }
}

void peer_main(ckpt_peer* p)
{
    (void)hipSetDevice(p->device);
    while (!p->stop.load()) {
        pollfd q{p->lfd, POLLIN, 0};
        const int r = ::poll(&q, 1, 200);
        if (r <= 0) continue;
        const int fd = ::accept(p->lfd, nullptr, nullptr);
        if (fd < 0) continue;
        tune_socket(fd);
        {
            std::lock_guard<std::mutex> l(p->m);
            p->cfd = fd;
        }
        // A sender may connect long before its first snapshot: wait for the
        // first bytes without a deadline, answering fetches on other
        // connections meanwhile.
        int w;
        while ((w = wait_readable(p, fd)) == 2) side_connection(p);
        char magic[8];
        if (w == 1 && recv_all(fd, magic, 8, std::chrono::steady_clock::now() + std::chrono::seconds(10)) == 0) {
            if (std::memcmp(magic, kFetchMagic, 8) == 0) serve_fetch(p, fd);
            else if (std::memcmp(magic, kWireMagic, 8) == 0) {
                try {
                    serve(p, fd);
                } catch (const std::bad_alloc&) { // a sender's sizes this host cannot hold
                    set_err(p, "out of host memory while receiving a replica");
                }
            }
            else set_err(p, "unknown request on a new connection");
        }
        {
            std::lock_guard<std::mutex> l(p->m);
            p->cfd = -1;
        }
        ::close(fd);
    }
}

} // namespace

extern "C" {

ckpt_status ckpt_peer_create(const ckpt_config* cfg, uint32_t port, ckpt_peer** out)
{
    if (!out || port > 65535) return CKPT_EINVAL;
    *out = nullptr;
    ckpt_config d{};
    if (cfg) d = *cfg;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || d.device < 0 || d.device >= ndev) return CKPT_EINVAL;
    const int fd = ::socket(AF_INET, SOCK_STREAM, 0);
    if (fd < 0) return CKPT_EHIP;
    int one = 1;
    (void)setsockopt(fd, SOL_SOCKET, SO_REUSEADDR, &one, sizeof one);
    sockaddr_in a{};
    a.sin_family = AF_INET;
    a.sin_port = htons((uint16_t)port);
    a.sin_addr.s_addr = htonl(INADDR_LOOPBACK);
    socklen_t len = sizeof a;
    if (::bind(fd, (sockaddr*)&a, sizeof a) != 0 || ::listen(fd, 4) != 0 ||
        ::getsockname(fd, (sockaddr*)&a, &len) != 0) {
        ::close(fd);
        return CKPT_EHIP;
    }
    ckpt_peer* p = new ckpt_peer();
    p->device = d.device;
    p->group_cfg = d.group_bytes ? d.group_bytes : kPeerDefaultGroup;
    p->grid_cap = d.grid_blocks ? d.grid_blocks : 0x7fffffff;
    p->lfd = fd;
    p->port = ntohs(a.sin_port);
    p->th = std::thread(peer_main, p);
    *out = p;
    return CKPT_OK;
}

ckpt_status ckpt_peer_port(const ckpt_peer* p, uint32_t* port)
{
    if (!p || !port) return CKPT_EINVAL;
    *port = p->port;
    return CKPT_OK;
}

ckpt_status ckpt_peer_destroy(ckpt_peer* p)
{
    if (!p) return CKPT_OK;
    p->stop.store(true);
    {
        std::lock_guard<std::mutex> l(p->m);
        if (p->cfd >= 0) ::shutdown(p->cfd, SHUT_RDWR);
        if (p->sfd >= 0) ::shutdown(p->sfd, SHUT_RDWR);
    }
    if (p->th.joinable()) p->th.join();
    ::close(p->lfd);
    (void)hipSetDevice(p->device);
    free_geometry(p);
    delete p;
    return CKPT_OK;
}

ckpt_status ckpt_peer_wait(ckpt_peer* p, uint64_t snap_id, int32_t timeout_ms, int32_t* result)
{
    if (!p || !result) return CKPT_EINVAL;
    std::unique_lock<std::mutex> l(p->m);
    if (!p->cv.wait_for(l, std::chrono::milliseconds(std::max(0, timeout_ms)),
                        [&] { return p->results.count(snap_id) != 0; }))
        return CKPT_ERANGE;
    *result = p->results[snap_id];
    return CKPT_OK;
}

ckpt_status ckpt_peer_replica(ckpt_peer* p, uint64_t* snap_id, uint64_t* step, const void** data, uint64_t* bytes,
                              const uint64_t** chunk_ids, const uint64_t** sums, uint64_t* n_chunks,
                              const void** envelope, uint64_t* envelope_len)
{
    if (!p) return CKPT_EINVAL;
    std::lock_guard<std::mutex> l(p->m);
    const int b = p->committed;
    if (b < 0) return CKPT_ENOSNAP;
    if (snap_id) *snap_id = p->snap[b];
    if (step) *step = p->step[b];
    if (data) *data = p->h_buf[b];
    if (bytes) *bytes = p->R;
    if (chunk_ids) *chunk_ids = p->ids.data();
    if (sums) *sums = p->h_sums[b];
    if (n_chunks) *n_chunks = p->n;
    if (envelope) *envelope = p->env[b].data();
    if (envelope_len) *envelope_len = p->env[b].size();
    return CKPT_OK;
}

ckpt_status ckpt_peer_last_bad(ckpt_peer* p, uint64_t* bad, uint32_t cap, uint32_t* n)
{
    if (!p || !n) return CKPT_EINVAL;
    std::lock_guard<std::mutex> l(p->m);
    *n = (uint32_t)p->last_bad.size();
    if (bad) std::memcpy(bad, p->last_bad.data(), 8 * std::min<uint64_t>(cap, p->last_bad.size()));
    return CKPT_OK;
}

ckpt_status ckpt_peer_timing(ckpt_peer* p, double* recv_ms, double* check_ms)
{
    if (!p || !recv_ms || !check_ms) return CKPT_EINVAL;
    std::lock_guard<std::mutex> l(p->m);
    *recv_ms = p->recv_ms;
    *check_ms = p->check_ms;
    return CKPT_OK;
}

const char* ckpt_peer_last_error(const ckpt_peer* p)
{
    if (!p) return "null peer";
    static thread_local std::string copy; // the receiver thread may replace the text at any time
    std::lock_guard<std::mutex> l(const_cast<ckpt_peer*>(p)->m);
    copy = p->err;
    return copy.c_str();
}

} // extern "C"
