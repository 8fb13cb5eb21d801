// ckpt_wire.h -- the host-to-host (H2H) replication stream between a rank
// and its ring peer (paper Sec. V-B "Host-to-host": after the local offload
// completes, a background worker sends the optimizer-state part of the
// snapshot and the metadata envelope to the peer in chunks).  Here the
// transport is a TCP stream; every integer is little-endian.
//
// Per snapshot, sender -> peer:
//   WireHead                       (64 bytes)
//   u64 chunk_id[m]                (ids in the sender's image, increasing)
//   u64 sum[m]                     (the sums stored at pack time)
//   u8  envelope[env_len]          (the snapshot's envelope)
//   u8  data[R]                    (the m chunks back to back; chunk j at
//                                   j * chunk_bytes, only the image's last
//                                   chunk may be short)
// peer -> sender:
//   WireAck                        (32 bytes)
//   u64 bad_chunk_id[n_bad]        (sender's ids of chunks whose sum failed)
//
// A replacement rank fetching its predecessor's state (Sec. V-C, third
// recovery stage) opens a connection of its own:
// replacement -> peer:
//   WireFetch                      (32 bytes)
// peer -> replacement:
//   WireAck                        (status CKPT_OK, or CKPT_ENOSNAP when the
//                                   peer holds no committed replica; snap_id)
//   then, with CKPT_OK, the newest committed replica in the per-snapshot
//   format above (WireHead, ids, sums, envelope, data); the peer then
//   closes the connection.
#pragma once

#include <arpa/inet.h>
#include <errno.h>
#include <netinet/in.h>
#include <netinet/tcp.h>
#include <poll.h>
#include <stdint.h>
#include <string.h>
#include <sys/socket.h>
#include <unistd.h>

#include <algorithm>
#include <chrono>

namespace ckpt {

constexpr char kWireMagic[8] = {'C', 'K', 'P', 'T', 'H', '2', 'H', '1'};
constexpr char kAckMagic[8] = {'C', 'K', 'P', 'T', 'A', 'C', 'K', '1'};
constexpr char kFetchMagic[8] = {'C', 'K', 'P', 'T', 'G', 'E', 'T', '1'};

struct WireHead {
    char magic[8];
    uint64_t snap_id;
    uint64_t step;
    uint64_t chunk_bytes;
    uint64_t image_bytes; // sender's full image
    uint64_t m;           // chunks in this replica
    uint64_t replica_bytes;
    uint64_t env_len;
};
static_assert(sizeof(WireHead) == 64, "wire header is 64 bytes");

struct WireAck {
    char magic[8];
    uint64_t snap_id;
    int32_t status; // CKPT_OK, CKPT_ECORRUPT, or another CKPT_E* code
    uint32_t n_bad;
    uint64_t reserved;
};
static_assert(sizeof(WireAck) == 32, "wire ack is 32 bytes");

struct WireFetch {
    char magic[8];
    uint64_t reserved[3];
};
static_assert(sizeof(WireFetch) == 32, "fetch request is 32 bytes");

// Replica bytes of m chunks of chunk_bytes each, the last one possibly the
// image's short last chunk.
inline uint64_t replica_bytes(const uint64_t* ids, uint64_t m, uint64_t chunk_bytes, uint64_t image_bytes)
{
    if (m == 0) return 0;
    const uint64_t last = ids[m - 1];
    const uint64_t last_len = (last + 1) * chunk_bytes <= image_bytes ? chunk_bytes : image_bytes - last * chunk_bytes;
    return (m - 1) * chunk_bytes + last_len;
}

// Blocking send / receive of exactly n bytes.  Return 0 on success, -1 on
// error or timeout, -2 when the other side closed.  `deadline` bounds the
// wait for progress: every piece moved pushes it to at least kWireGrace from
// now, so a transfer may take as long as it needs while data flows and only a
// stalled connection times out.  The caller's deadline variable is updated,
// so a sequence of calls shares it.
constexpr auto kWireGrace = std::chrono::seconds(30);

inline int wire_wait(int fd, short ev, std::chrono::steady_clock::time_point deadline)
{
    for (;;) {
        const auto left = std::chrono::duration_cast<std::chrono::milliseconds>(deadline -
                                                                                std::chrono::steady_clock::now());
        if (left.count() <= 0) return -1;
        pollfd p{fd, ev, 0};
        const int r = ::poll(&p, 1, (int)std::min<long long>(left.count(), 1000));
        if (r > 0) return 0;
        if (r < 0 && errno != EINTR) return -1;
    }
}

inline void wire_progress(std::chrono::steady_clock::time_point& deadline)
{
    deadline = std::max(deadline, std::chrono::steady_clock::now() + kWireGrace);
}

inline int send_all(int fd, const void* buf, uint64_t n, std::chrono::steady_clock::time_point& deadline)
{
    const uint8_t* p = (const uint8_t*)buf;
    while (n) {
        if (wire_wait(fd, POLLOUT, deadline)) return -1;
        const ssize_t k = ::send(fd, p, (size_t)std::min<uint64_t>(n, 1ull << 30), MSG_NOSIGNAL);
        if (k < 0) {
            if (errno == EINTR || errno == EAGAIN) continue;
            return -1;
        }
        p += k;
        n -= (uint64_t)k;
        wire_progress(deadline);
    }
    return 0;
}

inline int recv_all(int fd, void* buf, uint64_t n, std::chrono::steady_clock::time_point& deadline)
{
    uint8_t* p = (uint8_t*)buf;
    while (n) {
        if (wire_wait(fd, POLLIN, deadline)) return -1;
        const ssize_t k = ::recv(fd, p, (size_t)std::min<uint64_t>(n, 1ull << 30), 0);
        if (k == 0) return -2;
        if (k < 0) {
            if (errno == EINTR || errno == EAGAIN) continue;
            return -1;
        }
        p += k;
        n -= (uint64_t)k;
        wire_progress(deadline);
    }
    return 0;
}

// One-off calls with a deadline of their own.
inline int send_all(int fd, const void* buf, uint64_t n, std::chrono::steady_clock::time_point&& deadline)
{
    auto d = deadline;
    return send_all(fd, buf, n, d);
}

inline int recv_all(int fd, void* buf, uint64_t n, std::chrono::steady_clock::time_point&& deadline)
{
    auto d = deadline;
    return recv_all(fd, buf, n, d);
}

inline void tune_socket(int fd)
{
    int one = 1;
    (void)setsockopt(fd, IPPROTO_TCP, TCP_NODELAY, &one, sizeof one);
    int buf = 16 << 20;
    (void)setsockopt(fd, SOL_SOCKET, SO_SNDBUF, &buf, sizeof buf);
    (void)setsockopt(fd, SOL_SOCKET, SO_RCVBUF, &buf, sizeof buf);
}

// Connect to a dotted IPv4 address.  Returns the socket, or -1 with errno
// set (EINVAL for an address that does not parse).
inline int dial(const char* host, uint32_t port)
{
    sockaddr_in a{};
    a.sin_family = AF_INET;
    a.sin_port = htons((uint16_t)port);
    if (inet_pton(AF_INET, host, &a.sin_addr) != 1) {
        errno = EINVAL;
        return -1;
    }
    const int fd = ::socket(AF_INET, SOCK_STREAM, 0);
    if (fd < 0) return -1;
    tune_socket(fd);
    if (::connect(fd, (sockaddr*)&a, sizeof a) != 0) {
        const int e = errno;
        ::close(fd);
        errno = e;
        return -1;
    }
    return fd;
}

} // namespace ckpt
