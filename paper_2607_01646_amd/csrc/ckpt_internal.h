// Internal interface between the libckpt runtime and its gfx950 kernels.
// Not installed; the public ABI is include/ckpt.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ckpt {

// One registered fragment as the kernels see it (32 bytes).
struct FragDev {
    uint64_t ptr;    // device address of the fragment's first byte (any alignment)
    uint64_t nbytes; // fragment bytes
    uint64_t off;    // image offset, a multiple of the alignment (>= 16)
    uint64_t end;    // image offset where the next fragment starts (or the image end)
};

// Tiling of the image.  Tile t covers image bytes [t*T, min((t+1)*T, I)),
// T = 1 << tile_shift divides the chunk size, so no tile crosses a chunk.
struct Geometry {
    uint64_t image_bytes;
    uint64_t n_tiles;
    uint64_t n_chunks;
    uint32_t tile_shift;
    uint32_t tiles_per_chunk; // chunk_bytes >> tile_shift
};

// Partial sums per tile: each wave of a tile's workgroup sums its own slice.
constexpr uint32_t kTileParts = 4;

// Tiles are at most 1 << kMaxTileShift = 8 KiB: each wave's slice of a tile
// is at most one batch of two 16-byte vectors per lane.
constexpr uint32_t kMaxTileShift = 13;

// The tile kernels.  Each covers tiles [t_lo, t_hi) and writes tile t's
// word-sums to partials[t * kTileParts ...] (one per wave slice; partials
// holds kTileParts entries per tile of the image); launches cover whole
// chunks.  grid_cap bounds the workgroups (one per tile when the cap is
// larger).  Non-null t0/t1 are timing events recorded around the dispatch
// itself.
//   pack:     fragment bytes -> image window; image byte x goes to dst + (x - dst_origin);
//             a non-null release is an HSA signal value the launch sets to 0
//             as it starts (after the stream's previous kernel finished)
//   sums:     the sums the pack would compute, from the fragments alone (no image
//             window is written); release as for the pack
//   scatter:  image window -> fragment bytes (image byte x read at src + (x - src_origin))
//   checksum: image window only
hipError_t launch_pack(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, uint8_t* dst, uint64_t dst_origin,
                       unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                       hipEvent_t t1 = nullptr, int64_t* release = nullptr);
hipError_t launch_sums(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, unsigned long long* partials,
                       uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr,
                       int64_t* release = nullptr);
hipError_t launch_scatter(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                          const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                          unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                          hipEvent_t t1 = nullptr);
hipError_t launch_checksum(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                           unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                           hipEvent_t t1 = nullptr);

// Chunk sums of the chunks covered by tiles [t_lo, t_hi): sums_out[c] is the
// sum of the partial sums of the chunk's tiles.  With expected non-null, bad[c] is set to 1
// where sums_out[c] != expected[c] (and to 0 elsewhere).  A non-null release
// is set to 0 as the launch starts, as for the pack.
hipError_t launch_chunk_reduce(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const unsigned long long* partials,
                               unsigned long long* sums_out, const unsigned long long* expected, uint8_t* bad,
                               hipStream_t s, int64_t* release = nullptr);

// Store 0 into *signal_value (an HSA signal's value) once the work enqueued
// on s before this call has completed.
hipError_t launch_release(int64_t* signal_value, hipStream_t s);

// Fill [p, p + n) (p 16-byte aligned, n a multiple of 16) with the 16-byte
// pattern w (the staging canary of ckpt_config.poison).
hipError_t launch_fill16(uint8_t* p, uint64_t n, const uint32_t w[4], hipStream_t s);

// ---- The allocation-free pack (ckpt_pack_noalloc) ----
// Its tables and partial sums live in a fixed device array of the kernel
// file (one per GPU, held until the process ends), laid out as: the fragment
// table (at most kNoallocMaxFrags entries), then the first- and
// last-fragment tables of one group of at most kNoallocGroupTiles tiles, then
// that group's partial sums.  Groups are whole chunks and are packed one
// after another on the caller's stream, reusing the tables.
constexpr uint32_t kNoallocMaxFrags = 65536;
constexpr uint64_t kNoallocGroupTiles = 131072; // 1 GiB of 8 KiB tiles
constexpr uint64_t kNoallocFragsOff = 0;
constexpr uint64_t kNoallocFirstOff = kNoallocFragsOff + (uint64_t)kNoallocMaxFrags * sizeof(FragDev);
constexpr uint64_t kNoallocLastOff = kNoallocFirstOff + kNoallocGroupTiles * 4;
constexpr uint64_t kNoallocPartialsOff = kNoallocLastOff + kNoallocGroupTiles * 4;
constexpr uint64_t kNoallocScratchBytes = kNoallocPartialsOff + kNoallocGroupTiles * kTileParts * 8; // 7 MiB
// Fragment descriptors per upload launch (they travel as kernel arguments).
constexpr uint32_t kUploadBatch = 96;

// Device address of the current device's scratch array, looked up once per
// device with that device current (the array's host-side name is only a
// handle, never a device address).
hipError_t noalloc_scratch(uint8_t** ptr);

// Write descriptors src[0, count) (host memory, count <= kUploadBatch) to
// dst[0, count) on the device, in stream order, through kernel arguments.
hipError_t launch_frag_upload(FragDev* dst, const FragDev* src, uint32_t count, hipStream_t s);

// Tile table of tiles [t_lo, t_hi) over the n fragments in frags (device):
// first[t - t_lo] / last[t - t_lo] = first / last fragment holding a byte of
// tile t (the first fragment whose padded span ends past the tile's first /
// last byte; the last fragment when none does), as the runtime's host planner
// computes it.
hipError_t launch_tile_table(const FragDev* frags, uint32_t n, const Geometry& g, uint64_t t_lo, uint64_t t_hi,
                             uint32_t* first, uint32_t* last, hipStream_t s);

// Tile size rule shared by the planners: the largest power of two no larger
// than 1 << kMaxTileShift (and at least 16) that divides the chunk size.
inline uint32_t tile_shift_for(uint64_t chunk_bytes)
{
    uint32_t ts = 4;
    while (ts < kMaxTileShift && chunk_bytes % (1ull << (ts + 1)) == 0) ++ts;
    return ts;
}

} // namespace ckpt
