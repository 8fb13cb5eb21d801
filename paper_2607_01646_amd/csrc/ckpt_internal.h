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
//   pack:     fragment bytes -> image window; image byte x goes to dst + (x - dst_origin)
//   scatter:  image window -> fragment bytes (image byte x read at src + (x - src_origin))
//   checksum: image window only
hipError_t launch_pack(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, uint8_t* dst, uint64_t dst_origin,
                       unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                       hipEvent_t t1 = nullptr);
hipError_t launch_scatter(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                          const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                          unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                          hipEvent_t t1 = nullptr);
hipError_t launch_checksum(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                           unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0 = nullptr,
                           hipEvent_t t1 = nullptr);

// Chunk sums of the chunks covered by tiles [t_lo, t_hi): sums_out[c] is the
// sum of the partial sums of the chunk's tiles.  With expected non-null, bad[c] is set to 1
// where sums_out[c] != expected[c] (and to 0 elsewhere).
hipError_t launch_chunk_reduce(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const unsigned long long* partials,
                               unsigned long long* sums_out, const unsigned long long* expected, uint8_t* bad,
                               hipStream_t s);

// Store 0 into *signal_value (an HSA signal's value) once the work enqueued
// on s before this call has completed.
hipError_t launch_release(int64_t* signal_value, hipStream_t s);

} // namespace ckpt
