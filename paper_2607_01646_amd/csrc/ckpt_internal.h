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

// Pack fragments into an image window and sum its chunks.
// Tiles [t_lo, t_hi) (whole chunks) are processed; image byte x is written to
// dst + (x - dst_origin); partials[t] receives tile t's sum and sums_out[c]
// the word-sum of chunk c.  Two kernel launches on stream s.
hipError_t launch_pack(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, uint8_t* dst, uint64_t dst_origin,
                       unsigned long long* partials, unsigned long long* sums_out, uint32_t grid_cap, hipStream_t s);

// Scatter an image window back into the fragments, recompute chunk sums and
// compare them with expected[]: recomputed[c] and bad[c] (1 = mismatch).
hipError_t launch_scatter_verify(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                                 const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src,
                                 uint64_t src_origin, unsigned long long* partials,
                                 const unsigned long long* expected, unsigned long long* recomputed, uint8_t* bad,
                                 uint32_t grid_cap, hipStream_t s);

// Recompute chunk sums of an image window only (no fragments touched).
hipError_t launch_checksum_verify(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src,
                                  uint64_t src_origin, unsigned long long* partials,
                                  const unsigned long long* expected, unsigned long long* recomputed, uint8_t* bad,
                                  uint32_t grid_cap, hipStream_t s);

// Store 0 into *signal_value (an HSA signal's value) once the work enqueued
// on s before this call has completed.
hipError_t launch_release(int64_t* signal_value, hipStream_t s);

} // namespace ckpt
