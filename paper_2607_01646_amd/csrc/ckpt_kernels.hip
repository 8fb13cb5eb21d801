// ckpt_kernels.hip -- gfx950 kernels of libckpt.
//
// Four bandwidth-bound tile kernels over the snapshot image (the contiguous
// buffer of the D2H phase, paper Sec. V-B):
//   PACK     gather fragment bytes into the image window and sum each chunk,
//   SCATTER  write an image window back into the fragments (recovery, paper
//            Sec. VI-E) while re-summing and checking each chunk,
//   VERIFY   re-sum and check an image window only,
//   SUMS     sum each chunk of the image the fragments would make, reading
//            the fragments only (direct D2H: the DMA engines gather the
//            fragments into the host image themselves).
// The chunk sum is the sum of the chunk's 8-byte little-endian words modulo
// 2^64 (padding included).  Bytes are moved as opaque 128-bit words: no
// floating-point instruction touches them, so NaN payloads, -0 and
// subnormals pass unchanged.
//
// Work split.  The image is cut into power-of-two tiles of at most 8 KiB
// that never cross a chunk.  A workgroup of 256 lanes (4 wave64) takes one
// tile (a separate instantiation strides over tiles when the grid is
// capped).  Wave w owns the tile's 2 KiB slice w, and each lane moves two
// 16-byte vectors of it, both loads issued before the stores; a tile shorter
// than 8 KiB leaves its last waves idle.  Consecutive tiles go to
// consecutive workgroups, which the hardware deals out round-robin over the
// 8 XCDs (measured faster than giving each XCD a contiguous range).  A tile
// inside one 16-byte-aligned fragment takes an unrolled non-temporal stream;
// otherwise each vector finds its fragment (binary search over the tile's
// fragment offsets in LDS), loads aligned 16-byte blocks and funnel-shifts
// them when the fragment is misaligned, masks the fragment tail and writes
// zeros for padding.
// Sum reduction: per lane in 64 bits, across the wave with lane shuffles;
// each wave stores its slice's sum (four partial sums per tile), with no
// workgroup barrier on the streaming path.  A small second kernel adds the
// partial sums of each chunk (and, when checking, compares with the stored
// sum).  The hot kernel thus has no atomics and no device-scope fence: on
// gfx950 such a fence writes back and invalidates the XCD's L2, which per
// tile would cost more than the tile's own traffic.
// Addition modulo 2^64 is associative and commutative, so any order of
// tiles gives the same bits.
#include <hip/hip_ext.h>

#include <algorithm>
#include <mutex>

#include "ckpt_internal.h"

namespace ckpt {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBlock = 256;      // lanes per workgroup (4 wave64)
constexpr int kLdsFrags = 256;  // fragment offsets cached per tile (an 8 KiB tile holds at most 33 non-empty ones)
constexpr int kUnroll = 2;      // 16-byte vectors per lane per batch: one batch covers an 8 KiB tile

enum Mode { PACK = 0, SCATTER = 1, VERIFY = 2, SUMS = 3 };

struct Args {
    const FragDev* frags;
    const uint32_t* tile_first; // first fragment holding a byte of tile t
    const uint32_t* tile_last;  // last fragment holding a byte of tile t
    Geometry g;
    uint64_t t_lo, t_hi;
    uint8_t* img; // PACK: destination window; SCATTER/VERIFY: source window; SUMS: unused
    uint64_t origin;
    unsigned long long* partials; // one sum per tile
    int64_t* release;             // PACK, SUMS: an HSA signal value to set to 0 (or null)
};

struct ReduceArgs {
    const unsigned long long* partials;
    uint64_t c_lo, c_hi; // chunks of this launch
    uint64_t n_tiles;
    uint32_t tiles_per_chunk;
    unsigned long long* sums_out; // PACK: chunk sums; SCATTER/VERIFY: recomputed sums
    const unsigned long long* expected; // null when only summing
    uint8_t* bad;
    int64_t* release; // an HSA signal value to set to 0 at the start (or null)
};

// Lane 0 of workgroup 0 stores 0 into *release: a system-scope release of
// "the kernels before this one on the stream have finished".  A kernel
// starts only once the previous kernel of its stream has completed, and a
// kernel's completion releases its writes at device scope (on a multi-XCD
// part that writes the L2 back), so a DMA engine waiting for the signal
// reads that kernel's bytes.  Carried by the next launch, it saves a
// one-lane kernel and a dispatch gap per chunk group.  The tile kernel does
// it after workgroup 0's tile: ahead of the tile, the test of the pointer
// put a second dependent argument load in front of every workgroup's work.
__device__ __forceinline__ void release_signal(int64_t* release)
{
    if (release && blockIdx.x == 0 && threadIdx.x == 0)
        __hip_atomic_store(release, (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

__device__ __forceinline__ unsigned long long vsum(u32x4 v)
{
    const unsigned long long w0 = (unsigned long long)v.x | ((unsigned long long)v.y << 32);
    const unsigned long long w1 = (unsigned long long)v.z | ((unsigned long long)v.w << 32);
    return w0 + w1;
}

__device__ __forceinline__ u32x4 load16(uint64_t a) { return *reinterpret_cast<const u32x4*>(a); }

__device__ __forceinline__ u32x4 make4(uint64_t r0, uint64_t r1)
{
    u32x4 v;
    v.x = (unsigned)r0;
    v.y = (unsigned)(r0 >> 32);
    v.z = (unsigned)r1;
    v.w = (unsigned)(r1 >> 32);
    return v;
}

// Bytes [p, p+16) of a fragment (ptr, nbytes), p a multiple of 16; bytes at
// or past nbytes read as zero.  Only aligned 16-byte blocks that contain at
// least one byte of the fragment are loaded.
__device__ u32x4 fetch_general(uint64_t ptr, uint64_t nbytes, uint64_t p)
{
    u32x4 r = {0u, 0u, 0u, 0u};
    if (p >= nbytes) return r;
    const uint64_t left = nbytes - p;
    const uint64_t a = ptr + p;
    uint32_t s = (uint32_t)(a & 15);
    if (s == 0 && left >= 16) return load16(a);
    const uint64_t a0 = a - s;
    const u32x4 lo = load16(a0); // holds byte a, a fragment byte
    u32x4 hi = r;
    if (s != 0 && a0 + 16 < ptr + nbytes) hi = load16(a0 + 16); // first byte is a fragment byte
    uint64_t w0 = (uint64_t)lo.x | ((uint64_t)lo.y << 32);
    uint64_t w1 = (uint64_t)lo.z | ((uint64_t)lo.w << 32);
    uint64_t w2 = (uint64_t)hi.x | ((uint64_t)hi.y << 32);
    const uint64_t w3 = (uint64_t)hi.z | ((uint64_t)hi.w << 32);
    if (s >= 8) {
        w0 = w1;
        w1 = w2;
        w2 = w3;
        s -= 8;
    }
    uint64_t r0 = w0, r1 = w1;
    if (s != 0) {
        r0 = (w0 >> (8 * s)) | (w1 << (64 - 8 * s));
        r1 = (w1 >> (8 * s)) | (w2 << (64 - 8 * s));
    }
    if (left < 16) {
        if (left < 8) {
            r0 &= (1ull << (8 * left)) - 1;
            r1 = 0;
        } else if (left == 8) {
            r1 = 0;
        } else {
            r1 &= (1ull << (8 * (left - 8))) - 1;
        }
    }
    return make4(r0, r1);
}

// Write the fragment bytes among [p, p+16) from v; p a multiple of 16.
// Stores never touch a byte outside the fragment.
__device__ void store_general(uint64_t ptr, uint64_t nbytes, uint64_t p, u32x4 v)
{
    if (p >= nbytes) return;
    const uint64_t left = nbytes - p;
    const uint64_t d = ptr + p;
    if ((d & 15) == 0 && left >= 16) {
        *reinterpret_cast<u32x4*>(d) = v;
        return;
    }
    const uint32_t nb = left < 16 ? (uint32_t)left : 16u;
    const unsigned w[4] = {v.x, v.y, v.z, v.w};
    if ((d & 3) == 0 && (nb & 3) == 0) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (4u * k < nb) reinterpret_cast<unsigned*>(d)[k] = w[k];
    } else if ((d & 1) == 0 && (nb & 1) == 0) {
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (2u * k < nb) reinterpret_cast<unsigned short*>(d)[k] = (unsigned short)(w[k >> 1] >> (16 * (k & 1)));
    } else {
#pragma unroll
        for (int k = 0; k < 16; ++k)
            if ((uint32_t)k < nb) reinterpret_cast<unsigned char*>(d)[k] = (unsigned char)(w[k >> 2] >> (8 * (k & 3)));
    }
}

template <bool NT>
__device__ __forceinline__ u32x4 ld(const u32x4* p)
{
    if (NT) return __builtin_nontemporal_load(p);
    return *p;
}

// Streaming 16-byte store: non-temporal and device scope (sc1).  The device
// scope sends the line past the XCD's L2 at once; on the 1.3B shard's pack
// this measured ~1% faster than the non-temporal store alone (same bytes and
// sums; sc1 on the loads was slower).  The address is a device pointer into
// global memory (fragments or the image), so the global form applies.
// A store of more than 8 bytes reads its data registers after issue: on the
// gfx940 family a VALU write to them needs two wait states first.  The
// compiler keeps that distance for its own stores but cannot see into this
// one, so the two wait states (s_nop 1) come with it.
__device__ __forceinline__ void st_stream(u32x4 v, u32x4* p)
{
    asm volatile("global_store_dwordx4 %0, %1, off nt sc1\n\ts_nop 1" : : "v"(p), "v"(v) : "memory");
}

template <bool NT>
__device__ __forceinline__ void st(u32x4 v, u32x4* p)
{
    if (NT) st_stream(v, p);
    else *p = v;
}

// One wave's slice of a tile inside one 16-byte-aligned span: the n <= 64 *
// UNROLL vectors at s (copied to d unless d is null) and their sum.  Lane l
// takes vectors l, l + 64, ...; every guarded load is issued before the
// first store, each a contiguous 1 KiB run per wave.  Written out without
// a loop: a runtime trip count here measured ~1.5% slower.
template <int UNROLL, bool NTL, bool NTS, bool STORE>
__device__ __forceinline__ unsigned long long slice_stream(const u32x4* __restrict__ s, u32x4* __restrict__ d,
                                                           uint32_t n, uint32_t lane)
{
    u32x4 r[UNROLL];
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
        if (lane + u * 64 < n) r[u] = ld<NTL>(s + lane + u * 64);
    unsigned long long acc = 0;
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
        if (lane + u * 64 < n) {
            if (STORE) st<NTS>(r[u], d + lane + u * 64);
            acc += vsum(r[u]);
        }
    return acc;
}

__device__ __forceinline__ unsigned long long shfl_xor64(unsigned long long v, int m)
{
    const unsigned lo = __shfl_xor((unsigned)v, m);
    const unsigned hi = __shfl_xor((unsigned)(v >> 32), m);
    return ((unsigned long long)hi << 32) | lo;
}

// Sum over one wave; every lane gets the result.
__device__ __forceinline__ unsigned long long wave_sum(unsigned long long v)
{
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) v += shfl_xor64(v, m);
    return v;
}

// Sum over the workgroup; the result is valid in thread 0.
template <int BLOCK>
__device__ __forceinline__ unsigned long long block_sum(unsigned long long v, unsigned long long* s_red)
{
    v = wave_sum(v);
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) s_red[wave] = v;
    __syncthreads();
    unsigned long long r = 0;
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < BLOCK / 64; ++w) r += s_red[w];
    }
    __syncthreads();
    return r;
}

// Index (relative to f0) of the fragment holding image byte x: the largest k
// with s_off[k] <= x.  Empty fragments share their offset with the next
// fragment, so the largest such k is never an empty one.
__device__ __forceinline__ uint32_t find_frag_lds(const uint64_t* s_off, uint32_t n, uint64_t x)
{
    uint32_t lo = 0, hi = n - 1;
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= x) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

__device__ __forceinline__ uint32_t find_frag_global(const FragDev* frags, uint32_t f0, uint32_t f1, uint64_t x)
{
    uint32_t lo = f0, hi = f1;
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo + 1) >> 1);
        if (frags[mid].off <= x) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// One tile: wave w owns vectors [w * slice, (w + 1) * slice) of it and
// stores that slice's sum to partials[t * WAVES + w].
template <int MODE, int BLOCK, int UNROLL, bool NTL, bool NTS>
__device__ __forceinline__ void do_tile(const Args& a, uint64_t t, uint64_t* s_off)
{
    static_assert(BLOCK / 64 == kTileParts, "one partial sum per wave");
    static_assert(BLOCK * UNROLL * 16 == (1u << kMaxTileShift), "one batch per lane covers the largest tile");
    constexpr uint32_t WAVES = BLOCK / 64;
    constexpr uint32_t kSlice = 64 * UNROLL; // vectors per wave slice
    const uint32_t tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    {
        const uint64_t base = t << a.g.tile_shift;
        uint64_t end = base + (1ull << a.g.tile_shift);
        if (end > a.g.image_bytes) end = a.g.image_bytes;
        const uint32_t nvec = (uint32_t)((end - base) >> 4);
        // Wave w owns vectors [v0, v1) of the tile (empty past a short tile's end).
        const uint32_t v0 = w * kSlice;
        const uint32_t v1 = v0 + kSlice < nvec ? v0 + kSlice : (nvec > v0 ? nvec : v0);
        uint8_t* win = MODE == SUMS ? nullptr : a.img + (base - a.origin);
        unsigned long long acc = 0;
        if (MODE == VERIFY) {
            acc = slice_stream<UNROLL, NTL, NTS, false>(reinterpret_cast<const u32x4*>(win) + v0, nullptr, v1 - v0, lane);
        } else {
            const uint32_t f0 = a.tile_first[t], f1 = a.tile_last[t];
            if (f0 == f1) {
                const FragDev F = a.frags[f0];
                const uint64_t p0 = base - F.off;
                if ((F.ptr & 15) == 0 && p0 + (end - base) <= F.nbytes) {
                    u32x4* fr = reinterpret_cast<u32x4*>(F.ptr + p0) + v0;
                    if (MODE == SUMS)
                        acc = slice_stream<UNROLL, NTL, NTS, false>(fr, nullptr, v1 - v0, lane);
                    else if (MODE == PACK)
                        acc = slice_stream<UNROLL, NTL, NTS, true>(fr, reinterpret_cast<u32x4*>(win) + v0, v1 - v0,
                                                                   lane);
                    else
                        acc = slice_stream<UNROLL, NTL, NTS, true>(reinterpret_cast<u32x4*>(win) + v0, fr, v1 - v0,
                                                                   lane);
                } else {
                    for (uint32_t v = v0 + lane; v < v1; v += 64) {
                        const uint64_t p = p0 + 16ull * v;
                        if (MODE == SUMS) {
                            acc += vsum(fetch_general(F.ptr, F.nbytes, p));
                        } else if (MODE == PACK) {
                            const u32x4 r = fetch_general(F.ptr, F.nbytes, p);
                            st_stream(r, reinterpret_cast<u32x4*>(win) + v);
                            acc += vsum(r);
                        } else {
                            u32x4* wv = reinterpret_cast<u32x4*>(win) + v;
                            const u32x4 r = __builtin_nontemporal_load(wv);
                            store_general(F.ptr, F.nbytes, p, r);
                            acc += vsum(r);
                        }
                    }
                }
            } else {
                // Several fragments: their offsets go to LDS for the search.
                // Both barriers are workgroup-uniform (f0, f1 depend on t only);
                // the first keeps the previous tile's readers ahead of the refill.
                const uint32_t nf = f1 - f0 + 1;
                const bool in_lds = nf <= (uint32_t)kLdsFrags;
                __syncthreads();
                if (in_lds) {
                    for (uint32_t k = tid; k < nf; k += BLOCK) s_off[k] = a.frags[f0 + k].off;
                }
                __syncthreads();
                for (uint32_t v = v0 + lane; v < v1; v += 64) {
                    const uint64_t x = base + 16ull * v;
                    const uint32_t i = in_lds ? f0 + find_frag_lds(s_off, nf, x) : find_frag_global(a.frags, f0, f1, x);
                    const FragDev F = a.frags[i];
                    const uint64_t p = x - F.off;
                    if (MODE == SUMS) {
                        acc += vsum(fetch_general(F.ptr, F.nbytes, p));
                    } else if (MODE == PACK) {
                        const u32x4 r = fetch_general(F.ptr, F.nbytes, p);
                        st_stream(r, reinterpret_cast<u32x4*>(win) + v);
                        acc += vsum(r);
                    } else {
                        u32x4* wv = reinterpret_cast<u32x4*>(win) + v;
                        const u32x4 r = __builtin_nontemporal_load(wv);
                        store_general(F.ptr, F.nbytes, p, r);
                        acc += vsum(r);
                    }
                }
            }
        }
        acc = wave_sum(acc);
        if (lane == 0) a.partials[t * WAVES + w] = acc;
    }
}

// Without LOOP the grid has one workgroup per tile and each takes exactly
// one (a grid-stride loop around the same body measured ~3% slower on the
// default launch); with LOOP a capped grid strides over the tiles.
template <int MODE, bool LOOP, int BLOCK = kBlock, int UNROLL = kUnroll, bool NTL = true, bool NTS = true>
__global__ __launch_bounds__(BLOCK) void tile_kernel(Args a)
{
    __shared__ uint64_t s_off[kLdsFrags];
    const uint64_t first = blockIdx.x;
    if (LOOP) {
        for (uint64_t t = a.t_lo + first; t < a.t_hi; t += gridDim.x) do_tile<MODE, BLOCK, UNROLL, NTL, NTS>(a, t, s_off);
    } else {
        const uint64_t t = a.t_lo + first;
        if (t < a.t_hi) do_tile<MODE, BLOCK, UNROLL, NTL, NTS>(a, t, s_off);
    }
    if (MODE == PACK || MODE == SUMS) release_signal(a.release);
}

// SUMS over runs of kSumsTiles tiles: workgroup b takes tiles
// [t_lo + kSumsTiles * b, t_lo + kSumsTiles * (b + 1)).  When they are all
// full 8 KiB tiles inside one 16-byte-aligned fragment, the workgroup streams
// them in one batch: wave w owns a quarter of the run, kSumsTiles 2 KiB
// slices (two vectors per lane per slice, all loads issued first), and
// stores each slice's sum in that slice's partial slot.  Otherwise each tile
// takes the per-tile path.  A read-only stream has no stores to keep the
// memory busy while a workgroup waits for its table lookups, so it needs
// more bytes per workgroup than the pack.  Measured on the 1.3B shard's
// layout: one 8 KiB tile per workgroup ~6.15 TB/s, two ~6.6 TB/s, four
// ~6.4 TB/s, eight ~6.0 TB/s.
constexpr uint32_t kSumsTiles = 2;

__global__ __launch_bounds__(kBlock) void sums_run_kernel(Args a)
{
    __shared__ uint64_t s_off[kLdsFrags];
    constexpr uint32_t kRun = kSumsTiles << kMaxTileShift; // bytes per workgroup
    const uint64_t t = a.t_lo + (uint64_t)kSumsTiles * blockIdx.x; // < t_hi (grid: ceil(tiles / kSumsTiles))
    bool fast = false;
    FragDev F{};
    if (t + kSumsTiles <= a.t_hi && a.g.tile_shift == kMaxTileShift) {
        const uint32_t f0 = a.tile_first[t], f1 = a.tile_last[t + kSumsTiles - 1];
        if (f0 == f1) { // the run holds bytes of this fragment only (or its padding)
            F = a.frags[f0];
            fast = (F.ptr & 15) == 0 && (t << kMaxTileShift) - F.off + kRun <= F.nbytes;
        }
    }
    if (fast) {
        const uint32_t lane = threadIdx.x & 63, w = threadIdx.x >> 6;
        const u32x4* src = reinterpret_cast<const u32x4*>(F.ptr + ((t << kMaxTileShift) - F.off)) +
                           w * (kSumsTiles * 128);
        u32x4 r[2 * kSumsTiles];
#pragma unroll
        for (uint32_t u = 0; u < 2 * kSumsTiles; ++u) r[u] = __builtin_nontemporal_load(src + lane + u * 64);
        unsigned long long* p = a.partials + t * kTileParts + w * kSumsTiles; // slice w * kSumsTiles of the run
#pragma unroll
        for (uint32_t k = 0; k < kSumsTiles; ++k) {
            const unsigned long long sk = wave_sum(vsum(r[2 * k]) + vsum(r[2 * k + 1]));
            if (lane == 0) p[k] = sk;
        }
    } else {
        for (uint32_t k = 0; k < kSumsTiles && t + k < a.t_hi; ++k)
            do_tile<SUMS, kBlock, kUnroll, true, true>(a, t + k, s_off);
    }
    release_signal(a.release);
}

// One workgroup per chunk: add the chunk's tile sums; when expected is given,
// also flag a mismatch.  A 64 MiB chunk has 32768 partial sums; each lane
// keeps eight independent loads in flight (a plain strided loop with one
// load at a time took ~70 us per 1 GiB of chunks).
constexpr int kReduceBlock = 1024;
constexpr int kReduceUnroll = 8;

__global__ __launch_bounds__(kReduceBlock) void chunk_reduce_kernel(ReduceArgs r)
{
    __shared__ unsigned long long s_red[kReduceBlock / 64];
    release_signal(r.release);
    const uint64_t c = r.c_lo + blockIdx.x;
    const uint64_t t0 = c * r.tiles_per_chunk;
    uint64_t t1 = t0 + r.tiles_per_chunk;
    if (t1 > r.n_tiles) t1 = r.n_tiles;
    const uint64_t end = t1 * kTileParts;
    uint64_t k = t0 * kTileParts + threadIdx.x;
    unsigned long long acc = 0;
    for (; k + (kReduceUnroll - 1) * kReduceBlock < end; k += kReduceUnroll * kReduceBlock) {
        unsigned long long v[kReduceUnroll];
#pragma unroll
        for (int u = 0; u < kReduceUnroll; ++u) v[u] = r.partials[k + u * kReduceBlock];
#pragma unroll
        for (int u = 0; u < kReduceUnroll; ++u) acc += v[u];
    }
    for (; k < end; k += kReduceBlock) acc += r.partials[k];
    const unsigned long long s = block_sum<kReduceBlock>(acc, s_red);
    if (threadIdx.x == 0) {
        r.sums_out[c] = s;
        if (r.expected) r.bad[c] = (s != r.expected[c]) ? 1 : 0;
    }
}

// With timing events, the launch records them around the dispatch itself
// (the same interval a kernel trace reports).
template <int MODE>
hipError_t launch_tiles(const Args& a, uint32_t grid_cap, hipStream_t s, hipEvent_t t0, hipEvent_t t1)
{
    if (a.t_hi <= a.t_lo) return hipSuccess;
    const uint64_t n = a.t_hi - a.t_lo;
    const uint32_t grid = (uint32_t)(n < grid_cap ? n : grid_cap);
    void (*kern)(Args) = grid == n ? tile_kernel<MODE, false> : tile_kernel<MODE, true>;
    if (t0 && t1)
        hipExtLaunchKernelGGL(kern, dim3(grid), dim3(kBlock), 0, s, t0, t1, 0, a);
    else
        hipLaunchKernelGGL(kern, dim3(grid), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

// One lane: publish "this point of the stream has been reached" to a DMA
// engine by storing 0 into an HSA signal value it polls.  The store is a
// system-scope release; the kernels before it on the stream have finished
// and their writes are past the L2 (the stream's kernel boundaries release
// at device scope, which on a multi-XCD part writes the L2 back).
__global__ void release_signal_kernel(int64_t* value)
{
    __hip_atomic_store(value, (int64_t)0, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(256) void fill16_kernel(u32x4* p, uint64_t n16, u32x4 w)
{
    for (uint64_t k = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; k < n16; k += (uint64_t)gridDim.x * blockDim.x)
        p[k] = w;
}

// ---- allocation-free pack: scratch, table upload, tile table ----

struct FragBatch {
    uint32_t count;
    FragDev f[kUploadBatch];
};

__global__ __launch_bounds__(128) void frag_upload_kernel(FragDev* dst, FragBatch b)
{
    const uint32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < b.count) dst[k] = b.f[k];
}

// One lane per tile: binary search for the first fragment whose padded span
// [off, end) ends past the tile's first byte, and for the first one ending
// past its last byte (end[] never decreases; empty fragments have empty spans).
__global__ __launch_bounds__(256) void tile_table_kernel(const FragDev* frags, uint32_t n, Geometry g, uint64_t t_lo,
                                                         uint64_t t_hi, uint32_t* first, uint32_t* last)
{
    const uint64_t t = t_lo + (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= t_hi) return;
    const uint64_t x0 = t << g.tile_shift;
    uint64_t x1 = x0 + (1ull << g.tile_shift);
    if (x1 > g.image_bytes) x1 = g.image_bytes;
    --x1;
    uint32_t r[2];
    const uint64_t xs[2] = {x0, x1};
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        uint32_t lo = 0, hi = n - 1; // the answer lies in [lo, hi]; n - 1 when no span ends past x
        while (lo < hi) {
            const uint32_t mid = lo + ((hi - lo) >> 1);
            if (frags[mid].end > xs[k]) hi = mid;
            else lo = mid + 1;
        }
        r[k] = lo;
    }
    first[t - t_lo] = r[0];
    last[t - t_lo] = r[1];
}

// The scratch of ckpt_pack_noalloc (layout in ckpt_internal.h).  Host code
// reaches it only through the address noalloc_scratch() looks up.
static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

} // namespace

hipError_t noalloc_scratch(uint8_t** ptr)
{
    constexpr int kMaxDevices = 64;
    static std::mutex m;
    static uint8_t* addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> l(m);
    if (!addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = (uint8_t*)p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

hipError_t launch_fill16(uint8_t* p, uint64_t n, const uint32_t w[4], hipStream_t s)
{
    if (n == 0) return hipSuccess;
    if (((uintptr_t)p & 15) || (n & 15)) return hipErrorInvalidValue;
    u32x4 v;
    v.x = w[0];
    v.y = w[1];
    v.z = w[2];
    v.w = w[3];
    const uint64_t n16 = n >> 4;
    const uint64_t blocks = std::min<uint64_t>((n16 + 255) / 256, 8192);
    hipLaunchKernelGGL(fill16_kernel, dim3((uint32_t)blocks), dim3(256), 0, s, reinterpret_cast<u32x4*>(p), n16, v);
    return hipGetLastError();
}

hipError_t launch_frag_upload(FragDev* dst, const FragDev* src, uint32_t count, hipStream_t s)
{
    if (count == 0) return hipSuccess;
    if (count > kUploadBatch) return hipErrorInvalidValue;
    FragBatch b;
    b.count = count;
    for (uint32_t k = 0; k < count; ++k) b.f[k] = src[k];
    hipLaunchKernelGGL(frag_upload_kernel, dim3(1), dim3(128), 0, s, dst, b);
    return hipGetLastError();
}

hipError_t launch_tile_table(const FragDev* frags, uint32_t n, const Geometry& g, uint64_t t_lo, uint64_t t_hi,
                             uint32_t* first, uint32_t* last, hipStream_t s)
{
    if (t_hi <= t_lo || n == 0) return hipSuccess;
    const uint64_t nt = t_hi - t_lo;
    hipLaunchKernelGGL(tile_table_kernel, dim3((uint32_t)((nt + 255) / 256)), dim3(256), 0, s, frags, n, g, t_lo, t_hi,
                       first, last);
    return hipGetLastError();
}

hipError_t launch_release(int64_t* signal_value, hipStream_t s)
{
    hipLaunchKernelGGL(release_signal_kernel, dim3(1), dim3(1), 0, s, signal_value);
    return hipGetLastError();
}

hipError_t launch_pack(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, uint8_t* dst, uint64_t dst_origin,
                       unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0, hipEvent_t t1,
                       int64_t* release)
{
    Args a{frags, tile_first, tile_last, g, t_lo, t_hi, dst, dst_origin, partials, release};
    return launch_tiles<PACK>(a, grid_cap, s, t0, t1);
}

hipError_t launch_sums(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                       const Geometry& g, uint64_t t_lo, uint64_t t_hi, unsigned long long* partials,
                       uint32_t grid_cap, hipStream_t s, hipEvent_t t0, hipEvent_t t1, int64_t* release)
{
    Args a{frags, tile_first, tile_last, g, t_lo, t_hi, nullptr, 0, partials, release};
    if (t_hi <= t_lo) return hipSuccess;
    const uint64_t runs = (t_hi - t_lo + kSumsTiles - 1) / kSumsTiles;
    if (runs > grid_cap) return launch_tiles<SUMS>(a, grid_cap, s, t0, t1); // a capped grid strides over tiles
    if (t0 && t1)
        hipExtLaunchKernelGGL(sums_run_kernel, dim3((uint32_t)runs), dim3(kBlock), 0, s, t0, t1, 0, a);
    else
        hipLaunchKernelGGL(sums_run_kernel, dim3((uint32_t)runs), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_scatter(const FragDev* frags, const uint32_t* tile_first, const uint32_t* tile_last,
                          const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                          unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0,
                          hipEvent_t t1)
{
    Args a{frags, tile_first, tile_last, g, t_lo, t_hi, const_cast<uint8_t*>(src), src_origin, partials, nullptr};
    return launch_tiles<SCATTER>(a, grid_cap, s, t0, t1);
}

hipError_t launch_checksum(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const uint8_t* src, uint64_t src_origin,
                           unsigned long long* partials, uint32_t grid_cap, hipStream_t s, hipEvent_t t0,
                           hipEvent_t t1)
{
    Args a{nullptr, nullptr, nullptr, g, t_lo, t_hi, const_cast<uint8_t*>(src), src_origin, partials, nullptr};
    return launch_tiles<VERIFY>(a, grid_cap, s, t0, t1);
}

hipError_t launch_chunk_reduce(const Geometry& g, uint64_t t_lo, uint64_t t_hi, const unsigned long long* partials,
                               unsigned long long* sums_out, const unsigned long long* expected, uint8_t* bad,
                               hipStream_t s, int64_t* release)
{
    if (t_hi <= t_lo) return hipSuccess;
    ReduceArgs r;
    r.partials = partials;
    r.c_lo = t_lo / g.tiles_per_chunk;
    r.c_hi = (t_hi + g.tiles_per_chunk - 1) / g.tiles_per_chunk;
    r.n_tiles = g.n_tiles;
    r.tiles_per_chunk = g.tiles_per_chunk;
    r.sums_out = sums_out;
    r.expected = expected;
    r.bad = bad;
    r.release = release;
    hipLaunchKernelGGL(chunk_reduce_kernel, dim3((uint32_t)(r.c_hi - r.c_lo)), dim3(kReduceBlock), 0, s, r);
    return hipGetLastError();
}

} // namespace ckpt
