// ckpt_noalloc.cpp -- ckpt_pack_noalloc: the pack and chunk sums of a
// snapshot (the packing half of the D2H phase, paper Sec. V-B) into a device
// image the caller owns, for callers that cannot allocate.  No context, no
// allocation of any kind: the fragment table, the tile table and the partial
// sums live in the kernel file's fixed scratch array; the layout is computed
// in two passes over the descriptors; descriptors reach the device as kernel
// arguments.  Everything is enqueued on the caller's stream.
#include <cstdarg>
#include <cstdio>

#include "ckpt_host.h"

namespace ckpt {
namespace {

thread_local char t_err[384];

ckpt_status fail_free(ckpt_status code, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(t_err, sizeof t_err, fmt, ap);
    va_end(ap);
    return code;
}

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

// [p, p + n) must be memory of `device` inside one allocation: the kernels
// read or write every byte of it.  `what` names it in the error text.
ckpt_status check_range(const void* p, uint64_t n, int device, const char* what)
{
    hipPointerAttribute_t pa;
    std::memset(&pa, 0, sizeof pa);
    if (hipPointerGetAttributes(&pa, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail_free(CKPT_EINVAL, "%s: %p is not memory the GPU runtime knows", what, p);
    }
    if (pa.type != hipMemoryTypeDevice && !pa.isManaged)
        return fail_free(CKPT_EINVAL, "%s: %p is not device memory", what, p);
    if (pa.type == hipMemoryTypeDevice && pa.device != device)
        return fail_free(CKPT_EINVAL, "%s: memory of device %d, not of device %d", what, pa.device, device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) == hipSuccess) {
        const uint64_t lo = (uint64_t)(uintptr_t)p, b = (uint64_t)(uintptr_t)base;
        if (lo < b || n > size || lo - b > size - n)
            return fail_free(CKPT_EINVAL, "%s: %llu bytes at %p run past the end of its allocation", what,
                             (unsigned long long)n, p);
    } else {
        (void)hipGetLastError();
    }
    return CKPT_OK;
}

// Restores the caller's current device on every return path.
struct DeviceGuard {
    int prev = -1;
    bool set = false;
    ~DeviceGuard()
    {
        if (set) (void)hipSetDevice(prev);
    }
};

} // namespace

const char* noalloc_error() { return t_err; }

} // namespace ckpt

using namespace ckpt;

extern "C" ckpt_status ckpt_pack_noalloc(const ckpt_tensor* t, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                                         int32_t device, void* image, uint64_t image_cap, uint64_t* sums,
                                         uint64_t sums_cap, void* stream, uint64_t* image_bytes, uint64_t* n_chunks)
{
    t_err[0] = 0;
    if (!t || !image || !sums) return fail_free(CKPT_EINVAL, "null argument");
    if (n == 0) return fail_free(CKPT_EINVAL, "need at least one fragment");
    if (n > kNoallocMaxFrags)
        return fail_free(CKPT_EINVAL, "%u fragments: the allocation-free pack takes at most %u", n, kNoallocMaxFrags);
    const uint64_t C = chunk_bytes ? chunk_bytes : kDefaultChunk;
    const uint32_t A = align_bytes ? align_bytes : kDefaultAlign;
    if (!geometry_ok(C, A)) return fail_free(CKPT_EINVAL, "bad geometry: chunk %llu, alignment %u", (unsigned long long)C, A);
    const uint32_t ts = tile_shift_for(C);
    const uint64_t tpc = C >> ts; // tiles per chunk
    if (tpc > kNoallocGroupTiles)
        return fail_free(CKPT_EINVAL, "a chunk of %llu tiles exceeds the scratch's %llu tiles (chunks up to 1 GiB)",
                         (unsigned long long)tpc, (unsigned long long)kNoallocGroupTiles);
    if (((uintptr_t)image & 15) || ((uintptr_t)sums & 7))
        return fail_free(CKPT_EINVAL, "image must be 16-byte aligned and sums 8-byte aligned");

    // Layout (registration order, each fragment at the previous end rounded
    // up to the alignment, the image ending on it too): first the size.
    uint64_t end = 0;
    for (uint32_t i = 0; i < n; ++i) {
        if (t[i].nbytes && !t[i].dev_ptr) return fail_free(CKPT_EINVAL, "fragment %u: null pointer", i);
        end = align_up(end, A) + t[i].nbytes;
    }
    const uint64_t I = align_up(end, A);
    if (I == 0) return fail_free(CKPT_EINVAL, "all fragments are empty");
    const uint64_t nc = (I + C - 1) / C;
    if (image_bytes) *image_bytes = I;
    if (n_chunks) *n_chunks = nc;
    if (image_cap < I)
        return fail_free(CKPT_EINVAL, "image of %llu bytes needs %llu", (unsigned long long)image_cap,
                         (unsigned long long)I);
    if (sums_cap < nc)
        return fail_free(CKPT_EINVAL, "%llu sums for %llu chunks", (unsigned long long)sums_cap, (unsigned long long)nc);

    DeviceGuard dg;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || device < 0 || device >= ndev)
        return fail_free(CKPT_EINVAL, "no device %d", device);
    if (hipGetDevice(&dg.prev) != hipSuccess) return fail_free(CKPT_EHIP, "hipGetDevice failed");
    if (dg.prev != device) {
        if (hipSetDevice(device) != hipSuccess) return fail_free(CKPT_EHIP, "hipSetDevice(%d) failed", device);
        dg.set = true;
    }
    for (uint32_t i = 0; i < n; ++i) {
        if (!t[i].nbytes) continue;
        char what[32];
        snprintf(what, sizeof what, "fragment %u", i);
        ckpt_status st = check_range(t[i].dev_ptr, t[i].nbytes, device, what);
        if (st) return st;
    }
    ckpt_status st = check_range(image, I, device, "image");
    if (!st) st = check_range(sums, nc * 8, device, "sums");
    if (st) return st;

    uint8_t* base = nullptr;
    hipError_t e = noalloc_scratch(&base);
    if (e != hipSuccess) return fail_free(CKPT_EHIP, "scratch address: %s", hipGetErrorString(e));
    FragDev* d_frags = reinterpret_cast<FragDev*>(base + kNoallocFragsOff);
    uint32_t* d_first = reinterpret_cast<uint32_t*>(base + kNoallocFirstOff);
    uint32_t* d_last = reinterpret_cast<uint32_t*>(base + kNoallocLastOff);
    unsigned long long* d_part = reinterpret_cast<unsigned long long*>(base + kNoallocPartialsOff);
    hipStream_t s = (hipStream_t)stream;

    // Second pass: the fragment table, in batches carried by kernel arguments.
    FragDev batch[kUploadBatch];
    uint32_t k = 0;
    uint64_t off = 0;
    for (uint32_t i = 0; i < n; ++i) {
        const uint64_t next = align_up(off + t[i].nbytes, A); // the next fragment's offset
        FragDev& f = batch[k++];
        f.ptr = (uint64_t)(uintptr_t)t[i].dev_ptr;
        f.nbytes = t[i].nbytes;
        f.off = off;
        f.end = (i + 1 < n) ? next : I;
        off = next;
        if (k == kUploadBatch || i + 1 == n) {
            e = launch_frag_upload(d_frags + (i + 1 - k), batch, k, s);
            if (e != hipSuccess) return fail_free(CKPT_EHIP, "table upload: %s", hipGetErrorString(e));
            k = 0;
        }
    }

    Geometry g;
    g.image_bytes = I;
    g.tile_shift = ts;
    g.n_tiles = (I + (1ull << ts) - 1) >> ts;
    g.n_chunks = nc;
    g.tiles_per_chunk = (uint32_t)tpc;
    // Groups of whole chunks, at most kNoallocGroupTiles tiles each, one after
    // another on the stream: each reuses the tile table and partial sums.
    const uint64_t G = std::max<uint64_t>(1, kNoallocGroupTiles / tpc);
    for (uint64_t lo = 0; lo < I; lo += G * C) {
        const uint64_t hi = std::min(lo + G * C, I);
        const uint64_t t_lo = lo >> ts, t_hi = (hi + (1ull << ts) - 1) >> ts;
        e = launch_tile_table(d_frags, n, g, t_lo, t_hi, d_first, d_last, s);
        if (e != hipSuccess) return fail_free(CKPT_EHIP, "tile table: %s", hipGetErrorString(e));
        // The kernels index the tables and partial sums by absolute tile;
        // the group's entries sit at the start of the scratch, so the bases
        // passed are moved back by t_lo entries (only [t_lo, t_hi) is read
        // or written through them).
        const uint32_t* first = reinterpret_cast<const uint32_t*>((uintptr_t)d_first - t_lo * 4);
        const uint32_t* last = reinterpret_cast<const uint32_t*>((uintptr_t)d_last - t_lo * 4);
        unsigned long long* part =
            reinterpret_cast<unsigned long long*>((uintptr_t)d_part - t_lo * kTileParts * 8);
        e = launch_pack(d_frags, first, last, g, t_lo, t_hi, (uint8_t*)image, 0, part, kDefaultGrid, s);
        if (e != hipSuccess) return fail_free(CKPT_EHIP, "pack launch: %s", hipGetErrorString(e));
        e = launch_chunk_reduce(g, t_lo, t_hi, part, (unsigned long long*)sums, nullptr, nullptr, s);
        if (e != hipSuccess) return fail_free(CKPT_EHIP, "reduce launch: %s", hipGetErrorString(e));
    }
    return CKPT_OK;
}
