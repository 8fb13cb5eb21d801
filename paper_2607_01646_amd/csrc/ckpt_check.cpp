// ckpt_check.cpp -- restore and verify of a committed host image (paper
// Sec. V-C third stage, Sec. VI-E): each span of image bytes goes host ->
// device staging on a copy stream, then the scatter or checksum kernel and
// the chunk-sum compare run on the kernel stream, span by span, so that the
// copies and the checks overlap.
#include "ckpt_host.h"

namespace ckpt {

// Where restore and verify stage image bytes on the device, and the streams
// and events that order them.  Unit u covers chunks [u*G, (u+1)*G).
struct Lane {
    hipStream_t s_copy, s_ker;
    uint8_t* base;   // staging: full image, or ring slots of G chunks each
    bool ring;
    uint64_t n_slots;
    uint64_t G;
    uint64_t n_units;
    std::vector<hipEvent_t>* area_free; // per slot (ring) or per unit
    std::vector<hipEvent_t>* loaded;    // per unit
    std::vector<hipEvent_t>* tk0;       // per unit, timing
    std::vector<hipEvent_t>* tk1;
    hipEvent_t done, t0, c0, c1;
};

Lane restore_lane(ckpt_ctx* c)
{
    return Lane{c->s_copy, c->s_pack, c->d_staging, c->ring || c->direct, c->n_slots, c->G, c->n_groups, &c->area_free,
                &c->ev_loaded, &c->tk0, &c->tk1, c->ev_done, c->tt0, c->tc0, c->tc1};
}

Lane verify_lane(ckpt_ctx* c)
{
    return Lane{c->s_vcopy, c->s_vker, c->d_vring, true, c->n_vslots, c->G, c->n_groups, &c->vfree,
                &c->vloaded, &c->vk0, &c->vk1, c->ev_vdone, c->vt0, c->vc0, c->vc1};
}

// Restore (scatter=true) or verify (scatter=false) the chunks of host image
// b against the sums in h_sums[b]: every chunk, or only the chunks `ids`
// (increasing) when given.  The caller has checked the arguments and, for a
// restore, drained every snapshot.
ckpt_status check_image(ckpt_ctx* c, int b, hipStream_t stream, bool scatter, const std::vector<uint64_t>* ids,
                        uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad,
                        const std::function<bool(uint64_t, uint64_t)>& fill)
{
    const Lane L = scatter ? restore_lane(c) : verify_lane(c);
    const int op = scatter ? CKPT_OP_RESTORE : CKPT_OP_VERIFY;
    const uint64_t unit = L.G * c->C;
    // Byte spans to move, each within one unit's size: whole units, or the
    // runs of consecutive chunk ids cut at that size.
    std::vector<std::pair<uint64_t, uint64_t>> spans;
    if (!ids) {
        for (uint64_t u = 0; u < L.n_units; ++u) spans.emplace_back(u * unit, std::min((u + 1) * unit, c->I));
    } else {
        for (size_t j = 0; j < ids->size();) {
            size_t k = j + 1;
            while (k < ids->size() && (*ids)[k] == (*ids)[k - 1] + 1 && k - j < L.G) ++k;
            spans.emplace_back((*ids)[j] * c->C, std::min(((*ids)[k - 1] + 1) * c->C, c->I));
            j = k;
        }
    }
    const uint64_t n_spans = spans.size();
    // Per-span events are reused round-robin past the unit count; timing is
    // kept for whole-image operations only.
    const bool timed = c->timing && !ids;
    unsigned long long* partials = c->d_partials + c->geo.n_tiles * kTileParts;
    HIPCHK(c, hipMemcpyAsync(c->d_expected, c->h_sums[b], c->n_chunks * 8, hipMemcpyHostToDevice, L.s_copy));
    if (scatter) {
        HIPCHK(c, hipEventRecord(c->ev_trigger, stream));
        HIPCHK(c, hipStreamWaitEvent(L.s_ker, c->ev_trigger, 0));
    }
    if (timed) HIPCHK(c, hipEventRecord(L.t0, L.s_copy));
    for (uint64_t u = 0; u < n_spans; ++u) {
        const uint64_t lo = spans[u].first, hi = spans[u].second;
        const uint64_t ev = u % L.n_units;
        const uint64_t area = L.ring ? u % L.n_slots : ev;
        uint8_t* stage = L.ring ? L.base + area * unit : L.base + lo;
        // A device slot is reused once the kernel of the span that last used
        // it has finished.  With pageable images the host paces every span
        // (it fills the pinned slot first), so it waits for that kernel itself
        // right before the copy: the same wait as a device-side one on the
        // copy stream, which here cost ~6% of the link (verify 53.5 against
        // 56.8 GB/s through the bounce rings).
        const bool host_wait = c->bounce && L.ring;
        if (!host_wait) HIPCHK(c, hipStreamWaitEvent(L.s_copy, (*L.area_free)[area], 0));
        if (timed && u == 0) HIPCHK(c, hipEventRecord(L.c0, L.s_copy));
        if (fill && !fill(lo, hi)) { // the span's bytes did not arrive: let the issued work finish, then fail
            (void)hipStreamSynchronize(L.s_copy);
            (void)hipStreamSynchronize(L.s_ker);
            return CKPT_EHIP;
        }
        const uint8_t* src = c->h_img[b] + lo;
        if (c->bounce) { // pageable image: through a pinned ring slot
            const uint64_t slot = u % c->n_bslots;
            if (u >= c->n_bslots) HIPCHK(c, hipEventSynchronize(c->bin_done[slot]));
            c->pool->copy(c->h_bin + slot * unit, src, hi - lo);
            src = c->h_bin + slot * unit;
        }
        if (host_wait) HIPCHK(c, hipEventSynchronize((*L.area_free)[area]));
        HIPCHK(c, hipMemcpyAsync(stage, src, hi - lo, hipMemcpyHostToDevice, L.s_copy));
        if (c->bounce) HIPCHK(c, hipEventRecord(c->bin_done[u % c->n_bslots], L.s_copy));
        if (timed && u + 1 == n_spans) HIPCHK(c, hipEventRecord(L.c1, L.s_copy));
        HIPCHK(c, hipEventRecord((*L.loaded)[ev], L.s_copy));
        HIPCHK(c, hipStreamWaitEvent(L.s_ker, (*L.loaded)[ev], 0));
        const uint64_t t_lo = lo >> c->geo.tile_shift, t_hi = (hi + (1ull << c->geo.tile_shift) - 1) >> c->geo.tile_shift;
        hipEvent_t k0 = timed ? (*L.tk0)[u] : nullptr, k1 = timed ? (*L.tk1)[u] : nullptr;
        hipError_t e;
        if (scatter)
            e = launch_scatter(c->d_frags, c->d_tile_first, c->d_tile_last, c->geo, t_lo, t_hi, stage, lo, partials,
                               c->grid_cap, L.s_ker, k0, k1);
        else
            e = launch_checksum(c->geo, t_lo, t_hi, stage, lo, partials, c->grid_cap, L.s_ker, k0, k1);
        if (e != hipSuccess) return fail(c, CKPT_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
        e = launch_chunk_reduce(c->geo, t_lo, t_hi, partials, c->d_recomputed, c->d_expected, c->d_bad, L.s_ker);
        if (e != hipSuccess) return fail(c, CKPT_EHIP, "kernel launch failed: %s", hipGetErrorString(e));
        HIPCHK(c, hipEventRecord((*L.area_free)[area], L.s_ker));
    }
    HIPCHK(c, hipMemcpyAsync(c->h_bad, c->d_bad, c->n_chunks, hipMemcpyDeviceToHost, L.s_ker));
    HIPCHK(c, hipMemcpyAsync(c->h_recomputed, c->d_recomputed, c->n_chunks * 8, hipMemcpyDeviceToHost, L.s_ker));
    HIPCHK(c, hipEventRecord(L.done, L.s_ker));
    if (scatter) HIPCHK(c, hipStreamWaitEvent(stream, L.done, 0));
    HIPCHK(c, hipEventSynchronize(L.done));
    if (timed) {
        ckpt_timing t{};
        for (uint64_t u = 0; u < L.n_units; ++u) t.kernel_ms += elapsed((*L.tk0)[u], (*L.tk1)[u]);
        t.kernels = (uint32_t)L.n_units;
        t.copies = (uint32_t)L.n_units;
        t.copy_ms = elapsed(L.c0, L.c1);
        t.total_ms = elapsed(L.t0, (*L.tk1)[L.n_units - 1]);
        t.kernel_bytes = scatter ? 2 * c->payload : c->I;
        t.copy_bytes = c->I;
        t.span_ms = -1.f;
        c->op_timing[op].t = t;
        c->op_timing[op].valid = true;
    }
    uint32_t nb = 0;
    auto flag = [&](uint64_t k) {
        if (!c->h_bad[k]) return;
        if (nb < cap) bad_chunks[nb] = (uint32_t)k;
        ++nb;
    };
    if (ids) {
        for (uint64_t k : *ids) flag(k);
    } else {
        c->last_sums.assign(c->h_recomputed, c->h_recomputed + c->n_chunks);
        c->have_last_sums = true;
        for (uint64_t k = 0; k < c->n_chunks; ++k) flag(k);
    }
    *n_bad = nb;
    if (nb)
        return fail(c, CKPT_ECORRUPT, "%u of %llu chunks failed their checksum", nb,
                    (unsigned long long)(ids ? ids->size() : c->n_chunks));
    return CKPT_OK;
}

} // namespace ckpt
