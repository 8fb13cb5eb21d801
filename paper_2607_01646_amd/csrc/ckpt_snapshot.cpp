// ckpt_snapshot.cpp -- issuing one snapshot (paper Sec. V-B, D2H phase;
// Sec. VI-A, ping-pong buffers and the wait before the optimizer step): the
// kernels on the pack stream, the DMA requests on the engines, the staging
// counters and the chunk-sum copy, for full or ring staging (issue_groups)
// and for direct D2H (issue_groups_direct).  The pipeline is drawn at the top
// of ckpt_runtime.cpp.
#include "ckpt_host.h"

namespace ckpt {

// The snapshot's chunk-sum copy (after the reduce has released dep_sums),
// and in image-file mode its commit record, behind the group copies.
ckpt_status issue_sums_copy(ckpt_ctx* c, SnapRec& r)
{
    RecRes* res = r.res;
    if (r.bounce) { // behind the snapshot's group copies
        {
            std::lock_guard<std::mutex> l(c->pump->m);
            PumpItem sums;
            sums.res = res;
            sums.sums = true;
            sums.image = (uint8_t*)c->h_sums[r.buf];
            sums.staging = (const uint8_t*)res->d_sums;
            sums.n = c->n_chunks * 8;
            sums.engine = c->d2h_engine[0];
            sums.buf = r.buf;
            sums.need_rec = c->pump->rec_pushed[r.buf];
            c->pump->issue_q.push_back(sums);
            if (c->file_map) { // then the commit record, once all of it has landed
                ++c->pump->rec_pushed[r.buf];
                PumpItem rec;
                rec.res = res;
                rec.groups = r.groups_copied;
                rec.buf = r.buf;
                rec.record = true;
                rec.snap_id = r.id;
                rec.step = r.step;
                rec.meta = std::make_shared<const std::vector<uint8_t>>(r.meta);
                c->pump->issue_q.push_back(std::move(rec));
            }
        }
        c->pump->cv.notify_all();
        return CKPT_OK;
    }
    ckpt_status st = dma(c, c->h_sums[r.buf], c->img_agent[r.buf], res->d_sums, c->gpu_agent, c->n_chunks * 8,
                         &res->dep_sums, res->done, c->d2h_engine[0]);
    if (st) hsa_signal_store_screlease(res->done, 0);
    return st;
}

uint64_t issue_pieces(ckpt_ctx* c, RecRes* res, uint64_t g, uint8_t* dst, hsa_agent_t dst_agent,
                      const hsa_signal_t* first_dep, hsa_amd_sdma_engine_id_t engine)
{
    const uint64_t lo = group_lo(c, g);
    for (uint64_t k = c->gap_first[g]; k < c->gap_first[g + 1]; ++k)
        std::memset(dst + (c->gaps[k].off - lo), 0, c->gaps[k].n);
    const uint64_t p0 = c->piece_first[g], p1 = c->piece_first[g + 1];
    const hsa_signal_t* dep = first_dep;
    for (uint64_t k = p0; k < p1; ++k) {
        const Piece& pc = c->pieces[k];
        const hsa_signal_t* done = k + 1 == p1 ? &res->copied[g] : &res->piece_done[k];
        hsa_signal_store_screlease(*done, 1);
        if (hsa_amd_memory_async_copy_on_engine(dst + (pc.off - lo), dst_agent, (const void*)(uintptr_t)pc.src,
                                                c->gpu_agent, pc.n, dep ? 1 : 0, dep, *done, engine,
                                                true) != HSA_STATUS_SUCCESS) {
            hsa_signal_store_screlease(*done, 0);
            return k - p0;
        }
        dep = done;
    }
    return p1 - p0;
}

// Direct D2H (no snapshot staging): per group, the sums kernel reads the
// fragments, and the group's pieces go from the tensors to host memory on a
// DMA engine once the next launch on the pack stream has released the
// group (its sums have been read; the trigger has long passed).  The copies
// finishing bump the group's counter, on which the gate waits.
ckpt_status issue_groups_direct(ckpt_ctx* c, SnapRec& r, hipStream_t after, uint64_t n_copy, int32_t stop,
                                hsa_signal_t& carried)
{
    RecRes* res = r.res;
    uint8_t* himg = c->h_img[r.buf];
    hsa_agent_t host = c->img_agent[r.buf];
    HIPCHK(c, hipEventRecord(c->ev_trigger, after));
    HIPCHK(c, hipStreamWaitEvent(c->s_pack, c->ev_trigger, 0));
    if (r.timed) HIPCHK(c, hipEventRecord(res->t0, c->s_pack));
    int64_t* pending = nullptr; // the previous group's release, carried by the next launch
    for (uint64_t g = 0; g < c->n_groups; ++g) {
        const uint64_t lo = group_lo(c, g);
        hipError_t e = launch_sums(c->d_frags, c->d_tile_first, c->d_tile_last, c->geo, tiles_lo(c, g),
                                   tiles_hi(c, g), c->d_partials, c->grid_cap, c->s_pack,
                                   r.timed && (r.per_launch || g == 0) ? res->k0[g] : nullptr,
                                   r.timed && (r.per_launch || g == 0) ? res->k1[g] : nullptr, pending);
        if (e != hipSuccess) return fail(c, CKPT_EHIP, "sums launch failed: %s", hipGetErrorString(e));
        pending = nullptr;
        carried.handle = 0;
        if (g >= n_copy) { // interrupted offload: this group never leaves the device, the gate waits for its sums
            HIPCHK(c, hipEventRecord(res->captured[g], c->s_pack));
            continue;
        }
        // A copied group needs no event: its copies wait for the release that
        // the next launch stores once this one has finished, so the counter
        // the gate waits for implies the group's sums have been read too.
        hsa_signal_store_screlease(res->dep[g], 1);
        pending = res->dep_val[g];
        carried = res->dep[g];
        hsa_signal_store_screlease(res->copied[g], 1);
        hsa_signal_store_screlease(res->flagged[g], 1);
        r.groups_copied = (uint32_t)(g + 1);
        const hsa_amd_sdma_engine_id_t eng = c->d2h_engine[g % c->n_d2h_engines];
        res->h_seq[g] = c->area_seq[g] + 1;
        ++c->area_seq[g];
        if (r.bounce) { // the pump issues the pieces once a ring slot is free
            {
                std::lock_guard<std::mutex> l(c->pump->m);
                PumpItem it;
                it.res = res;
                it.g = (uint32_t)g;
                it.image = himg + lo;
                it.lo = lo;
                it.n = group_hi(c, g) - lo;
                it.area_done = c->d_area_done + g;
                it.seq = &res->h_seq[g];
                it.engine = eng;
                it.buf = r.buf;
                c->pump->issue_q.push_back(it);
            }
            c->pump->cv.notify_all();
            continue;
        }
        const uint64_t want = c->piece_first[g + 1] - c->piece_first[g];
        const uint64_t got = issue_pieces(c, res, g, himg + lo, host, &res->dep[g], eng);
        ckpt_status st = CKPT_OK;
        if (got == want)
            st = dma(c, c->d_area_done + g, c->gpu_agent, &res->h_seq[g], host, 8, &res->copied[g], res->flagged[g],
                     c->h2d_engine);
        if (got != want || st) {
            // Let the issued pieces run (nothing else will release them),
            // wait until they have read the tensors, then count the group
            // as copied so that no gate waits forever; the snapshot is
            // marked interrupted and never restored.
            hsa_signal_store_screlease(res->dep[g], 0);
            carried.handle = 0;
            if (got && got < want) (void)poll_zero(res->piece_done[c->piece_first[g] + got - 1], 120);
            if (got == want) (void)poll_zero(res->copied[g], 120);
            (void)hsa_memory_copy(c->d_area_done + g, &res->h_seq[g], 8);
            hsa_signal_store_screlease(res->copied[g], 0);
            hsa_signal_store_screlease(res->flagged[g], 0);
            return st ? st : fail(c, CKPT_EHIP, "DMA of a fragment piece of group %llu could not be issued",
                                  (unsigned long long)g);
        }
    }
    if (stop >= 0) {
        r.aborted = true; // interrupted offload: never committed
        if (pending) {
            hipError_t e = launch_release(pending, c->s_pack);
            if (e != hipSuccess) return fail(c, CKPT_EHIP, "release launch failed: %s", hipGetErrorString(e));
            carried.handle = 0;
        }
        return CKPT_OK;
    }
    hipError_t e = launch_chunk_reduce(c->geo, 0, c->geo.n_tiles, c->d_partials, res->d_sums, nullptr, nullptr,
                                       c->s_pack, pending);
    if (e != hipSuccess) return fail(c, CKPT_EHIP, "reduce launch failed: %s", hipGetErrorString(e));
    carried.handle = 0;
    hsa_signal_store_screlease(res->dep_sums, 1);
    e = launch_release(res->dep_sums_val, c->s_pack);
    if (e != hipSuccess) return fail(c, CKPT_EHIP, "release launch failed: %s", hipGetErrorString(e));
    if (r.timed) HIPCHK(c, hipEventRecord(res->t_red, c->s_pack));
    hsa_signal_store_screlease(res->done, 1);
    return issue_sums_copy(c, r);
}

// The body of issue_snapshot.  `carried` is the signal of a group whose DMA
// has been issued while the launch that will release it has not yet been
// enqueued; on an error return the caller releases it from the host.
ckpt_status issue_groups(ckpt_ctx* c, SnapRec& r, hipStream_t after, uint64_t n_copy, int32_t stop,
                         hsa_signal_t& carried)
{
    RecRes* res = r.res;
    uint8_t* himg = c->h_img[r.buf];
    hsa_agent_t host = c->img_agent[r.buf];
    ckpt_status st = CKPT_OK;
    HIPCHK(c, hipEventRecord(c->ev_trigger, after));
    HIPCHK(c, hipStreamWaitEvent(c->s_pack, c->ev_trigger, 0));
    if (r.timed) HIPCHK(c, hipEventRecord(res->t0, c->s_pack));
    // Each launch packs LG groups; each copied group's DMA waits for the
    // signal of its launch's first group to drop to 0.  With a full-size
    // image the next launch on the pack stream (the next pack, or the
    // chunk-sum reduce after the last) sets it, which happens only after this
    // launch's pack has finished; in ring mode the next pack may first wait
    // for a slot, so a one-lane kernel releases the group right after its
    // pack instead.
    const bool carry = !c->ring;
    int64_t* pending = nullptr; // the previous launch's release, carried by the next launch
    for (uint64_t g = 0; g < c->n_groups; ++g) {
        const uint64_t lo = group_lo(c, g), hi = group_hi(c, g);
        const uint64_t area = area_of(c, g);
        const uint64_t j = g / c->LG;      // this group's launch
        const uint64_t g0 = j * c->LG;     // its first group
        const uint64_t g1 = std::min(g0 + c->LG, c->n_groups);
        if (g == g0) {
            // A staging area is free once every copy issued out of it so far
            // has finished (each finished copy bumps area_done by one); the
            // launch writes the areas of all its groups.  The pack stream
            // waits for that only while the host still sees the area's latest
            // copy running: each wait is a packet the command processor works
            // through between two packs, and with a full-size image the
            // previous snapshot has committed, so its copies are all done.
            for (uint64_t h = g0; h < g1; ++h) {
                const uint64_t a = area_of(c, h);
                if (c->area_seq[a] && hsa_signal_load_scacquire(c->area_flag[a]) != 0)
                    HIPCHK(c, hipStreamWaitValue64(c->s_pack, c->d_area_done + a, c->area_seq[a],
                                                  hipStreamWaitValueGte, ~0ull));
            }
            if (c->poison) { // debug check: the canary, then the pack over it (stream order)
                uint32_t w[4];
                std::memcpy(w, CKPT_CANARY, 16);
                hipError_t e = launch_fill16(staging_of(c, g0), group_hi(c, g1 - 1) - lo, w, c->s_pack);
                if (e != hipSuccess) return fail(c, CKPT_EHIP, "canary fill failed: %s", hipGetErrorString(e));
            }
            hipError_t e = launch_pack(c->d_frags, c->d_tile_first, c->d_tile_last, c->geo, tiles_lo(c, g0),
                                       tiles_hi(c, g1 - 1), staging_of(c, g0), lo, c->d_partials, c->grid_cap,
                                       c->s_pack, r.timed && (r.per_launch || j == 0) ? res->k0[j] : nullptr,
                                       r.timed && (r.per_launch || j == 0) ? res->k1[j] : nullptr,
                                       pending);
            if (e != hipSuccess) return fail(c, CKPT_EHIP, "pack launch failed: %s", hipGetErrorString(e));
            pending = nullptr; // enqueued: the GPU releases it
            carried.handle = 0;
            // The gate and the launch's copies need the packed bytes only; the
            // chunk sums are added up once, after the last launch (below).
            HIPCHK(c, hipEventRecord(res->captured[g1 - 1], c->s_pack));
            if (g0 < n_copy) {
                hsa_signal_store_screlease(res->dep[g0], 1); // before any copy is issued or a launch clears it
                if (carry) {
                    pending = res->dep_val[g0];
                    carried = res->dep[g0];
                } else {
                    e = launch_release(res->dep_val[g0], c->s_pack);
                    if (e != hipSuccess) return fail(c, CKPT_EHIP, "release launch failed: %s", hipGetErrorString(e));
                }
            }
        }
        if (g >= n_copy) continue; // interrupted offload: this group never leaves the device
        hsa_signal_store_screlease(res->copied[g], 1);
        hsa_signal_store_screlease(res->flagged[g], 1);
        r.groups_copied = (uint32_t)(g + 1);
        const hsa_amd_sdma_engine_id_t eng = c->d2h_engine[g % c->n_d2h_engines];
        res->h_seq[g] = c->area_seq[area] + 1;
        if (r.bounce) { // the pump issues the copies once a ring slot is free
            {
                std::lock_guard<std::mutex> l(c->pump->m);
                PumpItem it;
                it.res = res;
                it.g = (uint32_t)g;
                it.image = himg + lo;
                it.staging = staging_of(c, g);
                it.n = hi - lo;
                it.area_done = c->d_area_done + area;
                it.seq = &res->h_seq[g];
                it.engine = eng;
                it.buf = r.buf;
                c->pump->issue_q.push_back(it);
            }
            c->pump->cv.notify_all();
            ++c->area_seq[area];
            c->area_flag[area] = res->flagged[g];
            continue;
        }
        st = dma(c, himg + lo, host, staging_of(c, g), c->gpu_agent, hi - lo, &res->dep[g0], res->copied[g], eng);
        if (!st)
            st = dma(c, c->d_area_done + area, c->gpu_agent, &res->h_seq[g], host, 8, &res->copied[g],
                     res->flagged[g], c->h2d_engine);
        if (st) {
            // nothing will lower the signals of this group
            hsa_signal_store_screlease(res->copied[g], 0);
            hsa_signal_store_screlease(res->flagged[g], 0);
            return st;
        }
        ++c->area_seq[area];
        c->area_flag[area] = res->flagged[g];
    }
    if (stop >= 0) {
        r.aborted = true; // interrupted offload: never committed (its pack timing stays readable)
        if (pending) {    // the last copied group was the last group
            hipError_t e = launch_release(pending, c->s_pack);
            if (e != hipSuccess) return fail(c, CKPT_EHIP, "release launch failed: %s", hipGetErrorString(e));
            carried.handle = 0;
        }
    } else {
        // Every chunk's sum from its tiles' partial sums, in one launch: only
        // the sums copy below needs them, and one launch per group would cost
        // the caller host time per group.  It also releases the last group.
        hipError_t e = launch_chunk_reduce(c->geo, 0, c->geo.n_tiles, c->d_partials, res->d_sums, nullptr, nullptr,
                                           c->s_pack, pending);
        if (e != hipSuccess) return fail(c, CKPT_EHIP, "reduce launch failed: %s", hipGetErrorString(e));
        carried.handle = 0;
        hsa_signal_store_screlease(res->dep_sums, 1);
        e = launch_release(res->dep_sums_val, c->s_pack);
        if (e != hipSuccess) return fail(c, CKPT_EHIP, "release launch failed: %s", hipGetErrorString(e));
        if (r.timed) HIPCHK(c, hipEventRecord(res->t_red, c->s_pack));
        hsa_signal_store_screlease(res->done, 1);
        return issue_sums_copy(c, r);
    }
    return CKPT_OK;
}

ckpt_status issue_snapshot(ckpt_ctx* c, SnapRec& r, hipStream_t after, uint64_t n_copy, int32_t stop)
{
    hsa_signal_t carried{0};
    const ckpt_status st = c->direct ? issue_groups_direct(c, r, after, n_copy, stop, carried)
                                     : issue_groups(c, r, after, n_copy, stop, carried);
    // A DMA whose release never got enqueued would wait forever: let it run
    // (the snapshot is marked interrupted and is never restored).
    if (st && carried.handle) hsa_signal_store_screlease(carried, 0);
    return st;
}

} // namespace ckpt
