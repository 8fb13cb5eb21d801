// ckpt_bounce.cpp -- pageable host images behind pinned bounce rings: the
// per-context pump that moves each snapshot's chunk groups device -> ring
// (DMA engines) -> image (host copy threads), in snapshot and group order.
// See Pump in ckpt_host.h.
#include "ckpt_host.h"

namespace ckpt {

// Poll a signal that only the GPU side waits on until it reads 0.
bool poll_zero(hsa_signal_t sig, int seconds)
{
    const auto deadline = std::chrono::steady_clock::now() + std::chrono::seconds(seconds);
    while (hsa_signal_load_scacquire(sig) != 0) {
        if (std::chrono::steady_clock::now() > deadline) return false;
        std::this_thread::sleep_for(std::chrono::microseconds(20));
    }
    return true;
}

// Bounce mode, issuer thread (see Pump).
void pump_issue(ckpt_ctx* c)
{
    Pump* p = c->pump;
    const uint64_t unit = c->G * c->C;
    for (;;) {
        PumpItem it;
        uint64_t slot = UINT64_MAX; // taken ring slot, if any
        {
            std::unique_lock<std::mutex> l(p->m);
            p->cv.wait(l, [&] { return p->stop || !p->issue_q.empty(); });
            if (p->issue_q.empty()) return;
            it = p->issue_q.front();
            p->issue_q.pop_front();
            if (it.record) { // no copy: handled by the drainer in order
                p->drain_q.emplace_back(it, UINT64_MAX);
                p->cv.notify_all();
                continue;
            }
            if (it.sums) {
                // no ring slot: straight into the pinned sums array, once the
                // drainer has written every earlier record that reads it
                p->cv.wait(l, [&] { return p->stop || p->failed || p->rec_done[it.buf] >= it.need_rec; });
                bool ok = !p->failed && !p->stop;
                l.unlock();
                if (ok)
                    ok = hsa_amd_memory_async_copy_on_engine(it.image, c->img_agent[0], it.staging, c->gpu_agent,
                                                             it.n, 1, &it.res->dep_sums, it.res->done, it.engine,
                                                             true) == HSA_STATUS_SUCCESS;
                if (!ok) {
                    hsa_signal_store_screlease(it.res->done, 0);
                    it.res->failed.store(true, std::memory_order_release);
                    l.lock();
                    if (!p->failed) {
                        p->failed = true;
                        p->err = "DMA of the chunk sums could not be issued";
                    }
                }
                continue;
            }
            const uint64_t s = p->next_slot % c->n_bslots;
            p->cv.wait(l, [&] { return p->stop || p->failed || !p->busy[s]; });
            if (!p->failed) {
                if (p->busy[s]) return; // stopping
                p->busy[s] = 1;
                ++p->next_slot;
                slot = s;
            }
        }
        const char* what = nullptr;
        bool issued = false, counted = false;
        if (slot != UINT64_MAX) {
            if (c->direct) { // the group's fragment pieces, straight from the tensors into the slot
                const uint64_t want = c->piece_first[it.g + 1] - c->piece_first[it.g];
                const uint64_t got = issue_pieces(c, it.res, it.g, c->h_bout + slot * unit, c->img_agent[0],
                                                  &it.res->dep[it.g], it.engine);
                issued = got == want;
                if (!issued) {
                    // the pieces already issued must have finished before the slot is reused
                    if (got) (void)poll_zero(it.res->piece_done[c->piece_first[it.g] + got - 1], 120);
                    what = "DMA of a fragment piece to the bounce ring could not be issued";
                }
            } else {
                issued = hsa_amd_memory_async_copy_on_engine(c->h_bout + slot * unit, c->img_agent[0], it.staging,
                                                             c->gpu_agent, it.n, 1,
                                                             &it.res->dep[it.g / c->LG * c->LG],
                                                             it.res->copied[it.g], it.engine,
                                                             true) == HSA_STATUS_SUCCESS;
                if (!issued) what = "DMA of a chunk group to the bounce ring could not be issued";
            }
            if (issued)
                counted = hsa_amd_memory_async_copy_on_engine(it.area_done, c->gpu_agent, it.seq, c->img_agent[0], 8, 1,
                                                              &it.res->copied[it.g], it.res->flagged[it.g],
                                                              c->h2d_engine, true) == HSA_STATUS_SUCCESS;
            if (issued && !counted) what = "staging counter copy could not be issued";
        }
        if (!issued) hsa_signal_store_screlease(it.res->copied[it.g], 0);
        if (!counted) {
            // Nothing bumps the staging area's use counter through the
            // engines: once no copy reads the area, write it directly, so
            // that no later pack waits for it forever.
            if (!issued || poll_zero(it.res->copied[it.g], 120)) (void)hsa_memory_copy(it.area_done, it.seq, 8);
            hsa_signal_store_screlease(it.res->flagged[it.g], 0);
        }
        std::lock_guard<std::mutex> l(p->m);
        if (what && !p->failed) {
            p->failed = true;
            p->err = what;
        }
        if (!counted) it.res->failed.store(true, std::memory_order_release);
        if (slot != UINT64_MAX && !issued) {
            p->busy[slot] = 0;
            slot = UINT64_MAX;
        }
        p->drain_q.emplace_back(it, slot);
        p->cv.notify_all();
    }
}

// Bounce mode, drainer thread (see Pump).
void pump_drain(ckpt_ctx* c)
{
    Pump* p = c->pump;
    const uint64_t unit = c->G * c->C;
    for (;;) {
        std::pair<PumpItem, uint64_t> d;
        {
            std::unique_lock<std::mutex> l(p->m);
            p->cv.wait(l, [&] { return p->stop || !p->drain_q.empty(); });
            if (p->drain_q.empty()) return;
            d = p->drain_q.front();
            p->drain_q.pop_front();
        }
        const PumpItem& it = d.first;
        const uint64_t slot = d.second;
        if (it.record) { // the snapshot's commit record in the image file
            const auto deadline = std::chrono::steady_clock::now() + std::chrono::seconds(120);
            while (!res_done(it.res, it.groups, true) && std::chrono::steady_clock::now() < deadline)
                std::this_thread::sleep_for(std::chrono::microseconds(20));
            if (res_done(it.res, it.groups, true) && !it.res->failed.load(std::memory_order_acquire)) {
                file_commit(c, it);
                uint64_t ts = 0;
                (void)hsa_system_get_info(HSA_SYSTEM_INFO_TIMESTAMP, &ts);
                it.res->recorded_ts.store(ts, std::memory_order_relaxed);
                it.res->recorded.store(true, std::memory_order_release);
            }
            std::lock_guard<std::mutex> l(p->m);
            ++p->rec_done[it.buf];
            p->cv.notify_all();
            continue;
        }
        bool free_slot = slot != UINT64_MAX, ok = free_slot;
        if (ok) {
            ok = poll_zero(it.res->copied[it.g], 120);
            // The image's record (an older snapshot's) stops counting before
            // the first byte of a new one lands.
            if (ok && it.g == 0 && c->file_map) file_invalidate(c, it.buf);
            if (ok) c->pool->copy(it.image, c->h_bout + slot * unit, it.n);
            else free_slot = false; // the engine may still write it
        }
        {
            std::lock_guard<std::mutex> l(p->m);
            if (free_slot) p->busy[slot] = 0;
            if (slot != UINT64_MAX && !ok && !p->failed) {
                p->failed = true;
                p->err = "DMA of a chunk group to the bounce ring did not finish within 120 s";
            }
            p->cv.notify_all();
        }
        if (!ok) it.res->failed.store(true, std::memory_order_release);
        if (ok && it.g + 1 == c->n_groups) { // the image's last byte has landed (groups drain in order)
            uint64_t ts = 0;
            (void)hsa_system_get_info(HSA_SYSTEM_INFO_TIMESTAMP, &ts);
            it.res->landed_ts.store(ts, std::memory_order_relaxed);
        }
        it.res->landed.fetch_add(1, std::memory_order_acq_rel);
    }
}

void stop_pump(ckpt_ctx* c)
{
    if (!c->pump) return;
    {
        std::lock_guard<std::mutex> l(c->pump->m);
        c->pump->stop = true;
    }
    c->pump->cv.notify_all();
    if (c->pump->issuer.joinable()) c->pump->issuer.join();
    if (c->pump->drainer.joinable()) c->pump->drainer.join();
    delete c->pump;
    c->pump = nullptr;
}

} // namespace ckpt
