// ckpt_runtime.cpp -- host side of libckpt (the C ABI of include/ckpt.h).
//
// One snapshot (paper Sec. V-B, D2H phase; Sec. VI-A, ping-pong buffers and
// the wait before the optimizer step), chunk group by chunk group g:
//
//   pack stream  : [wait: area_done[area(g)] >= uses of the area issued so far]
//                  pack kernel (fragments -> staging, tile sums)
//                  event captured[g]            <- the gate waits on this
//                  release kernel: dep[g] = 0
//   SDMA engine e: (polls dep[g]) copy staging(g) -> pinned image   -> copied[g]
//   counter engine: (after copied[g]) 8-byte copy: area_done[area(g)] = use count
//   after the last group: one reduce kernel (tile sums -> chunk sums), release
//   dep_sums; SDMA copies the chunk sums.
//
// Every copy completes into a signal of its own that starts at 1 (the
// area-done copy of group g into flagged[g], the sums copy into `done`), so
// the snapshot is committed exactly when `done` and every flagged[g] have
// reached 0.
//
// The image copies go to the DMA engines through the HSA runtime that HIP
// itself runs on, two engines taking alternate groups (one engine alone
// does not fill the host link).  A plain hipMemcpyAsync D2H may instead be
// run as a copy kernel on the compute units, competing with the pack and
// with the training step.
//
// The two images alternate: one holds the newest committed snapshot, the
// other receives the snapshot in flight, and a new snapshot may start only
// once the previous one has committed (CKPT_EBUSY otherwise).  So a
// committed image exists at every point once the first snapshot has
// committed, and an interrupted snapshot is never the recovery point
// (invariant I4 of Sec. V-C).
//
// Recovery (Sec. V-C third stage, Sec. VI-E) reverses the path group by
// group: DMA host image -> staging on the copy stream, then the scatter
// kernel on the pack stream writes the fragments and re-checks the sums.
//
// Here: context set-up, registration and its layout, the snapshot records,
// the gate, restore and verify entry points, and the accessors.  Issuing a
// snapshot (ckpt_snapshot.cpp), the restore and verify pipeline
// (ckpt_check.cpp), the bounce-mode pump (ckpt_bounce.cpp), the image file
// (ckpt_file.cpp) and replication (ckpt_h2h.cpp) have files of their own;
// ckpt_host.h holds what they share.
#include "ckpt_host.h"

namespace ckpt {

ckpt_status fail(ckpt_ctx* c, ckpt_status code, const char* fmt, ...)
{
    if (c) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        c->err = buf;
    }
    return code;
}

const char* hsa_text(hsa_status_t s)
{
    const char* t = nullptr;
    if (hsa_status_string(s, &t) != HSA_STATUS_SUCCESS || !t) return "unknown HSA status";
    return t;
}

bool is_pow2(uint64_t x) { return x && !(x & (x - 1)); }
uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool geometry_ok(uint64_t C, uint32_t A) { return is_pow2(A) && A >= 16 && A <= 4096 && C && C % A == 0; }

// Layout and tile table of a fragment list (no GPU involved).
struct Plan {
    std::vector<uint64_t> off, end; // image offset and end of the padded span per fragment
    uint64_t I = 0, n_chunks = 0, n_tiles = 0;
    uint32_t tile_shift = 4;
    std::vector<uint32_t> tile_first, tile_last;
};

bool plan(const uint64_t* nb, uint32_t n, uint64_t C, uint32_t A, Plan* p, bool tiles = true)
{
    // Registration order; each fragment starts at the previous end rounded
    // up to the alignment; the image ends on the alignment too.
    p->off.resize(n);
    p->end.resize(n);
    uint64_t end = 0;
    for (uint32_t i = 0; i < n; ++i) {
        p->off[i] = round_up(end, A);
        end = p->off[i] + nb[i];
    }
    p->I = round_up(end, A);
    if (p->I == 0) return false;
    for (uint32_t i = 0; i < n; ++i) p->end[i] = (i + 1 < n) ? p->off[i + 1] : p->I;
    p->n_chunks = (p->I + C - 1) / C;
    // Tiles: the largest power of two <= 8 KiB dividing the chunk size.
    const uint32_t ts = tile_shift_for(C);
    p->tile_shift = ts;
    p->n_tiles = (p->I + (1ull << ts) - 1) >> ts;
    if (!tiles) return true;
    p->tile_first.resize(p->n_tiles);
    p->tile_last.resize(p->n_tiles);
    // The fragment holding byte x is the first one whose padded span
    // [off, end) ends past x (empty fragments have empty spans).
    uint32_t i = 0;
    for (uint64_t t = 0; t < p->n_tiles; ++t) {
        const uint64_t x0 = t << ts;
        const uint64_t x1 = std::min<uint64_t>(x0 + (1ull << ts), p->I) - 1;
        while (i + 1 < n && p->end[i] <= x0) ++i;
        p->tile_first[t] = i;
        uint32_t j = i;
        while (j + 1 < n && p->end[j] <= x1) ++j;
        p->tile_last[t] = j;
    }
    return true;
}

// Direct D2H plan: for each chunk group of `unit` bytes of an image of I
// bytes, the pieces of fragments inside it (src = byte offset inside
// fragment piece_frag[k]; off = image offset) and the padding runs between
// them, both in image order, with each group's first piece and run.  False
// when a group holds no fragment byte (never, for layouts of plan(): every
// chunk starts with a fragment byte).
bool direct_plan(const uint64_t* off, const uint64_t* nb, uint32_t n, uint64_t I, uint64_t unit,
                 std::vector<Piece>& pieces, std::vector<uint32_t>& piece_frag, std::vector<Piece>& gaps,
                 std::vector<uint64_t>& piece_first, std::vector<uint64_t>& gap_first)
{
    const uint64_t n_groups = (I + unit - 1) / unit;
    pieces.clear();
    piece_frag.clear();
    gaps.clear();
    piece_first.assign(n_groups + 1, 0);
    gap_first.assign(n_groups + 1, 0);
    uint32_t i = 0;
    for (uint64_t g = 0; g < n_groups; ++g) {
        const uint64_t lo = g * unit, hi = std::min(lo + unit, I);
        piece_first[g] = pieces.size();
        gap_first[g] = gaps.size();
        uint64_t x = lo; // next image byte not yet covered
        while (i < n && (nb[i] == 0 || off[i] + nb[i] <= lo)) ++i;
        for (uint32_t k = i; k < n && off[k] < hi; ++k) {
            if (!nb[k]) continue;
            const uint64_t a = std::max(lo, off[k]), b = std::min(hi, off[k] + nb[k]);
            if (a > x) gaps.push_back(Piece{0, x, a - x});
            pieces.push_back(Piece{a - off[k], a, b - a});
            piece_frag.push_back(k);
            x = b;
        }
        if (x < hi) gaps.push_back(Piece{0, x, hi - x});
        if (pieces.size() == piece_first[g]) return false;
    }
    piece_first[n_groups] = pieces.size();
    gap_first[n_groups] = gaps.size();
    return true;
}

ckpt_status make_event(ckpt_ctx* c, hipEvent_t* e, bool timed)
{
    HIPCHK(c, hipEventCreateWithFlags(e, timed ? hipEventDefault : hipEventDisableTiming));
    return CKPT_OK;
}

// ---- HSA: agents and engines ------------------------------------------------

struct AgentSearch {
    uint32_t bdf;
    uint32_t domain;
    hsa_agent_t found;
    bool ok;
};

hsa_status_t find_gpu_cb(hsa_agent_t a, void* data)
{
    AgentSearch* s = (AgentSearch*)data;
    hsa_device_type_t type;
    if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &type) != HSA_STATUS_SUCCESS || type != HSA_DEVICE_TYPE_GPU)
        return HSA_STATUS_SUCCESS;
    uint32_t bdf = 0, domain = 0;
    hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_BDFID, &bdf);
    hsa_agent_get_info(a, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_DOMAIN, &domain);
    if (bdf == s->bdf && domain == s->domain) {
        s->found = a;
        s->ok = true;
        return HSA_STATUS_INFO_BREAK;
    }
    return HSA_STATUS_SUCCESS;
}

// The HSA agent of the context's device (matched by PCI location) and the
// DMA engines for device-to-host copies.
ckpt_status setup_hsa(ckpt_ctx* c)
{
    static std::once_flag once;
    static hsa_status_t init_status = HSA_STATUS_SUCCESS;
    std::call_once(once, [] { init_status = hsa_init(); }); // reference-counted; HIP has initialized it too
    HSACHK(c, init_status);
    int bus = 0, dev = 0, dom = 0;
    HIPCHK(c, hipDeviceGetAttribute(&bus, hipDeviceAttributePciBusId, c->device));
    HIPCHK(c, hipDeviceGetAttribute(&dev, hipDeviceAttributePciDeviceId, c->device));
    HIPCHK(c, hipDeviceGetAttribute(&dom, hipDeviceAttributePciDomainID, c->device));
    AgentSearch s{(uint32_t)((bus << 8) | (dev << 3)), (uint32_t)dom, {0}, false};
    hsa_status_t st = hsa_iterate_agents(find_gpu_cb, &s);
    if (st != HSA_STATUS_SUCCESS && st != HSA_STATUS_INFO_BREAK) HSACHK(c, st);
    if (!s.ok) return fail(c, CKPT_EHIP, "no HSA agent at PCI %04x:%02x:%02x", dom, bus, dev);
    c->gpu_agent = s.found;
    HSACHK(c, hsa_system_get_info(HSA_SYSTEM_INFO_TIMESTAMP_FREQUENCY, &c->ts_freq));
    return CKPT_OK;
}

// Owner agent of the pinned memory the engines write for image b (the image
// itself, or the bounce ring), and the engines for copies from the device.
ckpt_status setup_image_agent(ckpt_ctx* c, int b, const void* pinned)
{
    hsa_amd_pointer_info_t info;
    std::memset(&info, 0, sizeof info);
    info.size = sizeof info;
    HSACHK(c, hsa_amd_pointer_info(const_cast<void*>(pinned), &info, nullptr, nullptr, nullptr));
    c->img_agent[b] = info.agentOwner;
    hsa_device_type_t type = HSA_DEVICE_TYPE_GPU;
    if (info.agentOwner.handle) hsa_agent_get_info(info.agentOwner, HSA_AGENT_INFO_DEVICE, &type);
    if (type != HSA_DEVICE_TYPE_CPU) { // take the first CPU agent
        hsa_status_t st = hsa_iterate_agents(
            [](hsa_agent_t a, void* data) -> hsa_status_t {
                hsa_device_type_t t;
                if (hsa_agent_get_info(a, HSA_AGENT_INFO_DEVICE, &t) == HSA_STATUS_SUCCESS && t == HSA_DEVICE_TYPE_CPU) {
                    *(hsa_agent_t*)data = a;
                    return HSA_STATUS_INFO_BREAK;
                }
                return HSA_STATUS_SUCCESS;
            },
            &c->img_agent[b]);
        if (st != HSA_STATUS_SUCCESS && st != HSA_STATUS_INFO_BREAK) HSACHK(c, st);
    }
    if (b == 0) {
        uint32_t mask = 0;
        HSACHK(c, hsa_amd_memory_copy_engine_status(c->img_agent[0], c->gpu_agent, &mask));
        c->n_d2h_engines = 0;
        const int cap = c->d2h_engines_cfg ? std::min<int>((int)c->d2h_engines_cfg, kMaxEngines) : kMaxEngines;
        for (int k = 0; k < 16 && c->n_d2h_engines < cap; ++k)
            if (mask & (1u << k)) c->d2h_engine[c->n_d2h_engines++] = (hsa_amd_sdma_engine_id_t)(1u << k);
        if (c->n_d2h_engines == 0) return fail(c, CKPT_EHIP, "no DMA engine available for device-to-host copies");
        // The 8-byte staging-counter copies (host -> device) get an engine
        // that carries no image copy when there is one: an engine runs its
        // requests in order, so a counter copy queued behind another group's
        // image copy would hold back the next pack of that staging area.
        uint32_t hmask = 0, used = 0;
        HSACHK(c, hsa_amd_memory_copy_engine_status(c->gpu_agent, c->img_agent[0], &hmask));
        for (int k = 0; k < c->n_d2h_engines; ++k) used |= (uint32_t)c->d2h_engine[k];
        c->h2d_engine = c->d2h_engine[0];
        bool own = false;
        for (int k = 0; k < 16 && !own; ++k)
            if ((hmask & (1u << k)) && !(used & (1u << k))) {
                c->h2d_engine = (hsa_amd_sdma_engine_id_t)(1u << k);
                own = true;
            }
        for (int k = 0; k < 16 && !own; ++k)
            if (hmask & (1u << k)) {
                c->h2d_engine = (hsa_amd_sdma_engine_id_t)(1u << k);
                own = true;
            }
    }
    return CKPT_OK;
}

void destroy_res(RecRes* r)
{
    for (auto e : r->captured)
        if (e) (void)hipEventDestroy(e);
    for (auto e : r->k0)
        if (e) (void)hipEventDestroy(e);
    for (auto e : r->k1)
        if (e) (void)hipEventDestroy(e);
    if (r->t0) (void)hipEventDestroy(r->t0);
    if (r->t_red) (void)hipEventDestroy(r->t_red);
    for (auto s : r->dep)
        if (s.handle) hsa_signal_destroy(s);
    for (auto s : r->copied)
        if (s.handle) hsa_signal_destroy(s);
    for (auto s : r->flagged)
        if (s.handle) hsa_signal_destroy(s);
    for (auto s : r->piece_done)
        if (s.handle) hsa_signal_destroy(s);
    if (r->dep_sums.handle) hsa_signal_destroy(r->dep_sums);
    if (r->done.handle) hsa_signal_destroy(r->done);
    if (r->h_seq) (void)hipHostFree(r->h_seq);
    if (r->d_sums) (void)hipFree(r->d_sums);
    delete r;
}

ckpt_status gpu_only_signal(ckpt_ctx* c, hsa_signal_t* s, int64_t** val)
{
    HSACHK(c, hsa_amd_signal_create(1, 0, nullptr, HSA_AMD_SIGNAL_AMD_GPU_ONLY, s));
    volatile hsa_signal_value_t* p = nullptr;
    HSACHK(c, hsa_amd_signal_value_pointer(*s, &p));
    if (val) *val = (int64_t*)p;
    return CKPT_OK;
}

// A signal only the GPU waits on (no interrupt event behind it); the host
// may still read it.
ckpt_status gpu_consumed_signal(ckpt_ctx* c, hsa_signal_t* s)
{
    HSACHK(c, hsa_signal_create(0, 1, &c->gpu_agent, s));
    return CKPT_OK;
}

ckpt_status new_res(ckpt_ctx* c, RecRes** out)
{
    RecRes* r = new RecRes();
    const uint64_t n = c->n_groups;
    r->captured.assign(n, nullptr);
    r->k0.assign(n, nullptr);
    r->k1.assign(n, nullptr);
    r->dep.assign(n, hsa_signal_t{0});
    r->dep_val.assign(n, nullptr);
    r->copied.assign(n, hsa_signal_t{0});
    r->flagged.assign(n, hsa_signal_t{0});
    ckpt_status st = CKPT_OK;
    for (uint64_t g = 0; g < n && st == CKPT_OK; ++g) {
        st = make_event(c, &r->captured[g], false);
        if (st == CKPT_OK) st = make_event(c, &r->k0[g], true);
        if (st == CKPT_OK) st = make_event(c, &r->k1[g], true);
        if (st == CKPT_OK) st = gpu_only_signal(c, &r->dep[g], &r->dep_val[g]);
        if (st == CKPT_OK) st = gpu_consumed_signal(c, &r->copied[g]);
        if (st == CKPT_OK) st = gpu_consumed_signal(c, &r->flagged[g]);
    }
    if (c->direct) { // a completion signal per piece (its group's last piece signals `copied`)
        r->piece_done.assign(c->pieces.size(), hsa_signal_t{0});
        for (uint64_t g = 0; g < n && st == CKPT_OK; ++g)
            for (uint64_t k = c->piece_first[g]; k + 1 < c->piece_first[g + 1] && st == CKPT_OK; ++k)
                st = gpu_consumed_signal(c, &r->piece_done[k]);
    }
    if (st == CKPT_OK) st = make_event(c, &r->t0, true);
    if (st == CKPT_OK) st = make_event(c, &r->t_red, true);
    if (st == CKPT_OK) st = gpu_only_signal(c, &r->dep_sums, &r->dep_sums_val);
    if (st == CKPT_OK && hsa_signal_create(0, 0, nullptr, &r->done) != HSA_STATUS_SUCCESS) {
        r->done.handle = 0;
        st = fail(c, CKPT_EHIP, "hsa_signal_create failed");
    }
    if (st == CKPT_OK && hipHostMalloc((void**)&r->h_seq, std::max<uint64_t>(n, 1) * 8, hipHostMallocDefault) != hipSuccess) {
        r->h_seq = nullptr;
        st = fail(c, CKPT_ENOMEM, "pinned use-number slots");
    }
    if (st == CKPT_OK && hipMalloc(&r->d_sums, std::max<uint64_t>(c->n_chunks, 1) * 8) != hipSuccess) {
        r->d_sums = nullptr;
        st = fail(c, CKPT_ENOMEM, "hipMalloc of %llu chunk sums failed", (unsigned long long)c->n_chunks);
    }
    if (st != CKPT_OK) {
        destroy_res(r);
        return st;
    }
    *out = r;
    return CKPT_OK;
}

ckpt_status get_res(ckpt_ctx* c, RecRes** out)
{
    if (!c->free_res.empty()) {
        *out = c->free_res.back();
        c->free_res.pop_back();
        return CKPT_OK;
    }
    return new_res(c, out);
}

bool res_done(const RecRes* res, uint32_t groups_copied, bool bounce)
{
    if (hsa_signal_load_scacquire(res->done) != 0) return false;
    for (uint32_t g = 0; g < groups_copied; ++g)
        if (hsa_signal_load_scacquire(res->flagged[g]) != 0) return false;
    if (bounce && res->landed.load(std::memory_order_acquire) < groups_copied) return false;
    return true;
}

bool copies_done(const SnapRec& r)
{
    // an interrupted or failed snapshot never gets a record
    return res_done(r.res, r.groups_copied, r.bounce) &&
           (!r.file || r.aborted || r.res->failed.load(std::memory_order_acquire) ||
            r.res->recorded.load(std::memory_order_acquire));
}

bool pump_failed(ckpt_ctx* c, std::string* why)
{
    if (!c->pump) return false;
    std::lock_guard<std::mutex> l(c->pump->m);
    if (why) *why = c->pump->err;
    return c->pump->failed;
}

// Wait (bounded) until every copy of a snapshot has finished.
ckpt_status wait_copies(ckpt_ctx* c, SnapRec& r)
{
    // The wait's timeout is only a hint (in system-timestamp ticks): wait in
    // one-second slices against our own deadline.
    const auto deadline = std::chrono::steady_clock::now() + std::chrono::seconds(120);
    while (hsa_signal_wait_scacquire(r.res->done, HSA_SIGNAL_CONDITION_EQ, 0, c->ts_freq, HSA_WAIT_STATE_BLOCKED) != 0)
        if (std::chrono::steady_clock::now() > deadline)
            return fail(c, CKPT_EHIP, "snapshot %llu: chunk sums not copied after 120 s", (unsigned long long)r.id);
    // The per-group signals have the GPU as their only waiter; the host
    // polls their values (the engines run the groups in order, so this
    // rarely finds one still pending once the sums have landed).
    for (uint32_t g = 0; g < r.groups_copied; ++g) {
        while (hsa_signal_load_scacquire(r.res->flagged[g]) != 0) {
            if (std::chrono::steady_clock::now() > deadline)
                return fail(c, CKPT_EHIP, "snapshot %llu: group %u not copied after 120 s", (unsigned long long)r.id, g);
            std::this_thread::sleep_for(std::chrono::microseconds(20));
        }
    }
    if (r.bounce) { // every group also has to reach the pageable image
        while (r.res->landed.load(std::memory_order_acquire) < r.groups_copied) {
            if (std::chrono::steady_clock::now() > deadline)
                return fail(c, CKPT_EHIP, "snapshot %llu: image not written after 120 s", (unsigned long long)r.id);
            std::this_thread::sleep_for(std::chrono::microseconds(50));
        }
        std::string why;
        if (r.res->failed.load(std::memory_order_acquire) || pump_failed(c, &why))
            return fail(c, CKPT_EHIP, "snapshot %llu: bounce copy failed: %s", (unsigned long long)r.id, why.c_str());
        while (r.file && !r.aborted && !r.res->recorded.load(std::memory_order_acquire)) {
            if (std::chrono::steady_clock::now() > deadline)
                return fail(c, CKPT_EHIP, "snapshot %llu: commit record not written after 120 s", (unsigned long long)r.id);
            std::this_thread::sleep_for(std::chrono::microseconds(50));
        }
    }
    return CKPT_OK;
}

// Has the snapshot committed?  (Never true for an interrupted one.)
bool query_committed(SnapRec& r)
{
    if (r.aborted) return false;
    if (!r.committed && copies_done(r)) {
        if (r.res->failed.load(std::memory_order_acquire)) { // a group never reached the image
            r.aborted = true;
            return false;
        }
        r.committed = true;
    }
    return r.committed;
}

// Drop records that are neither among the newest four nor held by an image
// and whose copies are all finished.
void prune(ckpt_ctx* c)
{
    for (auto it = c->recs.begin(); it != c->recs.end();) {
        SnapRec& r = it->second;
        const bool held = (c->holder[0] == r.id || c->holder[1] == r.id);
        if (!held && r.id + 4 < c->next_id && copies_done(r)) {
            c->free_res.push_back(r.res);
            it = c->recs.erase(it);
        } else {
            ++it;
        }
    }
}

// Wait for every enqueued kernel and copy of the context.
ckpt_status drain(ckpt_ctx* c)
{
    for (hipStream_t st : {c->s_pack, c->s_copy, c->s_vcopy, c->s_vker})
        if (st) HIPCHK(c, hipStreamSynchronize(st));
    for (auto& kv : c->recs) {
        ckpt_status st = wait_copies(c, kv.second);
        if (st) return st;
    }
    return CKPT_OK;
}

// Resolve snap_id (0 = newest committed) to a committed, still-held record.
ckpt_status pick_target_image(ckpt_ctx* c, int* out)
{
    // At most one uncommitted snapshot; find the newest live one.
    int in_flight = 0;
    SnapRec* newest_live = nullptr;
    for (auto& kv : c->recs) {
        SnapRec& r = kv.second;
        if (r.aborted) continue;
        if (!query_committed(r)) ++in_flight;
        if (!newest_live || r.id > newest_live->id) newest_live = &r;
    }
    // One image always holds the newest committed snapshot and the other
    // receives the one in flight (Sec. VI-A): a snapshot may start only once
    // the previous one has committed.
    if (in_flight >= 1) return fail(c, CKPT_EBUSY, "the previous snapshot has not committed yet");
    // Target: the image not holding the newest live snapshot; with no live
    // snapshot, an image that holds nothing committed.
    int buf = 0;
    if (newest_live) {
        buf = 1 - newest_live->buf;
    } else {
        for (int b = 0; b < 2; ++b) {
            auto it = c->recs.find(c->holder[b]);
            if (c->holder[b] == 0 || it == c->recs.end() || it->second.aborted) {
                buf = b;
                break;
            }
        }
    }
    if (rep_busy(c, buf))
        return fail(c, CKPT_EBUSY, "the snapshot in host image %d is still being sent to a peer", buf);
    *out = buf;
    return CKPT_OK;
}

ckpt_status pick_committed(ckpt_ctx* c, uint64_t snap_id, SnapRec** out)
{
    SnapRec* best = nullptr;
    for (auto& kv : c->recs) {
        SnapRec& r = kv.second;
        if (!query_committed(r) || c->holder[r.buf] != r.id) continue;
        if (snap_id != 0 && r.id != snap_id) continue;
        if (!best || r.id > best->id) best = &r;
    }
    if (!best) {
        if (snap_id != 0 && !c->recs.count(snap_id) && snap_id >= c->next_id)
            return fail(c, CKPT_ERANGE, "snapshot %llu does not exist", (unsigned long long)snap_id);
        return fail(c, CKPT_ENOSNAP, "no committed snapshot%s", snap_id ? " with that id is still held" : "");
    }
    *out = best;
    return CKPT_OK;
}

// Zero a pinned host image from several threads, so that its pages are
// resident before the first snapshot streams into it.
void parallel_zero(uint8_t* p, uint64_t n)
{
    unsigned nt = std::thread::hardware_concurrency();
    nt = std::max(1u, std::min(nt, 16u));
    if (n < (64ull << 20)) nt = 1;
    std::vector<std::thread> th;
    const uint64_t per = (n / nt + 4095) & ~4095ull;
    for (unsigned k = 0; k < nt; ++k) {
        const uint64_t lo = std::min<uint64_t>(k * per, n), hi = std::min<uint64_t>(lo + per, n);
        th.emplace_back([=] { std::memset(p + lo, 0, hi - lo); });
    }
    for (auto& t : th) t.join();
}

float elapsed(hipEvent_t a, hipEvent_t b)
{
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, a, b) != hipSuccess) return -1.f;
    return ms;
}

// Restore (scatter=true) or verify (scatter=false) from a committed image.
// Restore first waits for every outstanding snapshot (it rewrites the live
// tensors and shares the snapshot staging).  Verify only reads a committed
// image, which no in-flight snapshot targets, through its own staging ring
// and streams, so it may run while a newer snapshot streams out: the host
// link is full duplex.
ckpt_status run_check(ckpt_ctx* c, uint64_t snap_id, hipStream_t stream, bool scatter, uint32_t* bad_chunks,
                      uint32_t cap, uint32_t* n_bad)
{
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    if (!n_bad || (cap && !bad_chunks)) return fail(c, CKPT_EINVAL, "null output pointer");
    HIPCHK(c, hipSetDevice(c->device));
    ckpt_status st = CKPT_OK;
    if (scatter) {
        st = drain(c);
        if (st) return st;
    }
    SnapRec* r = nullptr;
    st = pick_committed(c, snap_id, &r);
    if (st) return st;
    return check_image(c, r->buf, stream, scatter, nullptr, bad_chunks, cap, n_bad);
}

void free_ctx(ckpt_ctx* c)
{
    rep_stop(c); // reads host images and snapshot records
    stop_pump(c);
    delete c->pool;
    c->pool = nullptr;
    for (auto& kv : c->recs) c->free_res.push_back(kv.second.res);
    c->recs.clear();
    for (auto r : c->free_res) destroy_res(r);
    c->free_res.clear();
    for (auto e : c->area_free) (void)hipEventDestroy(e);
    for (auto e : c->ev_loaded) (void)hipEventDestroy(e);
    for (auto* v : {&c->tk0, &c->tk1, &c->vfree, &c->vloaded, &c->vk0, &c->vk1, &c->bin_done})
        for (auto e : *v) (void)hipEventDestroy(e);
    for (hipEvent_t e : {c->ev_trigger, c->ev_done, c->tt0, c->tc0, c->tc1, c->ev_vdone, c->vt0, c->vc0, c->vc1})
        if (e) (void)hipEventDestroy(e);
    (void)hipFree(c->d_vring);
    (void)hipFree(c->d_frags);
    (void)hipFree(c->d_tile_first);
    (void)hipFree(c->d_tile_last);
    (void)hipFree(c->d_staging);
    (void)hipFree(c->d_partials);
    (void)hipFree(c->d_expected);
    (void)hipFree(c->d_recomputed);
    (void)hipFree(c->d_bad);
    (void)hipFree(c->d_area_done);
    for (int b = 0; b < 2; ++b) {
        if (c->file_map) {
            // part of the file mapping
        } else if (c->h_img[b] && c->img_map_bytes) {
            (void)munmap(c->h_img[b], c->img_map_bytes);
        } else if (c->h_img[b]) {
            (void)hipHostFree(c->h_img[b]);
        }
        if (c->h_sums[b]) (void)hipHostFree(c->h_sums[b]);
    }
    if (c->file_map) (void)munmap(c->file_map, c->fhead.file_bytes);
    if (c->file_fd >= 0) (void)::close(c->file_fd);
    if (c->h_bout) (void)hipHostFree(c->h_bout);
    if (c->h_bin) (void)hipHostFree(c->h_bin);
    if (c->h_bad) (void)hipHostFree(c->h_bad);
    if (c->h_recomputed) (void)hipHostFree(c->h_recomputed);
    if (!c->own_pack) c->s_pack = nullptr; // the caller's stream
    for (hipStream_t st : {c->s_pack, c->s_copy, c->s_vcopy, c->s_vker})
        if (st) (void)hipStreamDestroy(st);
}

// Issue one SDMA copy; on failure the dependency chain of the snapshot is
// released so no engine is left polling.
ckpt_status dma(ckpt_ctx* c, void* dst, hsa_agent_t dst_agent, const void* src, hsa_agent_t src_agent, uint64_t n,
                const hsa_signal_t* dep, hsa_signal_t completion, hsa_amd_sdma_engine_id_t engine)
{
    HSACHK(c, hsa_amd_memory_async_copy_on_engine(dst, dst_agent, src, src_agent, n, dep ? 1 : 0, dep, completion,
                                                  engine, true));
    return CKPT_OK;
}

// The envelope of a snapshot (format in include/ckpt.h, ckpt_envelope).
std::vector<uint8_t> build_envelope(const ckpt_ctx* c, uint64_t step, const std::vector<uint8_t>& meta,
                                    const uint64_t* sums)
{
    const uint32_t nf = (uint32_t)c->frags.size();
    const uint64_t meta_pad = round_up(meta.size(), 8);
    const uint64_t total = 56 + 24ull * nf + 8 * c->n_chunks + meta_pad + 8;
    // x86-64 and gfx950 are little-endian: fields are stored in native order.
    std::vector<uint8_t> buf(total, 0);
    uint8_t* p = buf.data();
    struct __attribute__((packed)) Head {
        char magic[8];
        uint32_t version, align;
        uint64_t step, chunk, image, n_chunks;
        uint32_t n_frag, meta_len;
    } h;
    static_assert(sizeof(Head) == 56, "envelope header is 56 bytes");
    std::memcpy(h.magic, "CKPTENV1", 8);
    h.version = 1;
    h.align = c->A;
    h.step = step;
    h.chunk = c->C;
    h.image = c->I;
    h.n_chunks = c->n_chunks;
    h.n_frag = nf;
    h.meta_len = (uint32_t)meta.size();
    std::memcpy(p, &h, sizeof h);
    p += sizeof h;
    for (uint32_t i = 0; i < nf; ++i) {
        struct __attribute__((packed)) Ent {
            uint64_t off, nbytes;
            uint32_t dtype, cls;
        } e{c->frags[i].off, c->frags[i].nbytes, c->frags[i].dtype, c->frags[i].cls};
        std::memcpy(p, &e, sizeof e);
        p += sizeof e;
    }
    std::memcpy(p, sums, c->n_chunks * 8);
    p += c->n_chunks * 8;
    if (!meta.empty()) std::memcpy(p, meta.data(), meta.size());
    p += meta_pad;
    uint64_t s = 0;
    for (const uint8_t* q = buf.data(); q < p; q += 8) {
        uint64_t w;
        std::memcpy(&w, q, 8);
        s += w;
    }
    std::memcpy(p, &s, 8);
    return buf;
}


} // namespace ckpt

extern "C" {

ckpt_status ckpt_create(const ckpt_config* cfg, ckpt_ctx** out)
{
    if (!out) return CKPT_EINVAL;
    *out = nullptr;
    ckpt_config d{};
    if (cfg) d = *cfg;
    const uint64_t C = d.chunk_bytes ? d.chunk_bytes : kDefaultChunk;
    const uint32_t A = d.align_bytes ? d.align_bytes : kDefaultAlign;
    if (!geometry_ok(C, A)) return CKPT_EINVAL;
    if (d.host_buffers != 0 && d.host_buffers != 2) return CKPT_EINVAL;
    if (d.device_staging_bytes && d.device_staging_bytes < 2 * C) return CKPT_EINVAL;
    if (d.bounce_bytes && d.bounce_bytes < 2 * C) return CKPT_EINVAL;
    if (d.host_threads > 256) return CKPT_EINVAL;
    if (d.direct_d2h && (d.device_staging_bytes || d.poison)) return CKPT_EINVAL; // no snapshot staging
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || d.device < 0 || d.device >= ndev) return CKPT_EINVAL;
    ckpt_ctx* c = new ckpt_ctx();
    c->device = d.device;
    c->C = C;
    c->A = A;
    c->staging_cap = d.device_staging_bytes;
    c->group_cfg = d.group_bytes ? d.group_bytes : kDefaultGroup;
    c->group_set = d.group_bytes != 0;
    c->grid_cap = d.grid_blocks ? d.grid_blocks : kDefaultGrid;
    c->bounce_cfg = d.bounce_bytes;
    if (d.pack_launch_bytes) c->launch_cfg = d.pack_launch_bytes;
    c->d2h_engines_cfg = d.d2h_engines;
    c->poison = d.poison != 0;
    c->direct = d.direct_d2h != 0;
    c->host_threads = d.host_threads ? d.host_threads : kDefaultHostThreads;
    ckpt_status st = CKPT_OK;
    if (hipSetDevice(c->device) != hipSuccess)
        st = CKPT_EHIP;
    if (d.side_stream) { // the caller's dedicated stream carries the pack
        c->s_pack = (hipStream_t)d.side_stream;
        c->own_pack = false;
    }
    for (hipStream_t* sp : {&c->s_pack, &c->s_copy, &c->s_vcopy, &c->s_vker})
        if (st == CKPT_OK && !*sp && hipStreamCreateWithFlags(sp, hipStreamNonBlocking) != hipSuccess) st = CKPT_EHIP;
    for (hipEvent_t* e : {&c->ev_trigger, &c->ev_done, &c->ev_vdone})
        if (st == CKPT_OK) st = make_event(c, e, false);
    for (hipEvent_t* e : {&c->tt0, &c->tc0, &c->tc1, &c->vt0, &c->vc0, &c->vc1})
        if (st == CKPT_OK) st = make_event(c, e, true);
    if (st == CKPT_OK) st = setup_hsa(c);
    if (st != CKPT_OK) {
        free_ctx(c);
        delete c;
        return st;
    }
    *out = c;
    return CKPT_OK;
}

ckpt_status ckpt_destroy(ckpt_ctx* ctx)
{
    if (!ctx) return CKPT_OK;
    (void)hipSetDevice(ctx->device);
    (void)drain(ctx);
    free_ctx(ctx);
    delete ctx;
    return CKPT_OK;
}

ckpt_status ckpt_register_tensors(ckpt_ctx* c, const ckpt_tensor* t, uint32_t n)
{
    if (!c) return CKPT_EINVAL;
    if (c->registered) return fail(c, CKPT_ESTATE, "tensors already registered");
    if (!t || n == 0) return fail(c, CKPT_EINVAL, "need at least one fragment");
    HIPCHK(c, hipSetDevice(c->device));
    std::vector<uint64_t> nb(n);
    for (uint32_t i = 0; i < n; ++i) {
        if (t[i].nbytes && !t[i].dev_ptr) return fail(c, CKPT_EINVAL, "fragment %u: null pointer", i);
        nb[i] = t[i].nbytes;
        if (!nb[i]) continue;
        // The kernels dereference every fragment byte: the fragment has to be
        // memory of this context's GPU and lie inside one allocation, or the
        // first pack would fault instead of this call failing.
        hipPointerAttribute_t pa;
        std::memset(&pa, 0, sizeof pa);
        if (hipPointerGetAttributes(&pa, t[i].dev_ptr) != hipSuccess) {
            (void)hipGetLastError(); // leave no error behind for the next call to report
            return fail(c, CKPT_EINVAL, "fragment %u: %p is not memory the GPU runtime knows", i, t[i].dev_ptr);
        }
        if (pa.type != hipMemoryTypeDevice && !pa.isManaged)
            return fail(c, CKPT_EINVAL, "fragment %u: %p is not device memory (memory type %d)", i, t[i].dev_ptr,
                        (int)pa.type);
        if (pa.type == hipMemoryTypeDevice && pa.device != c->device)
            return fail(c, CKPT_EINVAL, "fragment %u: memory of device %d, the context is on device %d", i, pa.device,
                        c->device);
        hipDeviceptr_t base = nullptr;
        size_t size = 0;
        if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)t[i].dev_ptr) == hipSuccess) {
            const uint64_t lo = (uint64_t)(uintptr_t)t[i].dev_ptr, b = (uint64_t)(uintptr_t)base;
            if (lo < b || nb[i] > size || lo - b > size - nb[i])
                return fail(c, CKPT_EINVAL, "fragment %u: %llu bytes at %p run past the end of its allocation", i,
                            (unsigned long long)nb[i], t[i].dev_ptr);
        } else {
            (void)hipGetLastError();
        }
    }
    Plan pl;
    if (!plan(nb.data(), n, c->C, c->A, &pl)) return fail(c, CKPT_EINVAL, "all fragments are empty");
    c->frags.resize(n);
    uint64_t payload = 0;
    for (uint32_t i = 0; i < n; ++i) {
        Frag& f = c->frags[i];
        f.ptr = (uint64_t)(uintptr_t)t[i].dev_ptr;
        f.nbytes = nb[i];
        f.dtype = t[i].dtype;
        f.cls = t[i].cls;
        f.off = pl.off[i];
        payload += nb[i];
    }
    c->I = pl.I;
    c->payload = payload;
    c->n_chunks = pl.n_chunks;
    c->geo.image_bytes = c->I;
    c->geo.tile_shift = pl.tile_shift;
    c->geo.tiles_per_chunk = (uint32_t)(c->C >> pl.tile_shift);
    c->geo.n_tiles = pl.n_tiles;
    c->geo.n_chunks = c->n_chunks;

    // Groups: whole chunks per pack launch and DMA request.  In ring mode a
    // group fills one slot: group_bytes when given, else a quarter of the
    // ring (four slots; fewer groups cost less host time per snapshot), at
    // least one chunk and never more than half the ring.
    if (c->staging_cap) {
        c->ring = true;
        const uint64_t want = std::max<uint64_t>(1, (c->group_set ? c->group_cfg : c->staging_cap / 4) / c->C);
        c->G = std::max<uint64_t>(1, std::min<uint64_t>(want, c->staging_cap / (2 * c->C)));
    } else {
        c->G = std::max<uint64_t>(1, c->group_cfg / c->C);
    }
    c->n_groups = (c->n_chunks + c->G - 1) / c->G;
    // Pack launches of whole groups (full-image staging): a larger launch
    // spends less time in the gaps between launches, but slows concurrent
    // training kernels more, so the default is one group per launch; each
    // group keeps its own DMA request.  In ring mode a launch fills one slot.
    c->LG = (c->ring || c->direct || !c->launch_cfg) ? 1 : std::max<uint64_t>(1, c->launch_cfg / (c->G * c->C));
    c->n_launches = (c->n_groups + c->LG - 1) / c->LG;
    if (c->ring) c->n_slots = std::max<uint64_t>(1, std::min<uint64_t>(c->staging_cap / (c->G * c->C), c->n_groups));
    if (c->direct) c->n_slots = std::min<uint64_t>(kDirectRestoreSlots, c->n_groups);
    const uint64_t unit = c->G * c->C; // bytes of one chunk group
    if (c->bounce_cfg) {
        if (c->bounce_cfg / unit < 2)
            return fail(c, CKPT_EINVAL, "bounce ring of %llu bytes holds fewer than two chunk groups of %llu bytes",
                        (unsigned long long)c->bounce_cfg, (unsigned long long)unit);
        c->bounce = true;
        c->n_bslots = std::min<uint64_t>(c->bounce_cfg / unit, std::max<uint64_t>(2, c->n_groups));
    }

    std::vector<FragDev> fd(n);
    for (uint32_t i = 0; i < n; ++i) {
        fd[i].ptr = c->frags[i].ptr;
        fd[i].nbytes = nb[i];
        fd[i].off = pl.off[i];
        fd[i].end = pl.end[i];
    }
    if (c->direct) { // each group's fragment pieces and padding runs, copied and zeroed per snapshot
        std::vector<uint64_t> fo(n);
        for (uint32_t i = 0; i < n; ++i) fo[i] = c->frags[i].off;
        std::vector<uint32_t> pf;
        if (!direct_plan(fo.data(), nb.data(), n, c->I, c->G * c->C, c->pieces, pf, c->gaps, c->piece_first,
                         c->gap_first))
            return fail(c, CKPT_EINVAL, "a chunk group holds no fragment byte");
        if (c->pieces.size() > kMaxDirectPieces)
            return fail(c, CKPT_EINVAL, "direct D2H: %llu fragment pieces, at most %llu",
                        (unsigned long long)c->pieces.size(), (unsigned long long)kMaxDirectPieces);
        for (size_t k = 0; k < c->pieces.size(); ++k) c->pieces[k].src += c->frags[pf[k]].ptr;
    }
    const uint64_t nt = pl.n_tiles;
    const uint64_t n_areas = c->ring ? c->n_slots : c->n_groups;

#define ALLOC(ptr, bytes)                                                                                   \
    do {                                                                                                    \
        if (hipMalloc((void**)&(ptr), (bytes)) != hipSuccess) {                                             \
            (ptr) = nullptr;                                                                                \
            return fail(c, CKPT_ENOMEM, "hipMalloc(%llu) failed for " #ptr, (unsigned long long)(bytes));    \
        }                                                                                                   \
    } while (0)
    ALLOC(c->d_frags, n * sizeof(FragDev));
    ALLOC(c->d_tile_first, nt * 4);
    ALLOC(c->d_tile_last, nt * 4);
    ALLOC(c->d_partials, 2 * nt * kTileParts * 8);
    ALLOC(c->d_expected, c->n_chunks * 8);
    ALLOC(c->d_recomputed, c->n_chunks * 8);
    ALLOC(c->d_bad, c->n_chunks);
    ALLOC(c->d_area_done, n_areas * 8);
    ALLOC(c->d_staging, (c->ring || c->direct) ? c->n_slots * c->G * c->C : c->I);
    c->n_vslots = std::min<uint64_t>(kVerifySlots, c->n_groups);
    ALLOC(c->d_vring, c->n_vslots * c->G * c->C);
#undef ALLOC
    HIPCHK(c, hipMemcpy(c->d_frags, fd.data(), n * sizeof(FragDev), hipMemcpyHostToDevice));
    HIPCHK(c, hipMemcpy(c->d_tile_first, pl.tile_first.data(), nt * 4, hipMemcpyHostToDevice));
    HIPCHK(c, hipMemcpy(c->d_tile_last, pl.tile_last.data(), nt * 4, hipMemcpyHostToDevice));
    HIPCHK(c, hipMemset(c->d_area_done, 0, n_areas * 8));
    c->area_seq.assign(n_areas, 0);
    c->area_flag.assign(n_areas, hsa_signal_t{0});
    if (c->bounce) {
        for (uint8_t** ring : {&c->h_bout, &c->h_bin}) {
            if (hipHostMalloc((void**)ring, c->n_bslots * unit, hipHostMallocDefault) != hipSuccess) {
                *ring = nullptr;
                return fail(c, CKPT_ENOMEM, "pinned bounce ring of %llu bytes", (unsigned long long)(c->n_bslots * unit));
            }
            parallel_zero(*ring, c->n_bslots * unit);
        }
        c->img_map_bytes = round_up(c->I, 2ull << 20);
    }
    if (c->file_mode >= 0) {
        ckpt_status st = open_image_file(c);
        if (st) return st;
    }
    for (int b = 0; b < 2; ++b) {
        if (c->file_map) {
            // images live in the file
        } else if (c->bounce) {
            void* m = mmap(nullptr, c->img_map_bytes, PROT_READ | PROT_WRITE, MAP_PRIVATE | MAP_ANONYMOUS, -1, 0);
            if (m == MAP_FAILED)
                return fail(c, CKPT_ENOMEM, "host image of %llu bytes", (unsigned long long)c->img_map_bytes);
            c->h_img[b] = (uint8_t*)m;
            (void)madvise(m, c->img_map_bytes, MADV_HUGEPAGE);
        } else if (hipHostMalloc((void**)&c->h_img[b], c->I, hipHostMallocDefault) != hipSuccess) {
            c->h_img[b] = nullptr;
            return fail(c, CKPT_ENOMEM, "pinned host image of %llu bytes", (unsigned long long)c->I);
        }
        if (!c->file_map) parallel_zero(c->h_img[b], c->I);
        if (hipHostMalloc((void**)&c->h_sums[b], c->n_chunks * 8, hipHostMallocDefault) != hipSuccess) {
            c->h_sums[b] = nullptr;
            return fail(c, CKPT_ENOMEM, "pinned sums");
        }
        ckpt_status st = setup_image_agent(c, b, c->bounce ? (const void*)c->h_bout : (const void*)c->h_img[b]);
        if (st) return st;
    }
    if (hipHostMalloc((void**)&c->h_bad, c->n_chunks, hipHostMallocDefault) != hipSuccess ||
        hipHostMalloc((void**)&c->h_recomputed, c->n_chunks * 8, hipHostMallocDefault) != hipSuccess)
        return fail(c, CKPT_ENOMEM, "pinned result buffers");
    c->area_free.resize(n_areas, nullptr);
    for (auto& e : c->area_free) {
        ckpt_status st = make_event(c, &e, false);
        if (st) return st;
        HIPCHK(c, hipEventRecord(e, c->s_copy)); // every area starts free
    }
    c->ev_loaded.resize(c->n_groups, nullptr);
    c->tk0.resize(c->n_groups, nullptr);
    c->tk1.resize(c->n_groups, nullptr);
    for (uint64_t g = 0; g < c->n_groups; ++g) {
        ckpt_status st = make_event(c, &c->ev_loaded[g], false);
        if (!st) st = make_event(c, &c->tk0[g], true);
        if (!st) st = make_event(c, &c->tk1[g], true);
        if (st) return st;
    }
    c->vfree.resize(c->n_vslots, nullptr);
    for (auto& e : c->vfree) {
        ckpt_status st = make_event(c, &e, false);
        if (st) return st;
        HIPCHK(c, hipEventRecord(e, c->s_vker)); // every slot starts free
    }
    c->vloaded.resize(c->n_groups, nullptr);
    c->vk0.resize(c->n_groups, nullptr);
    c->vk1.resize(c->n_groups, nullptr);
    for (uint64_t k = 0; k < c->n_groups; ++k) {
        ckpt_status st = make_event(c, &c->vloaded[k], false);
        if (!st) st = make_event(c, &c->vk0[k], true);
        if (!st) st = make_event(c, &c->vk1[k], true);
        if (st) return st;
    }
    if (c->bounce) {
        c->bin_done.resize(c->n_bslots, nullptr);
        for (auto& e : c->bin_done) {
            ckpt_status st = make_event(c, &e, false);
            if (st) return st;
        }
        c->pool = new CopyPool(c->host_threads);
        c->pump = new Pump();
        c->pump->busy.assign(c->n_bslots, 0);
        c->pump->issuer = std::thread(pump_issue, c);
        c->pump->drainer = std::thread(pump_drain, c);
    }
    HIPCHK(c, hipDeviceSynchronize());
    c->registered = true;
    if (c->file_mode == CKPT_FILE_ADOPT) {
        ckpt_status st = adopt_image_file(c);
        if (st) return st;
    }
    return CKPT_OK;
}

ckpt_status ckpt_snapshot_async(ckpt_ctx* c, void* after_stream, uint64_t step, const void* meta,
                                uint32_t meta_len, uint64_t* snap_id)
{
    if (!c || !snap_id) return fail(c, CKPT_EINVAL, "null argument");
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    if (meta_len && !meta) return fail(c, CKPT_EINVAL, "meta is null");
    if (meta_len > kMaxMeta) return fail(c, CKPT_EINVAL, "meta blob larger than 1 MiB");
    HIPCHK(c, hipSetDevice(c->device));
    prune(c);
    int buf = 0;
    ckpt_status st = pick_target_image(c, &buf);
    if (st) return st;

    RecRes* res = nullptr;
    st = get_res(c, &res);
    if (st) return st;
    const uint64_t id = c->next_id++;
    SnapRec& r = c->recs[id];
    r.id = id;
    r.step = step;
    r.res = res;
    r.buf = buf;
    r.meta.assign((const uint8_t*)meta, (const uint8_t*)meta + meta_len);
    r.timed = c->timing;
    r.per_launch = c->timing && !c->timing_span;
    r.bounce = c->bounce;
    r.file = c->file_map != nullptr;
    res->landed.store(0, std::memory_order_relaxed);
    res->landed_ts.store(0, std::memory_order_relaxed);
    res->recorded_ts.store(0, std::memory_order_relaxed);
    res->failed.store(false, std::memory_order_relaxed);
    res->recorded.store(false, std::memory_order_relaxed);
    c->holder[r.buf] = id;
    const int32_t stop = c->interrupt_next;
    c->interrupt_next = -1;
    const uint64_t n_copy = (stop < 0) ? c->n_groups : std::min<uint64_t>((uint64_t)stop, c->n_groups);
    hipStream_t after = (hipStream_t)after_stream;
    // Completion signals start at 0 ("nothing pending"); each is raised to 1
    // just before its copy is issued.
    hsa_signal_store_screlease(res->done, 0);
    r.groups_copied = 0;
    if (r.timed && n_copy > 0) hsa_amd_profiling_async_copy_enable(true);

    // On an error below, copies not issued never raise their signals, and
    // the snapshot is marked interrupted.
    st = issue_snapshot(c, r, after, n_copy, stop);
    if (st) {
        r.aborted = true;
        r.timed = false;
        *snap_id = id;
        return st;
    }
    for (Replicator* R : c->reps) { // H2H once the offload commits, to every peer
        if (r.aborted) break;
        RepJob j;
        j.id = id;
        j.step = step;
        j.buf = r.buf;
        j.res = res;
        j.groups_copied = r.groups_copied;
        j.bounce = r.bounce;
        j.meta = r.meta;
        std::lock_guard<std::mutex> l(R->m);
        R->busy[r.buf] = true;
        while (!R->status.empty() && R->status.begin()->first + 64 < id &&
               R->status.begin()->second.state != REP_PENDING)
            R->status.erase(R->status.begin());
        R->status[id] = RepStatus{};
        R->q.push_back(std::move(j));
        R->cv.notify_all();
    }
    *snap_id = id;
    return CKPT_OK;
}

} // extern "C"

extern "C" {

ckpt_status ckpt_wait(ckpt_ctx* c, uint64_t snap_id, uint32_t mode, void* stream, uint32_t frag_lo,
                      uint32_t frag_hi)
{
    if (!c) return CKPT_EINVAL;
    if (mode == CKPT_WAIT_REPLICATED) {
        if (c->reps.empty()) return fail(c, CKPT_ESTATE, "no replication peer");
        // Every peer's answer; the worst one decides (failed, then corrupt).
        // No deadline of its own: each peer's worker bounds its waits (the
        // local commit, and no progress on its connection), so every job
        // ends with a verdict however long a flowing transfer takes.
        ckpt_status worst = CKPT_OK;
        std::string why;
        size_t asked = 0;
        for (size_t k = 0; k < c->reps.size(); ++k) {
            Replicator* R = c->reps[k];
            if (snap_id < R->first_id) continue; // this peer was added after the snapshot
            ++asked;
            std::unique_lock<std::mutex> l(R->m);
            auto s = R->status.find(snap_id);
            if (s == R->status.end())
                return fail(c, CKPT_ERANGE, "snapshot %llu is not being replicated", (unsigned long long)snap_id);
            R->cv.wait(l, [&] { return s->second.state != REP_PENDING; });
            if (s->second.state == REP_FAILED) {
                worst = CKPT_EHIP;
                why = "peer " + std::to_string(k) + ": " + s->second.err;
            } else if (s->second.state == REP_CORRUPT && worst == CKPT_OK) {
                worst = CKPT_ECORRUPT;
                why = "peer " + std::to_string(k) + " found " + std::to_string(s->second.bad.size()) +
                      " corrupt chunks";
            }
        }
        if (!asked)
            return fail(c, CKPT_ERANGE, "snapshot %llu was not sent to any current peer", (unsigned long long)snap_id);
        if (worst == CKPT_OK) return CKPT_OK;
        if (worst == CKPT_ECORRUPT)
            return fail(c, CKPT_ECORRUPT, "snapshot %llu: %s", (unsigned long long)snap_id, why.c_str());
        return fail(c, CKPT_EHIP, "snapshot %llu not replicated: %s", (unsigned long long)snap_id, why.c_str());
    }
    auto it = c->recs.find(snap_id);
    if (it == c->recs.end()) return fail(c, CKPT_ERANGE, "snapshot %llu not retained", (unsigned long long)snap_id);
    SnapRec& r = it->second;
    HIPCHK(c, hipSetDevice(c->device));
    if (mode == CKPT_WAIT_COMMITTED) {
        if (r.aborted) return fail(c, CKPT_ESTATE, "snapshot %llu was interrupted", (unsigned long long)snap_id);
        ckpt_status st = wait_copies(c, r);
        if (st) return st;
        r.committed = true;
        return CKPT_OK;
    }
    if (mode != CKPT_WAIT_CAPTURED) return fail(c, CKPT_EINVAL, "unknown wait mode %u", mode);
    const uint32_t n = (uint32_t)c->frags.size();
    if (frag_hi > n) frag_hi = n;
    if (frag_lo >= frag_hi) return fail(c, CKPT_EINVAL, "empty fragment range [%u, %u) of %u", frag_lo, frag_hi, n);
    // Last image byte of the range's non-empty fragments; packs run in group
    // order on one stream, so waiting for that byte's group covers the rest.
    uint64_t last = 0;
    bool any = false;
    for (uint32_t i = frag_hi; i-- > frag_lo;) {
        if (c->frags[i].nbytes) {
            last = c->frags[i].off + c->frags[i].nbytes - 1;
            any = true;
            break;
        }
    }
    if (!any) return CKPT_OK; // only empty fragments: nothing to protect
    if (c->direct) {
        // The copies of each group holding a byte of the range (the engines
        // finish groups out of order), each ending by setting the group's
        // counter to this snapshot's use number.  A group's copies start only
        // once the launch after its sums has started, so its counter also
        // covers the sums of every group up to it (launches run in order).
        // Groups an interrupted snapshot never copies have an event after
        // their sums instead.
        uint64_t first = 0;
        for (uint32_t i = frag_lo; i < frag_hi; ++i)
            if (c->frags[i].nbytes) {
                first = c->frags[i].off;
                break;
            }
        const uint64_t unit = c->G * c->C;
        const uint64_t g0 = first / unit, g1 = last / unit;
        if (g1 >= r.groups_copied) HIPCHK(c, hipStreamWaitEvent((hipStream_t)stream, r.res->captured[g1], 0));
        for (uint64_t g = g0; g <= g1 && g < r.groups_copied; ++g)
            HIPCHK(c, hipStreamWaitValue64((hipStream_t)stream, c->d_area_done + g, r.res->h_seq[g],
                                           hipStreamWaitValueGte, ~0ull));
        return CKPT_OK;
    }
    const uint64_t g = last / (c->G * c->C);
    const uint64_t gl = std::min((g / c->LG + 1) * c->LG, c->n_groups) - 1; // its launch's last group
    HIPCHK(c, hipStreamWaitEvent((hipStream_t)stream, r.res->captured[gl], 0));
    return CKPT_OK;
}

ckpt_status ckpt_snapshot_state(ckpt_ctx* c, uint64_t snap_id, uint32_t* state)
{
    if (!c || !state) return CKPT_EINVAL;
    auto it = c->recs.find(snap_id);
    if (it == c->recs.end()) return fail(c, CKPT_ERANGE, "snapshot %llu not retained", (unsigned long long)snap_id);
    SnapRec& r = it->second;
    if (r.aborted) *state = CKPT_SNAP_ABORTED;
    else if (!query_committed(r)) *state = CKPT_SNAP_IN_FLIGHT;
    else *state = (c->holder[r.buf] == r.id) ? CKPT_SNAP_COMMITTED : CKPT_SNAP_SUPERSEDED;
    return CKPT_OK;
}

ckpt_status ckpt_restore(ckpt_ctx* c, uint64_t snap_id, void* stream, uint32_t* bad_chunks, uint32_t cap,
                         uint32_t* n_bad)
{
    if (!c) return CKPT_EINVAL;
    return run_check(c, snap_id, (hipStream_t)stream, true, bad_chunks, cap, n_bad);
}

ckpt_status ckpt_verify(ckpt_ctx* c, uint64_t snap_id, uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad)
{
    if (!c) return CKPT_EINVAL;
    return run_check(c, snap_id, nullptr, false, bad_chunks, cap, n_bad);
}

ckpt_status ckpt_layout(ckpt_ctx* c, uint64_t* frag_off, uint64_t* image_bytes, uint64_t* n_chunks)
{
    if (!c) return CKPT_EINVAL;
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    if (frag_off)
        for (size_t i = 0; i < c->frags.size(); ++i) frag_off[i] = c->frags[i].off;
    if (image_bytes) *image_bytes = c->I;
    if (n_chunks) *n_chunks = c->n_chunks;
    return CKPT_OK;
}

ckpt_status ckpt_chunk_fragments(ckpt_ctx* c, uint64_t k, uint64_t* byte_lo, uint64_t* byte_hi,
                                 uint32_t* frag_first, uint32_t* frag_last)
{
    if (!c) return CKPT_EINVAL;
    if (!c->registered) return fail(c, CKPT_ESTATE, "no tensors registered");
    if (k >= c->n_chunks) return fail(c, CKPT_EINVAL, "chunk %llu out of range", (unsigned long long)k);
    const uint64_t lo = k * c->C, hi = std::min(lo + c->C, c->I);
    const uint32_t n = (uint32_t)c->frags.size();
    // First fragment whose padded span ends past lo; last whose offset is below hi.
    uint32_t l = 0, h = n;
    while (l < h) {
        const uint32_t m = (l + h) / 2;
        const uint64_t end = (m + 1 < n) ? c->frags[m + 1].off : c->I;
        if (end > lo) h = m;
        else l = m + 1;
    }
    const uint32_t a = l;
    l = 0;
    h = n;
    while (l < h) {
        const uint32_t m = (l + h) / 2;
        if (c->frags[m].off >= hi) h = m;
        else l = m + 1;
    }
    const uint32_t b = l ? l - 1 : 0;
    if (byte_lo) *byte_lo = lo;
    if (byte_hi) *byte_hi = hi;
    if (frag_first) *frag_first = a;
    if (frag_last) *frag_last = b;
    return CKPT_OK;
}

ckpt_status ckpt_host_image(ckpt_ctx* c, uint64_t snap_id, void** image, uint64_t* image_bytes, uint64_t** sums)
{
    if (!c) return CKPT_EINVAL;
    auto it = c->recs.find(snap_id);
    if (it == c->recs.end()) return fail(c, CKPT_ERANGE, "snapshot %llu not retained", (unsigned long long)snap_id);
    SnapRec& r = it->second;
    if (!query_committed(r) || c->holder[r.buf] != r.id)
        return fail(c, CKPT_ENOSNAP, "snapshot not committed or superseded");
    if (image) *image = c->h_img[r.buf];
    if (image_bytes) *image_bytes = c->I;
    if (sums) *sums = c->h_sums[r.buf];
    return CKPT_OK;
}

ckpt_status ckpt_last_sums(ckpt_ctx* c, uint64_t* sums, uint64_t n)
{
    if (!c || !sums) return CKPT_EINVAL;
    if (!c->have_last_sums) return fail(c, CKPT_ESTATE, "no restore or verify has run");
    if (n < c->n_chunks) return fail(c, CKPT_EINVAL, "need room for %llu sums", (unsigned long long)c->n_chunks);
    std::memcpy(sums, c->last_sums.data(), c->n_chunks * 8);
    return CKPT_OK;
}

ckpt_status ckpt_envelope(ckpt_ctx* c, uint64_t snap_id, void* out, uint64_t cap, uint64_t* len)
{
    if (!c || !len) return CKPT_EINVAL;
    auto it = c->recs.find(snap_id);
    if (it == c->recs.end()) return fail(c, CKPT_ERANGE, "snapshot %llu not retained", (unsigned long long)snap_id);
    SnapRec& r = it->second;
    if (!query_committed(r) || c->holder[r.buf] != r.id)
        return fail(c, CKPT_ENOSNAP, "snapshot not committed or superseded");
    const std::vector<uint8_t> buf = build_envelope(c, r.step, r.meta, c->h_sums[r.buf]);
    *len = buf.size();
    if (!out || cap < buf.size()) return fail(c, CKPT_EINVAL, "envelope needs %llu bytes", (unsigned long long)buf.size());
    std::memcpy(out, buf.data(), buf.size());
    return CKPT_OK;
}

ckpt_status ckpt_debug_interrupt_next(ckpt_ctx* c, int32_t groups)
{
    if (!c) return CKPT_EINVAL;
    c->interrupt_next = groups < 0 ? -1 : groups;
    return CKPT_OK;
}

ckpt_status ckpt_set_timing(ckpt_ctx* c, int32_t enable)
{
    if (!c) return CKPT_EINVAL;
    c->timing = enable != 0;
    c->timing_span = enable == 2;
    return CKPT_OK;
}

namespace ckpt {
// First pack launch's start to the end of the pack stream's snapshot work:
// every pack launch, the release kernels between them, the chunk-sum reduce
// and its release (an interrupted snapshot has no reduce: to its last pack).
float pack_span(ckpt_ctx* c, const SnapRec& r)
{
    if (r.aborted && !r.per_launch) return -1.f; // its last launch carries no event
    hipEvent_t end = r.aborted ? r.res->k1[c->n_launches - 1] : r.res->t_red;
    if (hipEventSynchronize(end) != hipSuccess) return -1.f;
    return elapsed(r.res->k0[0], end);
}
} // namespace ckpt

ckpt_status ckpt_last_timing(ckpt_ctx* c, uint32_t which, ckpt_timing* out)
{
    if (!c || !out || which > CKPT_OP_PACK) return fail(c, CKPT_EINVAL, "bad timing query");
    if (which == CKPT_OP_PACK) {
        SnapRec* best = nullptr; // newest timed snapshot, committed or not
        for (auto& kv : c->recs)
            if (kv.second.timed && (!best || kv.first > best->id)) best = &kv.second;
        if (!best) return fail(c, CKPT_ESTATE, "no timed snapshot retained");
        RecRes* r = best->res;
        if (!best->per_launch) return fail(c, CKPT_ESTATE, "the newest timed snapshot has no per-launch events");
        HIPCHK(c, hipEventSynchronize(r->k1[c->n_launches - 1])); // packs run in order on one stream
        ckpt_timing t{};
        for (uint64_t j = 0; j < c->n_launches; ++j) t.kernel_ms += elapsed(r->k0[j], r->k1[j]);
        t.kernels = (uint32_t)c->n_launches;
        t.copy_ms = -1.f;
        t.total_ms = -1.f;
        t.kernel_bytes = c->direct ? c->payload : 2 * c->payload; // direct: the sums read the fragments only
        t.span_ms = pack_span(c, *best);
        *out = t;
        return CKPT_OK;
    }
    if (which == CKPT_OP_SNAPSHOT) {
        SnapRec* best = nullptr; // newest timed, committed snapshot
        for (auto& kv : c->recs)
            if (kv.second.timed && !kv.second.aborted && (!best || kv.first > best->id)) best = &kv.second;
        if (!best) return fail(c, CKPT_ESTATE, "no timed snapshot retained");
        ckpt_status st = wait_copies(c, *best);
        if (st) return st;
        RecRes* r = best->res;
        ckpt_timing t{};
        if (best->per_launch) {
            for (uint64_t j = 0; j < c->n_launches; ++j) t.kernel_ms += elapsed(r->k0[j], r->k1[j]);
        } else {
            t.kernel_ms = -1.f;
        }
        t.kernels = (uint32_t)c->n_launches;
        t.copies = (uint32_t)c->n_groups;
        t.span_ms = pack_span(c, *best);
        // DMA span: first image copy start to last image copy end (engine
        // timestamps; in direct mode a group's first piece starts its copies
        // and its last, which signals `copied`, ends them).
        uint64_t t_start = UINT64_MAX, t_end = 0;
        bool ok = true;
        for (uint64_t g = 0; g < c->n_groups; ++g) {
            hsa_amd_profiling_async_copy_time_t ct;
            if (hsa_amd_profiling_get_async_copy_time(r->copied[g], &ct) != HSA_STATUS_SUCCESS) {
                ok = false;
                break;
            }
            if (c->direct && c->piece_first[g + 1] - c->piece_first[g] > 1) {
                hsa_amd_profiling_async_copy_time_t c0;
                if (hsa_amd_profiling_get_async_copy_time(r->piece_done[c->piece_first[g]], &c0) != HSA_STATUS_SUCCESS) {
                    ok = false;
                    break;
                }
                ct.start = c0.start;
            }
            t_start = std::min<uint64_t>(t_start, ct.start);
            t_end = std::max<uint64_t>(t_end, ct.end);
        }
        t.copy_ms = (ok && t_end > t_start) ? (float)((double)(t_end - t_start) * 1e3 / (double)c->ts_freq) : -1.f;
        // Trigger to commit: the first launch's pack, then from its copy's
        // start to the commit -- the last of: the last group copy's end, the
        // sums copy's end and, with pageable images, the last group landing in
        // the image (and the file record).  One clock throughout except the
        // first pack (HIP events); the first copy starts right after it.
        t.total_ms = -1.f;
        hsa_amd_profiling_async_copy_time_t cs;
        if (ok && t_end > t_start && hsa_amd_profiling_get_async_copy_time(r->done, &cs) == HSA_STATUS_SUCCESS) {
            uint64_t commit = std::max<uint64_t>(t_end, cs.end);
            if (best->bounce) commit = std::max<uint64_t>(commit, r->landed_ts.load(std::memory_order_relaxed));
            if (best->file) commit = std::max<uint64_t>(commit, r->recorded_ts.load(std::memory_order_relaxed));
            const float k0 = elapsed(r->k0[0], r->k1[0]);
            if (k0 >= 0.f) t.total_ms = k0 + (float)((double)(commit - t_start) * 1e3 / (double)c->ts_freq);
        }
        t.kernel_bytes = c->direct ? c->payload : 2 * c->payload;
        t.copy_bytes = c->I;
        *out = t;
        return CKPT_OK;
    }
    if (!c->op_timing[which].valid) return fail(c, CKPT_ESTATE, "no timed operation of that kind");
    *out = c->op_timing[which].t;
    return CKPT_OK;
}

ckpt_status ckpt_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                      uint64_t* frag_off, uint64_t* image_bytes, uint64_t* n_chunks)
{
    const uint64_t C = chunk_bytes ? chunk_bytes : kDefaultChunk;
    const uint32_t A = align_bytes ? align_bytes : kDefaultAlign;
    if (!nbytes || n == 0 || !geometry_ok(C, A)) return CKPT_EINVAL;
    Plan p;
    if (!plan(nbytes, n, C, A, &p, false)) return CKPT_EINVAL;
    if (frag_off) std::memcpy(frag_off, p.off.data(), 8ull * n);
    if (image_bytes) *image_bytes = p.I;
    if (n_chunks) *n_chunks = p.n_chunks;
    return CKPT_OK;
}

ckpt_status ckpt_debug_tile_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                                 uint64_t* tile_bytes, uint64_t* n_tiles, uint32_t* tile_first,
                                 uint32_t* tile_last)
{
    const uint64_t C = chunk_bytes ? chunk_bytes : kDefaultChunk;
    const uint32_t A = align_bytes ? align_bytes : kDefaultAlign;
    if (!nbytes || n == 0 || !geometry_ok(C, A)) return CKPT_EINVAL;
    Plan p;
    if (!plan(nbytes, n, C, A, &p, tile_first != nullptr)) return CKPT_EINVAL;
    if (tile_bytes) *tile_bytes = 1ull << p.tile_shift;
    if (n_tiles) *n_tiles = p.n_tiles;
    if (tile_first) std::memcpy(tile_first, p.tile_first.data(), 4 * p.n_tiles);
    if (tile_last && tile_first) std::memcpy(tile_last, p.tile_last.data(), 4 * p.n_tiles);
    return CKPT_OK;
}
ckpt_status ckpt_debug_direct_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                                   uint64_t group_bytes, uint64_t* counts, uint64_t* pieces, uint64_t* gaps,
                                   uint64_t* piece_first, uint64_t* gap_first)
{
    const uint64_t C = chunk_bytes ? chunk_bytes : kDefaultChunk;
    const uint32_t A = align_bytes ? align_bytes : kDefaultAlign;
    if (!nbytes || n == 0 || !counts || !geometry_ok(C, A)) return CKPT_EINVAL;
    Plan p;
    if (!plan(nbytes, n, C, A, &p, false)) return CKPT_EINVAL;
    const uint64_t unit = std::max<uint64_t>(1, (group_bytes ? group_bytes : kDefaultGroup) / C) * C;
    std::vector<Piece> pc, gp;
    std::vector<uint32_t> pf;
    std::vector<uint64_t> p0, g0;
    if (!direct_plan(p.off.data(), nbytes, n, p.I, unit, pc, pf, gp, p0, g0)) return CKPT_EINVAL;
    counts[0] = p0.size() - 1;
    counts[1] = pc.size();
    counts[2] = gp.size();
    if (!pieces) return CKPT_OK;
    if (!gaps || !piece_first || !gap_first) return CKPT_EINVAL;
    for (size_t k = 0; k < pc.size(); ++k) {
        pieces[4 * k] = pf[k];
        pieces[4 * k + 1] = pc[k].src;
        pieces[4 * k + 2] = pc[k].off;
        pieces[4 * k + 3] = pc[k].n;
    }
    for (size_t k = 0; k < gp.size(); ++k) {
        gaps[2 * k] = gp[k].off;
        gaps[2 * k + 1] = gp[k].n;
    }
    std::memcpy(piece_first, p0.data(), 8 * p0.size());
    std::memcpy(gap_first, g0.data(), 8 * g0.size());
    return CKPT_OK;
}

ckpt_status ckpt_latest(ckpt_ctx* c, uint64_t* snap_id, uint64_t* step)
{
    if (!c || !snap_id) return CKPT_EINVAL;
    *snap_id = 0;
    for (auto& kv : c->recs) {
        SnapRec& r = kv.second;
        if (query_committed(r) && c->holder[r.buf] == r.id && r.id > *snap_id) {
            *snap_id = r.id;
            if (step) *step = r.step;
        }
    }
    return CKPT_OK;
}
const char* ckpt_last_error(const ckpt_ctx* c) { return c ? c->err.c_str() : noalloc_error(); }

} // extern "C"
