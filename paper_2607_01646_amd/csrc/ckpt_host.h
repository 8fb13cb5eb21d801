// ckpt_host.h -- internal to libckpt's host side: the context, the records
// of snapshots in flight, the bounce-mode pump, the replication worker and
// the image file, shared by ckpt_runtime.cpp (core path), ckpt_bounce.cpp
// (pageable images behind pinned rings), ckpt_h2h.cpp (replication to a ring
// peer) and ckpt_file.cpp (crash-surviving images).  Not installed.
#pragma once

#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <fcntl.h>
#include <sys/mman.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <deque>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/ckpt.h"
#include "ckpt_internal.h"
#include "ckpt_wire.h"

namespace ckpt {

constexpr uint64_t kDefaultChunk = 64ull << 20;
constexpr uint32_t kDefaultAlign = 256;
constexpr uint64_t kDefaultGroup = 1ull << 30;
constexpr uint64_t kDefaultLaunch = 0; // full-image staging: bytes per pack launch (0 = one group)
constexpr uint32_t kMaxMeta = 1u << 20;
constexpr uint32_t kDefaultGrid = 0x7fffffff; // one workgroup per tile unless capped
constexpr int kMaxEngines = 2;
constexpr uint64_t kVerifySlots = 2; // verify's device ring: two slots of one chunk group each
constexpr uint32_t kDefaultHostThreads = 12; // bounce mode: host copy threads (measured: 8 do not keep up with the link)

struct Frag {
    uint64_t ptr, nbytes, off;
    uint32_t dtype, cls;
};

// Direct D2H: the bytes of one fragment inside one chunk group (the DMA
// engines copy each piece straight from the tensor), or one run of image
// padding inside a group (zeroed on the host before the group's copies).
struct Piece {
    uint64_t src; // device address (pieces); unused for padding
    uint64_t off; // image offset
    uint64_t n;
};
constexpr uint64_t kMaxDirectPieces = 65536;
constexpr uint64_t kDirectRestoreSlots = 4; // restore's device ring in direct mode, in chunk groups

// GPU-side resources of one snapshot record, recycled between snapshots.
struct RecRes {
    std::vector<hipEvent_t> captured;   // per group, on the pack stream
    std::vector<hsa_signal_t> dep;      // per group: set to 0 by the GPU once g is packed
    std::vector<int64_t*> dep_val;      // value addresses of dep
    std::vector<hsa_signal_t> copied;   // per group: the group's image copy finished
    std::vector<hsa_signal_t> flagged;  // per group: the area-done copy after it finished
    std::vector<hsa_signal_t> piece_done; // direct D2H, per piece but each group's last (whose copy
                                          // signals `copied`): the piece's copy finished
    hsa_signal_t dep_sums{0}, done{0};  // sums packed; sums copied (the last copy issued)
    int64_t* dep_sums_val = nullptr;
    uint64_t* h_seq = nullptr;          // pinned, per group: area use number, source of the area-done copy
    unsigned long long* d_sums = nullptr;
    std::vector<hipEvent_t> k0, k1;     // timing: around each pack launch
    hipEvent_t t0 = nullptr;
    hipEvent_t t_red = nullptr;         // timing: after the chunk-sum reduce and its release
    std::atomic<uint32_t> landed{0};    // bounce mode: groups moved from the ring into the image
    std::atomic<bool> failed{false};    // bounce mode: a copy of this record could not be completed
    std::atomic<bool> recorded{false};  // image file: the commit record has been written
    // Timing, in the HSA system timestamp domain (that of the DMA engines'
    // copy timestamps): when the last group landed in the pageable image,
    // and when the commit record was written (0 = not yet).
    std::atomic<uint64_t> landed_ts{0};
    std::atomic<uint64_t> recorded_ts{0};
};

struct SnapRec {
    uint64_t id = 0, step = 0;
    int buf = -1;
    bool bounce = false;    // the image is pageable; groups land through the bounce ring
    bool file = false;      // the image lives in the image file: committed once its record is written
    bool aborted = false;
    bool committed = false; // cached once `done` has reached 0
    bool timed = false;
    bool per_launch = false; // timed with events around every pack launch (else around the first only)
    uint32_t groups_copied = 0;
    std::vector<uint8_t> meta;
    RecRes* res = nullptr;
};

struct OpTiming {
    bool valid = false;
    ckpt_timing t{};
};

// Host threads that copy between host buffers in parallel (bounce mode).
// copy() cuts one copy into parts, queues all but the first, runs the
// first itself, and returns when every part is done; several threads may
// call it at once.
class CopyPool {
public:
    explicit CopyPool(unsigned n) : n_(std::max(1u, n))
    {
        for (unsigned k = 0; k + 1 < n_; ++k) th_.emplace_back([this] { work(); });
    }
    ~CopyPool()
    {
        {
            std::lock_guard<std::mutex> l(m_);
            stop_ = true;
        }
        cv_.notify_all();
        for (auto& t : th_) t.join();
    }
    void copy(uint8_t* dst, const uint8_t* src, uint64_t n)
    {
        const uint64_t min_part = 4ull << 20;
        uint64_t parts = std::min<uint64_t>(n_, std::max<uint64_t>(1, n / min_part));
        if (parts <= 1) {
            std::memcpy(dst, src, n);
            return;
        }
        const uint64_t per = (n / parts + 4095) & ~4095ull;
        Batch b;
        b.left = 0;
        {
            std::lock_guard<std::mutex> l(m_);
            for (uint64_t k = 1; k < parts; ++k) {
                const uint64_t lo = std::min(k * per, n), hi = std::min(lo + per, n);
                if (hi <= lo) continue;
                q_.push_back(Part{dst + lo, src + lo, hi - lo, &b});
                ++b.left;
            }
        }
        cv_.notify_all();
        std::memcpy(dst, src, std::min(per, n));
        std::unique_lock<std::mutex> l(b.m);
        b.cv.wait(l, [&] { return b.left == 0; });
    }

private:
    struct Batch {
        unsigned left;
        std::mutex m;
        std::condition_variable cv;
    };
    struct Part {
        uint8_t* dst;
        const uint8_t* src;
        uint64_t n;
        Batch* b;
    };
    void work()
    {
        for (;;) {
            Part p;
            {
                std::unique_lock<std::mutex> l(m_);
                cv_.wait(l, [&] { return stop_ || !q_.empty(); });
                if (q_.empty()) return;
                p = q_.front();
                q_.pop_front();
            }
            std::memcpy(p.dst, p.src, p.n);
            std::lock_guard<std::mutex> l(p.b->m);
            if (--p.b->left == 0) p.b->cv.notify_all();
        }
    }
    unsigned n_;
    std::mutex m_;
    std::condition_variable cv_;
    std::deque<Part> q_;
    bool stop_ = false;
    std::vector<std::thread> th_;
};

// One group of a snapshot on its way through the bounce ring, or (sums)
// the snapshot's chunk-sum copy, which follows its groups.
struct PumpItem {
    RecRes* res = nullptr;
    uint32_t g = 0;
    bool sums = false;               // the chunk sums: device -> pinned sums array, no ring slot
    uint8_t* image = nullptr;        // destination: pageable host image (group) or pinned sums array
    const uint8_t* staging = nullptr; // source in device memory (null in direct mode: the pieces)
    uint64_t lo = 0;                 // group: image offset of its first byte
    uint64_t n = 0;
    uint64_t* area_done = nullptr;   // group: device counter bumped once the staging area has been read
    const uint64_t* seq = nullptr;   // group: pinned, the value it is set to
    hsa_amd_sdma_engine_id_t engine{};
    uint32_t groups = 0;             // record: the snapshot's group copies
    int buf = 0;                     // host image written
    bool record = false;             // image file: write the snapshot's commit record (no copy)
    uint64_t need_rec = 0;           // sums: records of image buf that must be written before its sums array is reused
    uint64_t snap_id = 0, step = 0;
    std::shared_ptr<const std::vector<uint8_t>> meta;
};

// Image file (ckpt_image_file): the two images, their sums and commit
// records in one shared mapping.  Layout: FileHead at 0, FileRec b at
// kRecOff + 512 * b, then per image its sums, its caller blob area and (2 MiB
// aligned) its bytes.
struct FileHead {
    char magic[8]; // "CKPTFIL1"
    uint32_t version, align;
    uint64_t chunk, image_bytes, n_chunks;
    uint32_t n_frag, pad;
    uint64_t table_sum; // word-sum of the fragment table (offset, bytes, dtype, class per fragment)
    uint64_t image_off[2], sums_off[2], meta_off[2];
    uint64_t file_bytes;
};
struct FileRec {
    uint64_t state;   // 1 = committed; stored last, 0 before the image is rewritten
    uint64_t seq;     // commit number: of two valid records the larger is the newest
    uint64_t snap_id, step, meta_len;
    uint64_t rec_sum; // word-sum of seq, snap_id, step, meta_len, the chunk sums and the zero-padded blob
};
constexpr uint64_t kRecOff = 4096;

// Bounce-mode D2H (one per context).  The issuer takes snapshot groups in
// order, waits for a free ring slot, and starts the DMA staging -> slot
// (after the group's pack, through its dependency signal) followed by the
// staging area's use-counter copy.  The drainer takes them in the same
// order, waits for each DMA, copies slot -> image on the copy pool, frees
// the slot and counts the group as landed.
//
// Every DMA of bounce mode is issued by the issuer, in snapshot and group
// order.  Each engine runs its requests in order, and a request waiting for
// a pack blocks the requests behind it; issuing the chunk-sum copy (which
// waits for the last pack) ahead of group copies that earlier packs depend
// on -- through the staging counters -- would stall the engine for good.
struct Pump {
    std::mutex m;
    std::condition_variable cv;
    std::deque<PumpItem> issue_q;
    std::deque<std::pair<PumpItem, uint64_t>> drain_q;
    std::vector<uint8_t> busy; // per ring slot
    uint64_t next_slot = 0;
    uint64_t rec_pushed[2] = {0, 0}, rec_done[2] = {0, 0}; // image-file commit records per host image
    bool stop = false;
    bool failed = false;
    std::string err;
    std::thread issuer, drainer;
};

// H2H replication (paper Sec. V-B, "Host-to-host"): one job per snapshot,
// handed to the worker when the snapshot is issued.  The worker waits for
// the local commit, sends the replicated chunks with their sums and the
// envelope, and waits for the peer's acknowledgement.
struct RepJob {
    uint64_t id = 0, step = 0;
    int buf = 0;
    RecRes* res = nullptr;
    uint32_t groups_copied = 0;
    bool bounce = false;
    std::vector<uint8_t> meta;
};

enum { REP_PENDING = 0, REP_OK = 1, REP_CORRUPT = 2, REP_FAILED = 3 };

struct RepStatus {
    int state = REP_PENDING;
    std::vector<uint64_t> bad; // sender chunk ids the peer found corrupt
    std::string err;
};

struct Replicator {
    int fd = -1;
    uint64_t first_id = 0; // the first snapshot this peer receives (peers may be added later)
    uint64_t cls_mask = 0;
    std::vector<uint64_t> ids; // replicated chunks, increasing
    uint64_t bytes = 0;        // replica bytes per snapshot
    std::mutex m;
    std::condition_variable cv;
    std::deque<RepJob> q;
    std::map<uint64_t, RepStatus> status;
    bool busy[2] = {false, false}; // a replication still reads host image b
    bool stop = false;
    bool broken = false; // the connection failed: later jobs fail at once
    std::string err;
    int fault_kind = 0;  // debug: 1 = flip one bit of the next stream, 2 = cut the next stream
    uint64_t fault_a = 0, fault_b = 0;
    double last_send_ms = 0, last_ack_ms = 0; // commit -> last byte sent, commit -> acknowledgement
    std::thread worker;
};

// What the last ckpt_restore_from_peer fetched.
struct PeerRestore {
    bool valid = false;
    uint64_t snap_id = 0, step = 0;
    std::vector<uint64_t> ids; // chunks written
    std::vector<uint8_t> envelope;
    double fetch_ms = 0, check_ms = 0;
};

} // namespace ckpt

using namespace ckpt;

struct ckpt_ctx {
    // configuration
    int device = 0;
    uint64_t C = kDefaultChunk;
    uint32_t A = kDefaultAlign;
    uint64_t staging_cap = 0; // 0 = full image
    uint64_t group_cfg = kDefaultGroup;
    bool group_set = false; // group_bytes given explicitly (ring mode: slots of that many bytes)
    uint32_t grid_cap = kDefaultGrid;
    bool timing = false;
    bool timing_span = false; // timing level 2: a snapshot's first launch and pack-stream end only

    // layout
    bool registered = false;
    std::vector<Frag> frags;
    uint64_t I = 0, n_chunks = 0, payload = 0;
    Geometry geo{};
    uint64_t G = 1;        // chunks per group
    uint64_t n_groups = 0; // groups
    uint64_t launch_cfg = kDefaultLaunch;
    uint64_t LG = 1;         // groups per pack launch (1 in ring mode)
    uint64_t n_launches = 0; // pack launches per snapshot
    bool ring = false;
    uint64_t n_slots = 0;  // ring slots of G chunks each (ring mode; direct mode: restore's ring)
    bool direct = false;   // direct D2H: no snapshot staging, the engines copy the fragments
    std::vector<Piece> pieces, gaps;              // direct D2H, by group (CSR below)
    std::vector<uint64_t> piece_first, gap_first; // [n_groups + 1]

    // device memory
    FragDev* d_frags = nullptr;
    uint32_t* d_tile_first = nullptr;
    uint32_t* d_tile_last = nullptr;
    uint8_t* d_staging = nullptr;
    unsigned long long* d_partials = nullptr; // [2][n_tiles * kTileParts] tile partial sums: pack, check
    unsigned long long* d_expected = nullptr;
    unsigned long long* d_recomputed = nullptr;
    uint8_t* d_bad = nullptr;
    uint64_t* d_area_done = nullptr;          // per staging area (direct D2H: per group): number of
                                              // finished copies out of it

    // pinned host memory
    uint8_t* h_img[2] = {nullptr, nullptr};
    uint64_t* h_sums[2] = {nullptr, nullptr};
    uint64_t holder[2] = {0, 0}; // snapshot id whose bytes each image holds (0 = none)
    uint8_t* h_bad = nullptr;
    unsigned long long* h_recomputed = nullptr;

    // HSA agents and DMA engines
    hsa_agent_t gpu_agent{0}, img_agent[2] = {{0}, {0}};
    hsa_amd_sdma_engine_id_t d2h_engine[kMaxEngines];
    int n_d2h_engines = 0;
    uint32_t d2h_engines_cfg = 0; // 0 = all available (up to kMaxEngines)
    bool poison = false;          // fill each staging area with the canary before it is packed again
    hsa_amd_sdma_engine_id_t h2d_engine{};
    uint64_t ts_freq = 1;

    // streams and events
    hipStream_t s_pack = nullptr, s_copy = nullptr;
    bool own_pack = true; // false: s_pack is the caller's side stream (never destroyed here)
    hipEvent_t ev_trigger = nullptr, ev_done = nullptr;
    std::vector<uint64_t> area_seq;     // per staging area: copies issued out of it
    std::vector<hsa_signal_t> area_flag; // per staging area: completion signal of its latest counter copy
                                         // (0 once that copy, and the image copy before it, are done)
    std::vector<hipEvent_t> area_free;  // restore/verify: per staging area
    std::vector<hipEvent_t> ev_loaded;  // restore/verify: per group
    std::vector<RecRes*> free_res;
    std::map<uint64_t, SnapRec> recs;
    uint64_t next_id = 1;
    int32_t interrupt_next = -1;

    // results of the last restore / verify
    bool have_last_sums = false;
    std::vector<uint64_t> last_sums;
    OpTiming op_timing[3];
    std::vector<hipEvent_t> tk0, tk1; // restore timing
    hipEvent_t tt0 = nullptr, tc0 = nullptr, tc1 = nullptr;

    // bounce mode: pageable images behind two pinned rings of chunk groups
    bool bounce = false;
    uint64_t bounce_cfg = 0;
    uint32_t host_threads = kDefaultHostThreads;
    uint64_t n_bslots = 0;            // slots per ring
    uint64_t img_map_bytes = 0;       // mapped length of each pageable image
    uint8_t* h_bout = nullptr;        // device -> host ring
    uint8_t* h_bin = nullptr;         // host -> device ring
    std::vector<hipEvent_t> bin_done; // per host -> device slot: its last copy to the device finished
    CopyPool* pool = nullptr;
    Pump* pump = nullptr;

    // H2H replication to ring peers (k distinct peers, in the order they were added)
    std::vector<Replicator*> reps;

    // the last restore from a ring peer's replica
    PeerRestore peer_restore;

    // image file (crash-surviving images; bounce mode only)
    std::string file_path;
    int file_mode = -1; // -1 none, else CKPT_FILE_CREATE / CKPT_FILE_ADOPT
    int file_fd = -1;
    uint8_t* file_map = nullptr;
    FileHead fhead{};
    uint64_t file_seq = 0; // last commit number written (drainer thread after registration)

    // verify: its own ring of chunk slots and streams
    uint8_t* d_vring = nullptr;
    uint64_t n_vslots = 0;
    hipStream_t s_vcopy = nullptr, s_vker = nullptr;
    hipEvent_t ev_vdone = nullptr, vt0 = nullptr, vc0 = nullptr, vc1 = nullptr;
    std::vector<hipEvent_t> vfree, vloaded, vk0, vk1;

    std::string err;
};

namespace ckpt {

// Record `fmt` as the context's last error and return `code`.
ckpt_status fail(ckpt_ctx* c, ckpt_status code, const char* fmt, ...);
const char* hsa_text(hsa_status_t s);

#define HIPCHK(ctx, expr)                                                                                    \
    do {                                                                                                     \
        hipError_t e_ = (expr);                                                                              \
        if (e_ != hipSuccess)                                                                                \
            return fail((ctx), CKPT_EHIP, "%s failed: %s (%d)", #expr, hipGetErrorString(e_), (int)e_);       \
    } while (0)

#define HSACHK(ctx, expr)                                                                                    \
    do {                                                                                                     \
        hsa_status_t s_ = (expr);                                                                            \
        if (s_ != HSA_STATUS_SUCCESS)                                                                        \
            return fail((ctx), CKPT_EHIP, "%s failed: %s (%d)", #expr, hsa_text(s_), (int)s_);               \
    } while (0)

uint64_t round_up(uint64_t x, uint64_t a);
bool geometry_ok(uint64_t C, uint32_t A);

// Chunk group g: image bytes [group_lo, group_hi), tiles [tiles_lo,
// tiles_hi), its staging area (a ring slot, or its own place in the full
// device image) and where that area starts.
inline uint64_t group_lo(const ckpt_ctx* c, uint64_t g) { return g * c->G * c->C; }
inline uint64_t group_hi(const ckpt_ctx* c, uint64_t g) { return std::min((g + 1) * c->G * c->C, c->I); }
inline uint64_t tiles_lo(const ckpt_ctx* c, uint64_t g) { return group_lo(c, g) >> c->geo.tile_shift; }
inline uint64_t tiles_hi(const ckpt_ctx* c, uint64_t g)
{
    return (group_hi(c, g) + (1ull << c->geo.tile_shift) - 1) >> c->geo.tile_shift;
}
inline uint64_t area_of(const ckpt_ctx* c, uint64_t g) { return c->ring ? g % c->n_slots : g; }
inline uint8_t* staging_of(const ckpt_ctx* c, uint64_t g)
{
    return c->ring ? c->d_staging + (g % c->n_slots) * c->G * c->C : c->d_staging + group_lo(c, g);
}

ckpt_status make_event(ckpt_ctx* c, hipEvent_t* e, bool timed);
// Milliseconds between two recorded timing events (-1 when unavailable).
float elapsed(hipEvent_t a, hipEvent_t b);
// Issue one SDMA copy of n bytes on `engine`, after *dep (when non-null),
// completing into `completion`.
ckpt_status dma(ckpt_ctx* c, void* dst, hsa_agent_t dst_agent, const void* src, hsa_agent_t src_agent, uint64_t n,
                const hsa_signal_t* dep, hsa_signal_t completion, hsa_amd_sdma_engine_id_t engine);
// Text of this thread's last failed ckpt_pack_noalloc ("" if none).
const char* noalloc_error();

// Snapshot records (ckpt_runtime.cpp)
ckpt_status get_res(ckpt_ctx* c, RecRes** out);
// Wait until every snapshot's copies have finished and the library's
// streams are idle.
ckpt_status drain(ckpt_ctx* c);
// The host image the next snapshot would fill (EBUSY while a snapshot is
// uncommitted or that image is being sent to the peer).
ckpt_status pick_target_image(ckpt_ctx* c, int* out);
// Restore (scatter) or verify host image b against h_sums[b] (ckpt_check.cpp): all chunks,
// or only `ids` (increasing).  Fills the bad list like ckpt_restore.  With
// `fill`, each span [lo, hi) of image bytes is first handed to fill, which
// puts them in place (the host -> device work of earlier spans runs
// meanwhile); false from fill ends the operation with EHIP once the work
// already issued has finished (the caller records the error text).
ckpt_status check_image(ckpt_ctx* c, int b, hipStream_t stream, bool scatter, const std::vector<uint64_t>* ids,
                        uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad,
                        const std::function<bool(uint64_t, uint64_t)>& fill = nullptr);
bool res_done(const RecRes* res, uint32_t groups_copied, bool bounce);
void parallel_zero(uint8_t* p, uint64_t n);
std::vector<uint8_t> build_envelope(const ckpt_ctx* c, uint64_t step, const std::vector<uint8_t>& meta,
                                    const uint64_t* sums);

// Issue snapshot r (ckpt_snapshot.cpp): its kernels on the pack stream after
// the work already on `after`, and its copies; groups from n_copy on stay on
// the device, and stop >= 0 marks the snapshot interrupted (never committed).
ckpt_status issue_snapshot(ckpt_ctx* c, SnapRec& r, hipStream_t after, uint64_t n_copy, int32_t stop);

// Direct D2H: zero group g's padding runs in `dst` (host memory holding the
// group's first image byte at dst), then copy its fragment pieces into place
// on `engine`, each after the previous one (the first after first_dep); the
// group's last piece signals res->copied[g].  Returns the pieces issued:
// fewer than the group's means a copy could not be issued (ckpt_snapshot.cpp).
uint64_t issue_pieces(ckpt_ctx* c, RecRes* res, uint64_t g, uint8_t* dst, hsa_agent_t dst_agent,
                      const hsa_signal_t* first_dep, hsa_amd_sdma_engine_id_t engine);

// Bounce mode (ckpt_bounce.cpp)
bool poll_zero(hsa_signal_t sig, int seconds);
void pump_issue(ckpt_ctx* c);
void pump_drain(ckpt_ctx* c);
void stop_pump(ckpt_ctx* c);

// Image file (ckpt_file.cpp)
ckpt_status open_image_file(ckpt_ctx* c);
ckpt_status adopt_image_file(ckpt_ctx* c);
void file_invalidate(ckpt_ctx* c, int b);
void file_commit(ckpt_ctx* c, const PumpItem& it);

// Replication to ring peers (ckpt_h2h.cpp)
constexpr size_t kMaxPeers = 8;
void rep_stop(ckpt_ctx* c);
// Whether a replication still reads host image b.
bool rep_busy(ckpt_ctx* c, int b);

} // namespace ckpt
