/*
 * ckpt.h -- C ABI of libckpt: per-iteration in-memory snapshots of one
 * rank's training state on an MI355X (gfx950), with a per-chunk integrity
 * sum, streamed to pinned host memory off the critical path.
 *
 * What the paper defines (PHOENIX):
 *   - Sec. V-B, "Device-to-host (D2H)": once per iteration the rank's full
 *     state (optimizer shard, parameter shard, metadata envelope with the
 *     step index, parallel configuration and RNG states) is packed into one
 *     contiguous buffer and copied asynchronously to pinned host memory on a
 *     dedicated stream, so that a rank can recover from host memory alone.
 *   - Sec. VI-A: two host buffers alternate roles -- one holds the committed
 *     snapshot of the previous iteration, the other receives the current one
 *     -- so an interrupted offload never destroys the last good snapshot.
 *     The training loop has one synchronization point: a wait right before
 *     the optimizer step, so the protected state is captured before the
 *     optimizer mutates it.
 *   - Sec. V-C, invariant I4 (step atomicity): a partially written snapshot
 *     is never used for recovery.
 *   - Sec. V-C (third recovery stage) and Sec. VI-E: recovery writes the
 *     saved state back into the live tensors.
 *
 * What this library adds: the packed buffer ("image") is cut into
 * fixed-size chunks; each chunk carries the sum of its 8-byte little-endian
 * words modulo 2^64.  The sums are computed on the GPU while packing and
 * re-checked on the GPU when a snapshot is restored or verified.  The wait
 * before the optimizer step is refined to chunk granularity: it covers only
 * the chunks holding the fragments the caller is about to overwrite.
 *
 * Further sections below: crash-surviving image files, host-to-host
 * replication of the optimizer chunks to k ring peers (and the receiving
 * peer), and a replacement rank's restore from a peer's replica.
 *
 * Image layout.  Fragments keep registration order.  off[0] = 0,
 * off[i] = align_up(off[i-1] + nbytes[i-1], align); the image is
 * align_up(off[n-1] + nbytes[n-1], align) bytes; padding bytes are zero and
 * are covered by the sums.  Chunk c is the window
 * [c*chunk_bytes, min((c+1)*chunk_bytes, image_bytes)).
 *
 * Conventions.
 *   - Every call returns ckpt_status: 0 on success, a negative CKPT_E* code
 *     on failure.  Nothing is thrown across the ABI.  The text of the last
 *     error of a context is available from ckpt_last_error().
 *   - "Device pointer" means memory of the context's GPU (hipMalloc,
 *     torch's caching allocator).  Streams are hipStream_t handles passed as
 *     void*; NULL means the device's null stream.
 *   - One host thread drives a context at a time; contexts are independent.
 *   - The library never allocates or frees the caller's tensors.  It owns
 *     its host images (pinned, or pageable behind pinned bounce rings),
 *     device staging, sums, events, streams and threads, and
 *     frees them in ckpt_destroy().
 */
#ifndef CKPT_H
#define CKPT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ckpt_status;

#define CKPT_OK 0
#define CKPT_EINVAL (-1)   /* bad argument (null pointer, size, alignment, range) */
#define CKPT_ESTATE (-2)   /* call not valid in the context's current state */
#define CKPT_ENOMEM (-3)   /* pinned host or device allocation failed */
#define CKPT_EHIP (-4)     /* a HIP runtime call failed; see ckpt_last_error() */
#define CKPT_ECORRUPT (-5) /* one or more chunk sums did not match; list filled */
#define CKPT_ENOSNAP (-6)  /* no committed snapshot (or the requested one is gone) */
#define CKPT_EBUSY (-7)    /* the previous snapshot has not committed (or its replica is being sent) */
#define CKPT_ERANGE (-8)   /* snapshot id unknown or no longer retained */

/* ckpt_wait modes */
#define CKPT_WAIT_CAPTURED 0  /* stream-ordered: the fragments may be overwritten (packed into device
                                 staging; with direct_d2h, summed and copied to the host) */
#define CKPT_WAIT_COMMITTED 1 /* host-blocking: image and sums landed in host memory */
#define CKPT_WAIT_REPLICATED 2 /* host-blocking: the ring peer has checked and committed the replica */

/* ckpt_snapshot_state results */
#define CKPT_SNAP_IN_FLIGHT 0
#define CKPT_SNAP_COMMITTED 1
#define CKPT_SNAP_ABORTED 2    /* interrupted; never committed (invariant I4) */
#define CKPT_SNAP_SUPERSEDED 3 /* committed once, host buffer since reused */

typedef struct ckpt_ctx ckpt_ctx;

typedef struct {
    uint64_t chunk_bytes;          /* chunk size; 0 = 64 MiB.  Multiple of align_bytes. */
    uint32_t align_bytes;          /* fragment alignment in the image; 0 = 256.  Power of two, 16..4096. */
    uint32_t host_buffers;         /* host images; 0 = 2 (ping-pong).  Only 2 is accepted. */
    uint64_t device_staging_bytes; /* 0 = a full-size device image; otherwise a ring of slots of at
                                      most this many bytes in all (at least 2 chunks); each slot
                                      holds one chunk group */
    uint64_t group_bytes;          /* bytes packed per kernel launch and copied per DMA request,
                                      rounded down to whole chunks.  Full-image mode: 0 = 1 GiB.
                                      Ring mode: 0 = a quarter of the ring (at least one chunk);
                                      groups are capped at half the ring, so that it always has
                                      two slots or more */
    int32_t device;                /* HIP device ordinal */
    uint32_t grid_blocks;          /* cap on workgroups per kernel launch; 0 = one per 8 KiB tile */
    uint64_t bounce_bytes;         /* 0 = the two host images are pinned and the DMA engines write
                                      them directly.  > 0 = the images are ordinary pageable memory
                                      (for states larger than the pinned memory the host grants):
                                      DMA goes through two pinned rings of this many bytes each
                                      (one per direction; whole chunk groups, at least two), and
                                      host threads move every landed group between ring and image.
                                      A snapshot then commits when its last group is in the image. */
    uint32_t host_threads;         /* bounce mode: threads moving bytes between rings and images;
                                      0 = 12 */
    void* side_stream;             /* the dedicated stream of Sec. V-B: a hipStream_t of `device`
                                      on which the snapshot's pack, chunk-sum and release kernels
                                      (and the restore's scatter kernels) run.  NULL = the library
                                      creates its own (non-blocking, default priority).  A caller's
                                      stream stays the caller's: it must stay valid until
                                      ckpt_destroy, which does not destroy it, and other work
                                      queued on it delays the pack.  Ignored by ckpt_peer_create. */
    uint64_t pack_launch_bytes;    /* full-image staging: bytes packed per kernel launch, whole chunk
                                      groups (each group still has its own DMA request); 0 = one
                                      group per launch.  Larger launches spend less time between
                                      launches (a snapshot's pack phase is shorter with the GPU
                                      otherwise idle) but slow concurrent training kernels more.
                                      Ring mode packs one group per launch. */
    uint32_t d2h_engines;          /* DMA engines the snapshot's group copies alternate over; 0 = all
                                      the device offers for device-to-host copies (up to 2).  One
                                      engine reaches ~41 GB/s on the MI355X, two the host link's
                                      ~57 GB/s. */
    uint32_t poison;               /* debug check: nonzero = before a staging area is packed again
                                      (after its previous copy has left the device), fill it with the
                                      16-byte canary CKPT_CANARY; with correct ordering the pack
                                      overwrites every byte first, so the canary never reaches a
                                      host image.  Costs one extra write of the staging per snapshot. */
    uint32_t direct_d2h;           /* nonzero = no device staging for snapshots: the DMA engines copy
                                      each fragment from the live tensors straight into its place in
                                      the host image (or the bounce ring), the padding between
                                      fragments is zeroed on the host, and the snapshot's kernels
                                      only compute the chunk sums (reading the fragments once: half
                                      the HBM traffic of pack + copy, and no device image).  The
                                      gate (ckpt_wait CAPTURED) then also waits for the copies of
                                      the chunk groups it covers, so an update issued before the
                                      copies finish waits for the host link.  Restore stages through
                                      a device ring of up to four chunk groups.  Not combinable with
                                      device_staging_bytes or poison; pack_launch_bytes is ignored.
                                      At most 65536 fragment pieces (fragments cut at group
                                      boundaries). */
} ckpt_config;

/* The canary of ckpt_config.poison: these 16 bytes, repeated. */
#define CKPT_CANARY "\xde\xad\xc0\xde\x5a\x5a\xa5\xa5" "CKPTPOIS"

typedef struct {
    const void* dev_ptr; /* device address of the fragment's first byte; any alignment */
    uint64_t nbytes;     /* bytes; 0 is allowed (the fragment takes no image space) */
    uint32_t dtype;      /* caller's tag, stored in the envelope; bytes are never interpreted */
    uint32_t cls;        /* caller's tag (parameter / master / moment ...), stored in the envelope */
} ckpt_tensor;

/* Create a context on cfg->device (NULL cfg = all defaults on device 0).
 * Allocates nothing large until ckpt_register_tensors().
 * Errors: EINVAL (bad config), EHIP. */
ckpt_status ckpt_create(const ckpt_config* cfg, ckpt_ctx** out);

/* Waits for the context's outstanding GPU work, then frees everything it
 * owns.  NULL is accepted. */
ckpt_status ckpt_destroy(ckpt_ctx* ctx);

/* Register the rank's state: n fragments in the order that defines the image
 * layout (Sec. V-B: the state is packed into one contiguous buffer).  The
 * tensors stay owned by the caller and must stay allocated and unmoved while
 * the context lives.  Computes the layout, uploads the fragment and tile
 * tables, allocates device staging and the two host images (pinned, or
 * pageable plus the bounce rings; both pre-faulted).  Callable
 * once per context; a different layout needs a new context.
 * Every non-empty fragment must be device (or managed) memory of the
 * context's GPU and lie inside one allocation; this is checked here, so a
 * wrong pointer or size fails now instead of faulting the first pack.
 * Overlapping fragments are not checked.
 * Errors: ESTATE (already registered), EINVAL (n == 0, a null pointer with
 * nbytes > 0, memory that is not this GPU's device memory, or nbytes running
 * past the end of the fragment's allocation), ENOMEM, EHIP. */
ckpt_status ckpt_register_tensors(ckpt_ctx* ctx, const ckpt_tensor* t, uint32_t n);

/* Start snapshot `step` (Sec. V-B D2H; Sec. VI-A ping-pong).  Stream-ordered
 * after all work already enqueued on after_stream (call it right after the
 * previous optimizer step).  Packs every fragment with its chunk sums into
 * device staging on the library's side stream, then copies the image and the
 * sums chunk group by chunk group into the host image that does not hold
 * the newest committed snapshot (with direct_d2h: sums the fragments in place
 * and copies them straight into that image).  One image always holds the newest
 * committed snapshot and the other receives the one in flight, so a
 * snapshot starts only once the previous one has committed (the caller's
 * wait before the optimizer step, Sec. VI-A, normally ensures that; with
 * CKPT_WAIT_COMMITTED it can wait explicitly).  Returns at once with *snap_id
 * (increasing from 1).  meta (may be NULL when meta_len == 0) is the caller's
 * envelope blob -- parallel configuration, RNG states -- copied before the
 * call returns; at most 1 MiB.
 * Errors: ESTATE (nothing registered), EBUSY (the previous snapshot has
 * not committed yet), EINVAL, EHIP. */
ckpt_status ckpt_snapshot_async(ckpt_ctx* ctx, void* after_stream, uint64_t step, const void* meta,
                                uint32_t meta_len, uint64_t* snap_id);

/* The synchronization point before the optimizer step (Sec. VI-A), refined to
 * chunk granularity.  mode CKPT_WAIT_CAPTURED: makes `stream` wait (no host
 * block) until every chunk holding bytes of fragments [frag_lo, frag_hi) of
 * snapshot snap_id has been packed (with direct_d2h: summed and copied to
 * host memory), so the caller may overwrite those
 * fragments afterwards on `stream` (frag_hi above the fragment count is
 * clamped to it).  mode CKPT_WAIT_COMMITTED: blocks the
 * host until the snapshot's image and sums are in host memory (fragment
 * range ignored).  Errors: ERANGE (unknown or expired snap_id), EINVAL,
 * ESTATE (COMMITTED on an aborted snapshot), EHIP. */
ckpt_status ckpt_wait(ckpt_ctx* ctx, uint64_t snap_id, uint32_t mode, void* stream, uint32_t frag_lo,
                      uint32_t frag_hi);

/* Non-blocking state query: CKPT_SNAP_* in *state. Errors: ERANGE. */
ckpt_status ckpt_snapshot_state(ckpt_ctx* ctx, uint64_t snap_id, uint32_t* state);

/* Recovery (Sec. V-C third stage; Sec. VI-E, local case): first waits for the
 * context's outstanding snapshot work, then copies the committed image
 * snap_id (0 = the newest committed) to the device chunk group by chunk
 * group and scatters every byte back into the registered fragments, while
 * recomputing every chunk sum on the GPU.  The work is ordered after what is
 * already enqueued on `stream`, and `stream` waits for it; the call returns
 * when it is done.  Chunks whose recomputed sum differs from the stored one
 * are listed in increasing order in bad_chunks (up to cap entries, NULL
 * allowed when cap == 0); *n_bad receives the true count.  All bytes are
 * written even when some chunk is bad; the caller then treats the fragments
 * overlapping those chunks as invalid (ckpt_chunk_fragments) and may restore
 * the other buffer instead.
 * Errors: ENOSNAP (nothing committed / snap_id superseded or aborted),
 * ECORRUPT (n_bad > 0), EINVAL, EHIP. */
ckpt_status ckpt_restore(ckpt_ctx* ctx, uint64_t snap_id, void* stream, uint32_t* bad_chunks, uint32_t cap,
                         uint32_t* n_bad);

/* Integrity check of a committed host image without touching the live
 * tensors: copies it to the device and recomputes every chunk sum on the
 * GPU.  Same snap_id, list and error conventions as ckpt_restore. */
ckpt_status ckpt_verify(ckpt_ctx* ctx, uint64_t snap_id, uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad);

/* Layout accessors.  frag_off may be NULL; otherwise it receives n offsets. */
ckpt_status ckpt_layout(ckpt_ctx* ctx, uint64_t* frag_off, uint64_t* image_bytes, uint64_t* n_chunks);

/* Locate: byte range of chunk c and the range [*frag_first, *frag_last] of
 * fragments that may hold its bytes (empty fragments inside it hold none).
 * Errors: EINVAL (c out of range). */
ckpt_status ckpt_chunk_fragments(ckpt_ctx* ctx, uint64_t c, uint64_t* byte_lo, uint64_t* byte_hi,
                                 uint32_t* frag_first, uint32_t* frag_last);

/* Borrowed view of a snapshot's host image and its stored sums (valid
 * until the buffer is reused or the context destroyed).  Writable: tests
 * inject bit flips through it.  Errors: ENOSNAP (not committed), ERANGE. */
ckpt_status ckpt_host_image(ckpt_ctx* ctx, uint64_t snap_id, void** image, uint64_t* image_bytes,
                            uint64_t** sums);

/* The sums recomputed by the last ckpt_restore / ckpt_verify (n_chunks
 * entries). Errors: ESTATE (none yet). */
ckpt_status ckpt_last_sums(ckpt_ctx* ctx, uint64_t* sums, uint64_t n);

/* Serialized metadata envelope of a committed snapshot: magic "CKPTENV1",
 * version, alignment, step, chunk bytes, image bytes, chunk count, fragment
 * count, blob length, fragment table (offset, bytes, dtype, class), chunk
 * sums, caller blob zero-padded to 8 bytes, and the word-sum of all of it;
 * little-endian.  *len receives the size; with cap too small nothing is
 * written and EINVAL is returned.  Errors: ENOSNAP, ERANGE, EINVAL. */
ckpt_status ckpt_envelope(ckpt_ctx* ctx, uint64_t snap_id, void* out, uint64_t cap, uint64_t* len);

/* Fault injection for tests of invariant I4: the next snapshot issues only its
 * first `groups` D2H copies and never commits (it reports ABORTED).  A
 * negative value cancels. */
ckpt_status ckpt_debug_interrupt_next(ckpt_ctx* ctx, int32_t groups);

/* GPU timing of the last operation of each kind, from HIP events recorded
 * on the library's own streams (enable with ckpt_set_timing(ctx, 1) before
 * the operation; timing adds one event pair per kernel launch and per copy
 * request, which lengthens the gaps between a snapshot's pack launches;
 * ckpt_set_timing(ctx, 2) times snapshots with events around the first pack
 * launch and after the pack stream's last kernel only: span_ms, total_ms and
 * copy_ms as at level 1, kernel_ms = -1, and no CKPT_OP_PACK result).
 * which: 0 = snapshot, 1 = restore, 2 = verify, 3 = pack only.
 * Errors: EINVAL (bad `which`), ESTATE (no timed operation of that kind). */
typedef struct {
    float kernel_ms;     /* sum of the tile-kernel launches' durations (pack, scatter or
                            checksum), from events recorded by the dispatch itself; the
                            small per-chunk reduce kernel is not included */
    uint32_t kernels;    /* number of tile-kernel launches (a snapshot's pack launches cover
                            pack_launch_bytes each) */
    uint32_t copies;     /* number of DMA copy requests (image bytes only) */
    float copy_ms;       /* first image copy start to last image copy end */
    float total_ms;      /* operation start (after the trigger) to its last event; for a
                            snapshot: to its commit (image and sums in host memory; with
                            pageable images, the last group landed in the image) */
    uint64_t kernel_bytes; /* algorithmic HBM bytes of the kernels: 2*payload (pack,
                              scatter) or image bytes (verify) */
    uint64_t copy_bytes;   /* image bytes moved over the host link */
    float span_ms;         /* snapshot / pack: the first pack launch's start to the end of the
                              pack stream's work -- every pack launch, the release kernels
                              between them, the chunk-sum reduce and its release, gaps
                              included (an interrupted snapshot: to its last pack launch);
                              -1 for restore and verify */
} ckpt_timing;
#define CKPT_OP_SNAPSHOT 0
#define CKPT_OP_RESTORE 1
#define CKPT_OP_VERIFY 2
#define CKPT_OP_PACK 3 /* the pack launches alone of the newest timed snapshot, committed or not
                          (an interrupted one included); waits for its pack; copies = 0 */
ckpt_status ckpt_set_timing(ckpt_ctx* ctx, int32_t enable);
ckpt_status ckpt_last_timing(ckpt_ctx* ctx, uint32_t which, ckpt_timing* out);

/* Host-only planning (no GPU, no context): the layout that
 * ckpt_register_tensors() would compute for fragments of these sizes with
 * this chunk size and alignment (0 = defaults).  frag_off (n entries) may be
 * NULL.  Lets a caller size pinned and device memory before registering.
 * Errors: EINVAL (bad geometry, n == 0, all fragments empty). */
ckpt_status ckpt_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                      uint64_t* frag_off, uint64_t* image_bytes, uint64_t* n_chunks);

/* Test access to the kernels' tile table (host-only): the tile size and, per
 * tile, the first and last fragment holding one of its bytes.  Call with
 * tile_first == NULL to get *n_tiles first. */
ckpt_status ckpt_debug_tile_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                                 uint64_t* tile_bytes, uint64_t* n_tiles, uint32_t* tile_first,
                                 uint32_t* tile_last);

/* Test access to the copy plan of ckpt_config.direct_d2h (host-only): for
 * fragments of these sizes, chunk size, alignment and group_bytes (0 =
 * defaults), counts[0..2] = chunk groups, fragment pieces, padding runs.
 * With pieces != NULL also fills, in image order: pieces (4 words each:
 * fragment index, byte offset inside the fragment, image offset, bytes),
 * gaps (2 words each: image offset, bytes) and piece_first / gap_first
 * (groups + 1 entries: each group's first piece and run).  Call with
 * pieces == NULL to get the counts first.  Errors: EINVAL. */
ckpt_status ckpt_debug_direct_plan(const uint64_t* nbytes, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                                   uint64_t group_bytes, uint64_t* counts, uint64_t* pieces, uint64_t* gaps,
                                   uint64_t* piece_first, uint64_t* gap_first);

/* ---- Crash-surviving local snapshots (Sec. V-B: the host copy lets a
 * rank come back from its own host memory alone; Sec. V-C: a local reset
 * re-enters as a replacement) ----
 *
 * ckpt_image_file, before ckpt_register_tensors and only in bounce mode
 * (cfg.bounce_bytes > 0): keep the two host images, their chunk sums and a
 * commit record for each in the file at path, mapped shared, so that they
 * outlive the process (under /dev/shm: until the host reboots).  A record is
 * written after the snapshot's last byte and its sums have landed, and is
 * cleared before its image is rewritten, so a process that dies at any point
 * leaves its newest committed snapshot restorable (invariant I4).
 *   CKPT_FILE_CREATE: create or truncate the file at registration.
 *   CKPT_FILE_ADOPT: open a file written by a context of the same layout
 *     (same fragment sizes, dtypes and classes in the same order, chunk size
 *     and alignment); its newest valid record becomes this context's
 *     committed snapshot (ckpt_latest names it; ckpt_restore restores it,
 *     re-checking every chunk sum).
 * File format (little-endian): a head at offset 0 {char magic[8] = "CKPTFIL1";
 * u32 version = 1; u32 align; u64 chunk_bytes; u64 image_bytes; u64 n_chunks;
 * u32 n_frag; u32 0; u64 table_sum = sum over fragments of off + nbytes +
 * (dtype | cls << 32) mod 2^64; u64 image_off[2]; u64 sums_off[2];
 * u64 meta_off[2]; u64 file_bytes}; at 4096 + 512 * b the record of image b
 * {u64 state (1 = committed); u64 seq (of two valid records the larger is the
 * newest); u64 snap_id; u64 step; u64 meta_len; u64 rec_sum = seq + snap_id +
 * step + meta_len + the word-sum of the image's n_chunks sums and of its blob
 * zero-padded to 8 bytes, mod 2^64}; image b's sums at sums_off[b], its blob
 * at meta_off[b] and its bytes at image_off[b].
 * Errors: EINVAL (bounce mode off, bad mode), ESTATE (already registered);
 * at registration: EINVAL (the file's layout differs), EHIP / ENOMEM (file
 * errors). */
#define CKPT_FILE_CREATE 0
#define CKPT_FILE_ADOPT 1
ckpt_status ckpt_image_file(ckpt_ctx* ctx, const char* path, uint32_t mode);

/* The newest committed snapshot still held (0 if none) and its step. */
ckpt_status ckpt_latest(ckpt_ctx* ctx, uint64_t* snap_id, uint64_t* step);

/* ---- Host-to-host replication to ring peers (Sec. V-B "Host-to-host";
 * Sec. VI-A: the wait before the optimizer step covers the peer replica;
 * Sec. V-C: k distinct peers tolerate k concurrent failures) ----
 *
 * ckpt_replicate_to: connect to a peer (ckpt_peer_*) listening at host:port
 * (dotted IPv4) and start a worker for it.  From then on every snapshot,
 * once committed locally, is sent to it: the chunks holding a byte of a
 * fragment whose class tag k has bit k set in cls_mask (the optimizer-state
 * classes, in the paper), their stored sums and the snapshot's envelope.
 * The peer re-checks every chunk sum on its GPU, commits its own ping-pong
 * copy and answers.  Call it again (after registration, up to 8 times, with
 * the same cls_mask, while no replication is in progress) to add further
 * peers; each receives the snapshots issued after it was added, and the
 * streams to the k peers run at the same time.
 * ckpt_wait(CKPT_WAIT_REPLICATED) blocks until every peer has answered (a
 * transfer may take as long as it needs while bytes flow; one that makes no
 * progress for 30 s, or whose local snapshot does not commit within 120 s,
 * fails with EHIP): OK
 * when all committed the replica; ECORRUPT when a peer found bad chunks (that
 * peer keeps its previous replica; ckpt_replica_result lists them); EHIP
 * when a connection failed (the failure wins over corruption).  While a
 * snapshot's replica is being sent its host image is held: a snapshot that
 * would reuse it returns EBUSY.
 * Errors: EINVAL (bad address, mask selecting nothing, a mask other than
 * the first peer's, more than 8 peers), ESTATE, EBUSY (adding a peer while
 * a replication is in progress), EHIP. */
ckpt_status ckpt_replicate_to(ckpt_ctx* ctx, const char* host, uint32_t port, uint64_t cls_mask);

/* Drop peer `peer` (0-based; later peers move down one place): its worker
 * stops, a replica it is sending fails, its connection closes.  For ring
 * repair after the peer's node is lost (Sec. V-C): drop it, then add the
 * replacement's peer with ckpt_replicate_to.  Snapshots sent only to dropped
 * peers count as not replicated (ERANGE from ckpt_wait(REPLICATED)).
 * Errors: ESTATE (no such peer). */
ckpt_status ckpt_replicate_remove(ckpt_ctx* ctx, uint32_t peer);

/* The replicated chunk ids (increasing; up to cap written) and their total
 * bytes (the same for every peer).  Errors: ESTATE (no peer). */
ckpt_status ckpt_replica_chunks(ckpt_ctx* ctx, uint64_t* ids, uint64_t cap, uint64_t* n, uint64_t* replica_bytes);

/* Non-blocking replication state of a snapshot over all its peers: *state =
 * 0 while any peer is pending, else 3 when any failed (not sent, or no
 * answer), else 2 when any found corrupt chunks (the union of their ids in
 * bad, up to cap; *n_bad the count), else 1 (every peer committed it).
 * Errors: ERANGE (not replicated: interrupted, or older than 64 snapshots). */
ckpt_status ckpt_replica_result(ckpt_ctx* ctx, uint64_t snap_id, int32_t* state, uint64_t* bad, uint32_t cap,
                                uint32_t* n_bad);

/* The same for peer `peer` alone (0-based, in the order the peers were added).
 * Errors: ESTATE (no such peer), ERANGE. */
ckpt_status ckpt_replica_peer_result(ckpt_ctx* ctx, uint32_t peer, uint64_t snap_id, int32_t* state, uint64_t* bad,
                                     uint32_t cap, uint32_t* n_bad);

/* Number of replication peers. */
ckpt_status ckpt_replica_peers(ckpt_ctx* ctx, uint32_t* n);

/* Host wall time of the last replication, from the local commit being
 * observed: to the last byte sent, and to the answer (the slowest peer). */
ckpt_status ckpt_replica_timing(ckpt_ctx* ctx, double* send_ms, double* ack_ms);

/* Fault injection for tests: kind 1 flips bit (b & 7) of replica byte a in
 * the next stream to peer `peer` (the local image is untouched); kind 2
 * closes that peer's connection after a replica bytes of its next stream;
 * 0 cancels.  ckpt_debug_h2h_fault acts on the first peer. */
ckpt_status ckpt_debug_h2h_fault_peer(ckpt_ctx* ctx, uint32_t peer, int32_t kind, uint64_t a, uint64_t b);
ckpt_status ckpt_debug_h2h_fault(ckpt_ctx* ctx, int32_t kind, uint64_t a, uint64_t b);

/* The receiving side: a ring peer holding its predecessor's replicas.  It
 * listens on 127.0.0.1:port (0 = any free port; see ckpt_peer_port), takes
 * one sender at a time, receives each snapshot's replica into the pinned
 * buffer that does not hold its newest committed replica, re-checks every
 * chunk sum on cfg->device with the library's checksum kernel (host->device
 * copies through a two-slot device ring, cfg->group_bytes per slot, each
 * slot checked while the next one is received), and
 * commits the buffer only when every sum matches (Sec. VI-A: the buffer
 * received from the ring predecessor alternates like the local one).  A
 * stream cut mid-snapshot leaves the previous replica in place; the peer
 * then waits for the next connection.  A replacement rank's fetch
 * (ckpt_restore_from_peer) is answered on a connection of its own, also
 * between two snapshots of a connected sender; a second sender is refused
 * while one is connected. */
typedef struct ckpt_peer ckpt_peer;
ckpt_status ckpt_peer_create(const ckpt_config* cfg, uint32_t port, ckpt_peer** out);
ckpt_status ckpt_peer_port(const ckpt_peer* peer, uint32_t* port);
/* Stops the receiver (closing any connection) and frees everything. */
ckpt_status ckpt_peer_destroy(ckpt_peer* peer);
/* Wait (up to timeout_ms) until snapshot snap_id of the sender has been
 * handled: *result = CKPT_OK (committed), CKPT_ECORRUPT (rejected),
 * CKPT_EHIP (the stream broke), CKPT_EINVAL (a chunk list out of order or
 * out of the image, a replica size that does not match it, or a geometry
 * other than the first snapshot's) or CKPT_ENOMEM (no room for the
 * replica buffers).  The header is checked before anything is allocated
 * for it (chunk size a multiple of 256, image at most 2^48 bytes, m chunks
 * within the image, replica size within those m chunks) and the chunk ids
 * as they arrive; a malformed header ends the connection with no result.
 * Either way the peer drops that sender and keeps its newest committed
 * replica.  Errors: ERANGE on timeout. */
ckpt_status ckpt_peer_wait(ckpt_peer* peer, uint64_t snap_id, int32_t timeout_ms, int32_t* result);
/* Borrowed view of the newest committed replica: sender's snapshot id and
 * step, the replica bytes (chunks back to back), the sender's chunk ids and
 * sums, and the envelope.  Valid until the peer starts receiving the
 * snapshot after the next committed one (that one reuses this buffer).
 * Errors: ENOSNAP (none committed). */
ckpt_status ckpt_peer_replica(ckpt_peer* peer, uint64_t* snap_id, uint64_t* step, const void** data,
                              uint64_t* bytes, const uint64_t** chunk_ids, const uint64_t** sums, uint64_t* n_chunks,
                              const void** envelope, uint64_t* envelope_len);
/* The sender's chunk ids that failed the check in the last rejected
 * snapshot (up to cap; *n the count). */
ckpt_status ckpt_peer_last_bad(ckpt_peer* peer, uint64_t* bad, uint32_t cap, uint32_t* n);
/* Host wall time of the last replica (ms): from its header to the last byte
 * received (recv_ms), and from there to the end of the GPU check (check_ms;
 * the check of each unit overlaps the receipt of the next). */
ckpt_status ckpt_peer_timing(ckpt_peer* peer, double* recv_ms, double* check_ms);
const char* ckpt_peer_last_error(const ckpt_peer* peer);

/* ---- A replacement rank's optimizer state from its ring peer (Sec. V-C,
 * third recovery stage: the optimizer shard comes back from the replica the
 * peer kept in memory; the parameter shard comes from the ranks that share
 * the failed rank's partition, which this library does not do) ----
 *
 * ckpt_restore_from_peer: ctx belongs to the replacement and is registered
 * with the failed rank's layout (the same fragment sizes, dtypes and
 * classes in the same order, chunk size and alignment).  Connects to the
 * peer at host:port (dotted IPv4; ckpt_peer_*), fetches the newest replica
 * the peer has committed, and checks that the replica's envelope describes
 * this layout byte for byte (rebuilt from the context's fragment table with
 * the envelope's step, sums and blob) and that its chunk sums agree with
 * the envelope.  The replicated chunks are received into the host image
 * that the next snapshot would fill, at their image offsets; a snapshot
 * held there is no longer restorable (ckpt_snapshot_state: SUPERSEDED).
 * As ckpt_restore but for those chunks only, each run of chunks as soon as
 * it has arrived: every fragment byte they hold is written back to the
 * registered tensors (parameter bytes sharing a chunk with optimizer bytes
 * included), each chunk's sum is recomputed on the GPU and compared with the
 * sum stored at pack time, and `stream` waits for the writes.  Fragment
 * bytes outside the replicated chunks are left as they are.  *snap_id / *step (may be NULL): the failed rank's snapshot id
 * and step.  Blocks until done (the transfer fails with EHIP once it makes no
 * progress for 30 s).  Does not change ckpt_last_sums or the restore timing.
 * Errors: EINVAL (bad argument, or the reply does not match this layout:
 * nothing written), ESTATE (not registered), EBUSY (a snapshot has not
 * committed, or the target image is being sent to this context's own peer),
 * ENOSNAP (the peer holds no committed replica), EHIP (connection or HIP
 * failure; a transfer that breaks midway leaves the chunks before the break
 * written), ECORRUPT (chunks failed their sum: their ids in bad_chunks up to
 * cap, *n_bad the count; every replicated chunk was still written). */
ckpt_status ckpt_restore_from_peer(ckpt_ctx* ctx, const char* host, uint32_t port, void* stream, uint64_t* snap_id,
                                   uint64_t* step, uint32_t* bad_chunks, uint32_t cap, uint32_t* n_bad);

/* What the last ckpt_restore_from_peer received (each output may be NULL):
 * the chunk ids it wrote (increasing; up to cap; *n_ids the count), the
 * replica's envelope (the format of ckpt_envelope, including the caller
 * blob of the failed rank's snapshot; nothing is written and EINVAL is
 * returned when env_cap is smaller than *env_len), and host wall times in
 * ms: connect to the last replica byte received (fetch_ms), and from there
 * to the end of the restore and check (check_ms).  Errors: ESTATE (none
 * yet), EINVAL. */
ckpt_status ckpt_peer_restore_info(ckpt_ctx* ctx, uint64_t* ids, uint64_t cap, uint64_t* n_ids, void* envelope,
                                   uint64_t env_cap, uint64_t* env_len, double* fetch_ms, double* check_ms);

/* ---- Allocation-free pack, for callers that cannot allocate (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc) ----
 *
 * ckpt_pack_noalloc: the pack and per-chunk sums of ckpt_snapshot_async --
 * the same kernels, layout and sums -- into a device image the caller owns,
 * with no context and no allocation: no hipMalloc, hipFree, pinned or
 * pageable allocation of any kind.  Nothing is copied to the host.
 *   t, n          fragment descriptors in layout order (host array; read
 *                 before the call returns); each non-empty one must be
 *                 memory of `device` inside one allocation.
 *   chunk_bytes, align_bytes   as in ckpt_config (0 = 64 MiB / 256).
 *   device        HIP device ordinal; the caller's current device is
 *                 restored before the call returns.
 *   image         device memory of `device`, 16-byte aligned, image_cap
 *                 bytes; receives image bytes [0, *image_bytes) (fragment
 *                 bytes and zero padding); bytes past that are not touched.
 *   sums          device memory of `device`, 8-byte aligned, sums_cap
 *                 entries; receives the *n_chunks chunk sums.
 *   stream        hipStream_t of `device` (NULL = null stream); the work is
 *                 enqueued on it and the call returns without waiting.
 *   image_bytes, n_chunks      host outputs (may be NULL), also set when the
 *                 capacities are too small.
 * The library keeps the fragment table, the tile table and the partial sums
 * in one fixed 7 MiB device array per GPU (held until the process ends).
 * Limits: at most 65536 fragments, chunks of at most 1 GiB (at 8 KiB tiles);
 * the image may be any size (it is packed in groups of at most 1 GiB that
 * reuse the array).  Every call on a GPU uses that GPU's array: calls whose
 * work overlaps on one GPU (different streams, not ordered by events) race
 * and give wrong sums; order them, e.g. one stream.
 * Errors: EINVAL (null pointer, n == 0 or above 65536, bad geometry, chunk
 * above the limit, image_cap / sums_cap too small, misaligned image or sums,
 * or memory that is not `device`'s or runs past its allocation; nothing is
 * enqueued), EHIP (a launch failed).  Text: ckpt_last_error(NULL) on the
 * same thread. */
ckpt_status ckpt_pack_noalloc(const ckpt_tensor* t, uint32_t n, uint64_t chunk_bytes, uint32_t align_bytes,
                              int32_t device, void* image, uint64_t image_cap, uint64_t* sums, uint64_t sums_cap,
                              void* stream, uint64_t* image_bytes, uint64_t* n_chunks);

/* Text of the context's last error ("" if none).  Valid until the next call.
 * With NULL: the text of this thread's last failed ckpt_pack_noalloc. */
const char* ckpt_last_error(const ckpt_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* CKPT_H */
