// ckpt_file.cpp -- crash-surviving local snapshots: the two host images,
// their chunk sums and commit records in one shared file mapping (format in
// include/ckpt.h, ckpt_image_file).  Records are cleared before an image is
// rewritten and written last after a snapshot commits (by the bounce pump's
// drainer, in snapshot order), so the newest committed snapshot stays
// restorable by a later process.
#include "ckpt_host.h"

namespace ckpt {

// ---- image file (ckpt_image_file) ----

uint64_t word_sum(const uint8_t* p, uint64_t n) // n a multiple of 8
{
    uint64_t s = 0;
    for (uint64_t k = 0; k < n; k += 8) {
        uint64_t w;
        std::memcpy(&w, p + k, 8);
        s += w;
    }
    return s;
}

FileRec* file_rec(const ckpt_ctx* c, int b) { return (FileRec*)(c->file_map + kRecOff + 512 * b); }

void file_layout(const ckpt_ctx* c, FileHead* h)
{
    std::memset(h, 0, sizeof *h);
    std::memcpy(h->magic, "CKPTFIL1", 8);
    h->version = 1;
    h->align = c->A;
    h->chunk = c->C;
    h->image_bytes = c->I;
    h->n_chunks = c->n_chunks;
    h->n_frag = (uint32_t)c->frags.size();
    for (const Frag& f : c->frags) h->table_sum += f.off + f.nbytes + (f.dtype | ((uint64_t)f.cls << 32));
    uint64_t o = kRecOff + 1024;
    for (int b = 0; b < 2; ++b) {
        h->sums_off[b] = round_up(o, 4096);
        h->meta_off[b] = h->sums_off[b] + round_up(8 * c->n_chunks, 4096);
        o = h->meta_off[b] + kMaxMeta;
    }
    for (int b = 0; b < 2; ++b) {
        h->image_off[b] = round_up(o, 2ull << 20);
        o = h->image_off[b] + round_up(c->I, 2ull << 20);
    }
    h->file_bytes = o;
}

uint64_t rec_checksum(const ckpt_ctx* c, const FileRec& r, int b)
{
    return r.seq + r.snap_id + r.step + r.meta_len + word_sum(c->file_map + c->fhead.sums_off[b], 8 * c->n_chunks) +
           word_sum(c->file_map + c->fhead.meta_off[b], round_up(r.meta_len, 8));
}

bool rec_valid(const ckpt_ctx* c, int b)
{
    const FileRec* r = file_rec(c, b);
    return __atomic_load_n(&r->state, __ATOMIC_ACQUIRE) == 1 && r->meta_len <= kMaxMeta &&
           rec_checksum(c, *r, b) == r->rec_sum;
}

// Before image b is rewritten its record stops naming a snapshot.
void file_invalidate(ckpt_ctx* c, int b) { __atomic_store_n(&file_rec(c, b)->state, (uint64_t)0, __ATOMIC_RELEASE); }

// After the snapshot's last byte and its sums have landed: sums, caller
// blob, then the record, its state last.
void file_commit(ckpt_ctx* c, const PumpItem& it)
{
    const int b = it.buf;
    std::memcpy(c->file_map + c->fhead.sums_off[b], c->h_sums[b], 8 * c->n_chunks);
    const uint64_t len = it.meta ? it.meta->size() : 0;
    uint8_t* meta = c->file_map + c->fhead.meta_off[b];
    if (len) std::memcpy(meta, it.meta->data(), len);
    std::memset(meta + len, 0, round_up(len, 8) - len);
    FileRec* r = file_rec(c, b);
    r->seq = ++c->file_seq;
    r->snap_id = it.snap_id;
    r->step = it.step;
    r->meta_len = len;
    r->rec_sum = rec_checksum(c, *r, b);
    __atomic_store_n(&r->state, (uint64_t)1, __ATOMIC_RELEASE);
}

// Map the image file at registration (bounce mode): create it, or check an
// existing one against this context's layout.
ckpt_status open_image_file(ckpt_ctx* c)
{
    file_layout(c, &c->fhead);
    const bool create = c->file_mode == CKPT_FILE_CREATE;
    c->file_fd = ::open(c->file_path.c_str(), create ? (O_RDWR | O_CREAT | O_TRUNC) : O_RDWR, 0600);
    if (c->file_fd < 0) return fail(c, CKPT_EHIP, "open %s: %s", c->file_path.c_str(), strerror(errno));
    if (create) {
        // Reserve the space now: a sparse file on a full tmpfs would fault
        // (SIGBUS) on first write instead of failing here.
        const int e = ::posix_fallocate(c->file_fd, 0, (off_t)c->fhead.file_bytes);
        if (e != 0) return fail(c, CKPT_ENOMEM, "reserving %llu bytes for %s: %s",
                                (unsigned long long)c->fhead.file_bytes, c->file_path.c_str(), strerror(e));
    } else {
        struct stat st;
        if (::fstat(c->file_fd, &st) != 0 || (uint64_t)st.st_size != c->fhead.file_bytes)
            return fail(c, CKPT_EINVAL, "%s does not hold images of this layout", c->file_path.c_str());
    }
    void* m = ::mmap(nullptr, c->fhead.file_bytes, PROT_READ | PROT_WRITE, MAP_SHARED, c->file_fd, 0);
    if (m == MAP_FAILED) return fail(c, CKPT_ENOMEM, "mmap %s: %s", c->file_path.c_str(), strerror(errno));
    c->file_map = (uint8_t*)m;
    (void)madvise(m, c->fhead.file_bytes, MADV_HUGEPAGE);
    if (create) {
        std::memcpy(c->file_map, &c->fhead, sizeof c->fhead);
        std::memset(c->file_map + kRecOff, 0, 1024);
    } else if (std::memcmp(c->file_map, &c->fhead, sizeof c->fhead) != 0) {
        return fail(c, CKPT_EINVAL, "%s holds images of another layout (fragments, chunk or alignment differ)",
                    c->file_path.c_str());
    }
    for (int b = 0; b < 2; ++b) {
        c->h_img[b] = c->file_map + c->fhead.image_off[b];
        if (create) parallel_zero(c->h_img[b], c->I); // fault the pages in now
    }
    return CKPT_OK;
}

// After registration: the image file's newest valid record becomes this
// context's committed snapshot.
ckpt_status adopt_image_file(ckpt_ctx* c)
{
    int best = -1;
    for (int b = 0; b < 2; ++b) {
        if (!rec_valid(c, b)) continue;
        c->file_seq = std::max(c->file_seq, file_rec(c, b)->seq);
        if (best < 0 || file_rec(c, b)->seq > file_rec(c, best)->seq) best = b;
    }
    if (best >= 0) {
        RecRes* res = nullptr;
        ckpt_status st = get_res(c, &res);
        if (st) return st;
        const FileRec* fr = file_rec(c, best);
        const uint64_t id = c->next_id++;
        SnapRec& r = c->recs[id];
        r.id = id;
        r.step = fr->step;
        r.buf = best;
        r.res = res;
        r.bounce = true;
        r.file = true;
        res->recorded.store(true, std::memory_order_relaxed);
        r.committed = true; // nothing in flight: its signals are all 0
        const uint8_t* meta = c->file_map + c->fhead.meta_off[best];
        r.meta.assign(meta, meta + fr->meta_len);
        std::memcpy(c->h_sums[best], c->file_map + c->fhead.sums_off[best], 8 * c->n_chunks);
        c->holder[best] = id;
    }
    return CKPT_OK;
}

} // namespace ckpt

extern "C" {

ckpt_status ckpt_image_file(ckpt_ctx* c, const char* path, uint32_t mode)
{
    if (!c || !path || !*path || mode > CKPT_FILE_ADOPT) return fail(c, CKPT_EINVAL, "bad image file arguments");
    if (c->registered) return fail(c, CKPT_ESTATE, "tensors already registered");
    if (!c->bounce_cfg) return fail(c, CKPT_EINVAL, "an image file needs bounce mode (bounce_bytes > 0)");
    c->file_path = path;
    c->file_mode = (int)mode;
    return CKPT_OK;
}

} // extern "C"
