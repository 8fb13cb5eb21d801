/*
 * ckpt_oracle.c -- plain CPU oracle for the in-memory snapshot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test suite, the package's smoke check and the
 * benchmark's CPU-baseline leg do.  It shares no code, header, table or
 * constant generator with the GPU path.
 *
 * What it computes.  PHOENIX (Sec. V-B, "Device-to-host (D2H)") packs one
 * rank's full training state -- optimizer shard, parameter shard and a
 * metadata envelope holding the step index, parallel configuration and RNG
 * states -- into one contiguous buffer and copies it to pinned host memory.
 * Recovery writes that buffer back into the live tensors (Sec. V-C, third
 * recovery stage; Sec. VI-E).  The paper fixes neither the buffer layout nor
 * any integrity check; this oracle follows the readings written below, which
 * are the definitions the GPU path must reproduce byte for byte:
 *
 *   1. Layout.  Fragments keep registration order.  off[0] = 0 and
 *      off[i] = align_up(off[i-1] + n[i-1], A).  The image is
 *      I = align_up(off[last] + n[last], A) bytes (0 when there are no
 *      fragments).  Chunk c is the byte window [c*C, min((c+1)*C, I));
 *      C must be a positive multiple of A, and A a positive multiple of 8.
 *   2. Pack.  image = zeros(I); image[off[i] .. off[i]+n[i]) = bytes of
 *      fragment i.  Padding stays zero.
 *   3. Checksum.  sum[c] = sum over the chunk's 8-byte words, each read as a
 *      little-endian unsigned 64-bit integer, modulo 2^64, starting at 0,
 *      padding included.  (Plain two's-complement wrap-around: not a
 *      ones'-complement, Fletcher or Adler sum.)
 *   4. Restore.  fragment i = image[off[i] .. off[i]+n[i]).  Verify
 *      recomputes 3 and reports every chunk whose sum differs from the
 *      stored one.
 *   5. Locate.  A bad chunk is reported with its byte range and every
 *      non-empty fragment whose byte range overlaps it.
 *
 * Every function works on a window [lo, hi) of the image so that a test can
 * check single chunks of a shard too large to pack whole on the host; the
 * window form is the same definition restricted to those bytes.
 *
 * The code is deliberately plain: byte loops, no SIMD, no threads, no
 * blocking.  It is meant to be read against the definitions above.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL (-1)

static uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

/* Definition 1 (layout).  Writes off[0..n), *image_bytes and *n_chunks. */
int oracle_layout(uint32_t n, const uint64_t *nbytes, uint64_t align, uint64_t chunk,
                  uint64_t *off, uint64_t *image_bytes, uint64_t *n_chunks)
{
    if (align == 0 || align % 8 != 0 || chunk == 0 || chunk % align != 0)
        return ORACLE_EINVAL;
    uint64_t end = 0; /* one past the last byte of fragment i-1 */
    for (uint32_t i = 0; i < n; ++i) {
        off[i] = (i == 0) ? 0 : round_up(end, align);
        end = off[i] + nbytes[i];
    }
    uint64_t I = (n == 0) ? 0 : round_up(end, align);
    *image_bytes = I;
    *n_chunks = (I + chunk - 1) / chunk;
    return ORACLE_OK;
}

/* Definition 2 (pack), restricted to image bytes [lo, hi): out[0 .. hi-lo). */
int oracle_pack_window(uint32_t n, const uint8_t *const *frag, const uint64_t *nbytes,
                       const uint64_t *off, uint64_t lo, uint64_t hi, uint8_t *out)
{
    if (hi < lo) return ORACLE_EINVAL;
    for (uint64_t x = 0; x < hi - lo; ++x) out[x] = 0;
    for (uint32_t i = 0; i < n; ++i) {
        uint64_t a = off[i], b = off[i] + nbytes[i]; /* fragment i's bytes in the image */
        if (a < lo) a = lo;
        if (b > hi) b = hi;
        for (uint64_t x = a; x < b; ++x)
            out[x - lo] = frag[i][x - off[i]];
    }
    return ORACLE_OK;
}

/* One little-endian 64-bit word from 8 bytes, independent of the host's order. */
static uint64_t le_word(const uint8_t *p)
{
    uint64_t w = 0;
    for (int k = 0; k < 8; ++k) w |= (uint64_t)p[k] << (8 * k);
    return w;
}

/* Definition 3 (checksum) for the chunks inside image bytes [lo, hi).
 * lo must start a chunk; hi must end one (a multiple of chunk, or the image
 * end, which is a multiple of the alignment and so of 8).  sums[k] belongs to
 * chunk lo/chunk + k. */
int oracle_chunk_sums(const uint8_t *window, uint64_t lo, uint64_t hi, uint64_t chunk,
                      uint64_t *sums)
{
    if (chunk == 0 || lo % chunk != 0 || hi < lo || (hi - lo) % 8 != 0) return ORACLE_EINVAL;
    uint64_t k = 0;
    for (uint64_t c0 = lo; c0 < hi; c0 += chunk, ++k) {
        uint64_t c1 = (c0 + chunk < hi) ? c0 + chunk : hi;
        uint64_t s = 0;
        for (uint64_t x = c0; x < c1; x += 8)
            s += le_word(window + (x - lo)); /* unsigned: wraps modulo 2^64 */
        sums[k] = s;
    }
    return ORACLE_OK;
}

/* Definition 4 (restore), restricted to image bytes [lo, hi): copies the
 * window's bytes back into the fragments that overlap it. */
int oracle_restore_window(const uint8_t *window, uint64_t lo, uint64_t hi, uint32_t n,
                          const uint64_t *off, const uint64_t *nbytes, uint8_t *const *frag)
{
    if (hi < lo) return ORACLE_EINVAL;
    for (uint32_t i = 0; i < n; ++i) {
        uint64_t a = off[i], b = off[i] + nbytes[i];
        if (a < lo) a = lo;
        if (b > hi) b = hi;
        for (uint64_t x = a; x < b; ++x)
            frag[i][x - off[i]] = window[x - lo];
    }
    return ORACLE_OK;
}

/* Definition 4 (verify) over the chunks of [lo, hi): recompute each sum and
 * list, in increasing order, the chunks whose stored sum differs.  Writes at
 * most cap indices; returns the true count (or ORACLE_EINVAL). */
int64_t oracle_verify(const uint8_t *window, uint64_t lo, uint64_t hi, uint64_t chunk,
                      const uint64_t *stored, uint32_t *bad, uint32_t cap)
{
    if (chunk == 0 || lo % chunk != 0 || hi < lo || (hi - lo) % 8 != 0) return ORACLE_EINVAL;
    int64_t count = 0;
    uint64_t k = 0;
    for (uint64_t c0 = lo; c0 < hi; c0 += chunk, ++k) {
        uint64_t s;
        uint64_t c1 = (c0 + chunk < hi) ? c0 + chunk : hi;
        oracle_chunk_sums(window + (c0 - lo), c0, c1, chunk, &s);
        if (s != stored[k]) {
            if ((uint64_t)count < cap) bad[count] = (uint32_t)(c0 / chunk);
            ++count;
        }
    }
    return count;
}

/* Definition 5 (locate): the byte range of chunk c and the non-empty
 * fragments overlapping it, by brute force over all fragments. */
int64_t oracle_locate(uint64_t c, uint64_t chunk, uint64_t image_bytes, uint32_t n,
                      const uint64_t *off, const uint64_t *nbytes,
                      uint64_t *range_lo, uint64_t *range_hi, uint32_t *frags, uint32_t cap)
{
    if (chunk == 0 || c * chunk >= image_bytes) return ORACLE_EINVAL;
    uint64_t a = c * chunk;
    uint64_t b = (a + chunk < image_bytes) ? a + chunk : image_bytes;
    *range_lo = a;
    *range_hi = b;
    int64_t count = 0;
    for (uint32_t i = 0; i < n; ++i) {
        if (nbytes[i] == 0) continue;
        if (off[i] < b && off[i] + nbytes[i] > a) {
            if ((uint64_t)count < cap) frags[count] = i;
            ++count;
        }
    }
    return count;
}

/* Little-endian stores for the envelope writer. */
static void put_le(uint8_t *p, uint64_t v, int width)
{
    for (int k = 0; k < width; ++k) p[k] = (uint8_t)(v >> (8 * k));
}

uint64_t oracle_envelope_bytes(uint32_t n_frag, uint64_t n_chunks, uint32_t meta_len)
{
    return 56 + 24 * (uint64_t)n_frag + 8 * n_chunks + round_up(meta_len, 8) + 8;
}

/*
 * Metadata envelope (Sec. V-B, D2H paragraph: step index, parallel
 * configuration and RNG states travel with the state).  Byte format, all
 * integers little-endian:
 *    0  u64 magic: the ASCII bytes "CKPTENV1"
 *    8  u32 version = 1
 *   12  u32 alignment A
 *   16  u64 step
 *   24  u64 chunk bytes C
 *   32  u64 image bytes I
 *   40  u64 chunk count
 *   48  u32 fragment count
 *   52  u32 caller blob length L
 *   56  fragment table, 24 B each: u64 offset, u64 bytes, u32 dtype tag, u32 class tag
 *    .  chunk sums, u64 each
 *    .  caller blob (parallel configuration, RNG states ...), zero-padded to 8 B
 *  end  u64 word-sum (definition 3) of every preceding byte of the envelope
 * Returns the envelope size, or 0 when cap is too small.
 */
uint64_t oracle_envelope(uint64_t step, uint64_t align, uint64_t chunk, uint64_t image_bytes,
                         uint64_t n_chunks, uint32_t n_frag, const uint64_t *off,
                         const uint64_t *nbytes, const uint32_t *dtype, const uint32_t *cls,
                         const uint64_t *sums, const uint8_t *meta, uint32_t meta_len,
                         uint8_t *out, uint64_t cap)
{
    uint64_t total = oracle_envelope_bytes(n_frag, n_chunks, meta_len);
    if (cap < total) return 0;
    for (uint64_t x = 0; x < total; ++x) out[x] = 0;
    const char magic[8] = {'C', 'K', 'P', 'T', 'E', 'N', 'V', '1'};
    for (int k = 0; k < 8; ++k) out[k] = (uint8_t)magic[k];
    put_le(out + 8, 1, 4);
    put_le(out + 12, align, 4);
    put_le(out + 16, step, 8);
    put_le(out + 24, chunk, 8);
    put_le(out + 32, image_bytes, 8);
    put_le(out + 40, n_chunks, 8);
    put_le(out + 48, n_frag, 4);
    put_le(out + 52, meta_len, 4);
    uint64_t p = 56;
    for (uint32_t i = 0; i < n_frag; ++i, p += 24) {
        put_le(out + p, off[i], 8);
        put_le(out + p + 8, nbytes[i], 8);
        put_le(out + p + 16, dtype[i], 4);
        put_le(out + p + 20, cls[i], 4);
    }
    for (uint64_t c = 0; c < n_chunks; ++c, p += 8) put_le(out + p, sums[c], 8);
    for (uint32_t k = 0; k < meta_len; ++k) out[p + k] = meta[k];
    p += round_up(meta_len, 8);
    uint64_t s = 0;
    for (uint64_t x = 0; x < p; x += 8) s += le_word(out + x);
    put_le(out + p, s, 8);
    return total;
}
