/*
 * abi_roundtrip.c -- drives libckpt through its C ABI alone (no Python, no
 * torch; the HIP runtime the program links) and checks the result against
 * the CPU oracle (oracle/ckpt_oracle.c, linked into this test program only).
 *
 * Steps: fragments of awkward sizes (and one view at an odd byte offset) in
 * device memory; snapshot; compare the committed host image and chunk sums
 * with the oracle; trash the fragments; restore and compare; verify; flip one
 * bit in the host image and check that verify reports exactly that chunk;
 * error codes of a few misuses.  Twice: with the staged pack, then with
 * direct D2H (ckpt_config.direct_d2h).  Exit status 0 = every check passed.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "ckpt.h"

/* oracle (test infrastructure) */
int oracle_layout(uint32_t n, const uint64_t *nbytes, uint64_t align, uint64_t chunk, uint64_t *off,
                  uint64_t *image_bytes, uint64_t *n_chunks);
int oracle_pack_window(uint32_t n, const uint8_t *const *frag, const uint64_t *nbytes, const uint64_t *off,
                       uint64_t lo, uint64_t hi, uint8_t *out);
int oracle_chunk_sums(const uint8_t *window, uint64_t lo, uint64_t hi, uint64_t chunk, uint64_t *sums);

#define CHECK(cond, ...)                                                                                    \
    do {                                                                                                    \
        if (!(cond)) {                                                                                      \
            fprintf(stderr, "FAIL line %d: ", __LINE__);                                                    \
            fprintf(stderr, __VA_ARGS__);                                                                   \
            fprintf(stderr, "\n");                                                                          \
            return 1;                                                                                       \
        }                                                                                                   \
    } while (0)
#define HIP(x) CHECK((x) == hipSuccess, "%s", #x)

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint8_t next_byte(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint8_t)rng;
}

enum { NF = 9 };

/* One context over the fragments: snapshot, oracle comparison, restore,
 * verify, a located flip and the error codes; direct selects
 * ckpt_config.direct_d2h.  The fragments hold their original bytes again
 * when it returns 0. */
static int roundtrip(uint8_t *const *dev, uint8_t *const *host, const uint64_t *sizes, uint64_t chunk, int direct)
{
    ckpt_config cfg;
    memset(&cfg, 0, sizeof cfg);
    cfg.chunk_bytes = chunk;
    cfg.group_bytes = 2 * chunk; /* several groups, fragments cut at their boundaries */
    cfg.direct_d2h = (uint32_t)direct;
    ckpt_ctx *ctx = NULL;
    CHECK(ckpt_create(&cfg, &ctx) == CKPT_OK && ctx, "create");
    uint64_t sid = 0;
    CHECK(ckpt_snapshot_async(ctx, NULL, 1, NULL, 0, &sid) == CKPT_ESTATE, "snapshot before register");
    ckpt_tensor t[NF];
    for (int i = 0; i < NF; ++i) {
        t[i].dev_ptr = dev[i];
        t[i].nbytes = sizes[i];
        t[i].dtype = (uint32_t)i;
        t[i].cls = (uint32_t)(i % 4);
    }
    CHECK(ckpt_register_tensors(ctx, t, NF) == CKPT_OK, "register: %s", ckpt_last_error(ctx));
    uint32_t nbad = 0, bad[64];
    CHECK(ckpt_restore(ctx, 0, NULL, bad, 64, &nbad) == CKPT_ENOSNAP, "restore before any snapshot");

    const char meta[] = "abi-roundtrip";
    CHECK(ckpt_snapshot_async(ctx, NULL, 7, meta, sizeof meta, &sid) == CKPT_OK, "snapshot: %s", ckpt_last_error(ctx));
    CHECK(ckpt_wait(ctx, sid, CKPT_WAIT_CAPTURED, NULL, 0, NF) == CKPT_OK, "wait captured");
    CHECK(ckpt_wait(ctx, sid, CKPT_WAIT_COMMITTED, NULL, 0, 0) == CKPT_OK, "wait committed: %s", ckpt_last_error(ctx));

    uint64_t off[NF], I = 0, nc = 0, ooff[NF], oI = 0, onc = 0;
    CHECK(ckpt_layout(ctx, off, &I, &nc) == CKPT_OK, "layout");
    CHECK(oracle_layout(NF, sizes, 256, chunk, ooff, &oI, &onc) == 0, "oracle layout");
    CHECK(I == oI && nc == onc && memcmp(off, ooff, sizeof off) == 0, "layout differs from the oracle");

    void *img = NULL;
    uint64_t img_bytes = 0, *sums = NULL;
    CHECK(ckpt_host_image(ctx, sid, &img, &img_bytes, &sums) == CKPT_OK, "host image");
    uint8_t *want = (uint8_t *)malloc(I);
    uint64_t *want_sums = (uint64_t *)malloc(nc * 8);
    CHECK(oracle_pack_window(NF, (const uint8_t *const *)host, sizes, ooff, 0, I, want) == 0, "oracle pack");
    CHECK(oracle_chunk_sums(want, 0, I, chunk, want_sums) == 0, "oracle sums");
    CHECK(img_bytes == I && memcmp(img, want, I) == 0, "host image differs from the oracle");
    CHECK(memcmp(sums, want_sums, nc * 8) == 0, "chunk sums differ from the oracle");

    for (int i = 0; i < NF; ++i)
        if (sizes[i]) HIP(hipMemset(dev[i], 0xA5, sizes[i]));
    HIP(hipDeviceSynchronize());
    CHECK(ckpt_restore(ctx, sid, NULL, bad, 64, &nbad) == CKPT_OK && nbad == 0, "restore: %s", ckpt_last_error(ctx));
    for (int i = 0; i < NF; ++i) {
        if (!sizes[i]) continue;
        uint8_t *back = (uint8_t *)malloc(sizes[i]);
        HIP(hipMemcpy(back, dev[i], sizes[i], hipMemcpyDeviceToHost));
        CHECK(memcmp(back, host[i], sizes[i]) == 0, "fragment %d not restored", i);
        free(back);
    }
    CHECK(ckpt_verify(ctx, sid, bad, 64, &nbad) == CKPT_OK && nbad == 0, "verify clean image");

    /* one flipped bit in chunk 2 */
    ((uint8_t *)img)[2 * chunk + 100] ^= 0x10;
    CHECK(ckpt_verify(ctx, sid, bad, 64, &nbad) == CKPT_ECORRUPT && nbad == 1 && bad[0] == 2, "flip not located");
    ((uint8_t *)img)[2 * chunk + 100] ^= 0x10;

    uint64_t env_len = 0;
    CHECK(ckpt_envelope(ctx, sid, NULL, 0, &env_len) == CKPT_EINVAL && env_len > 0, "envelope size query");
    uint8_t *env = (uint8_t *)malloc(env_len);
    CHECK(ckpt_envelope(ctx, sid, env, env_len, &env_len) == CKPT_OK && memcmp(env, "CKPTENV1", 8) == 0, "envelope");

    CHECK(ckpt_wait(ctx, 999, CKPT_WAIT_CAPTURED, NULL, 0, 1) == CKPT_ERANGE, "unknown snapshot");
    CHECK(ckpt_register_tensors(ctx, t, NF) == CKPT_ESTATE, "second register");
    CHECK(ckpt_destroy(ctx) == CKPT_OK, "destroy");

    free(env);
    free(want);
    free(want_sums);
    printf("OK %s pass: %llu image bytes, %llu chunks\n", direct ? "direct D2H" : "staged", (unsigned long long)I,
           (unsigned long long)nc);
    return 0;
}

int main(void)
{
    const uint64_t sizes[NF] = {1, 17, 4095, 0, 70001, 256, 3, 200000, 65536};
    const uint64_t chunk = 16384;
    uint8_t *host[NF], *dev[NF];
    uint8_t *backing = NULL;
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) {
        printf("SKIP no GPU\n");
        return 77;
    }
    /* fragment 2 is a view at byte offset 3 of a larger allocation */
    HIP(hipMalloc((void **)&backing, 8192));
    for (int i = 0; i < NF; ++i) {
        host[i] = (uint8_t *)malloc(sizes[i] ? sizes[i] : 1);
        for (uint64_t k = 0; k < sizes[i]; ++k) host[i][k] = next_byte();
        if (i == 2) {
            dev[i] = backing + 3;
        } else {
            HIP(hipMalloc((void **)&dev[i], sizes[i] ? sizes[i] : 1));
        }
        if (sizes[i]) HIP(hipMemcpy(dev[i], host[i], sizes[i], hipMemcpyHostToDevice));
    }

    if (roundtrip(dev, host, sizes, chunk, 0) != 0) return 1;
    if (roundtrip(dev, host, sizes, chunk, 1) != 0) return 1;
    for (int i = 0; i < NF; ++i) {
        if (i != 2) HIP(hipFree(dev[i]));
        free(host[i]);
    }
    HIP(hipFree(backing));
    printf("OK abi_roundtrip: %d fragments, staged and direct D2H\n", NF);
    return 0;
}
