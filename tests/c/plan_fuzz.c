/*
 * plan_fuzz.c -- host-only checks of libckpt's planner (no GPU needed),
 * built against a copy of the runtime compiled with AddressSanitizer and
 * UndefinedBehaviorSanitizer.
 *
 * For seeded random fragment lists (empty, tiny, unaligned, chunk-crossing
 * sizes) and several chunk/alignment geometries it compares ckpt_plan with
 * the oracle's layout, and ckpt_debug_tile_plan's per-tile first/last
 * fragment with a brute-force scan over the fragment extents.  It also
 * feeds the planner bad geometries and expects CKPT_EINVAL.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "ckpt.h"

int oracle_layout(uint32_t n, const uint64_t *nbytes, uint64_t align, uint64_t chunk, uint64_t *off,
                  uint64_t *image_bytes, uint64_t *n_chunks);

static uint64_t state = 0x243F6A8885A308D3ull;
static uint64_t next_u64(void)
{
    state ^= state << 13;
    state ^= state >> 7;
    state ^= state << 17;
    return state;
}

static uint64_t pick_size(uint64_t chunk)
{
    switch (next_u64() % 8) {
    case 0: return 0;
    case 1: return 1 + next_u64() % 16;
    case 2: return 1 + next_u64() % 4096;
    case 3: return chunk - 1 + next_u64() % 3;
    case 4: return 1 + next_u64() % (3 * chunk);
    case 5: return 8192 * (1 + next_u64() % 8);
    default: return 1 + next_u64() % 70000;
    }
}

static int fail(int round, const char *what)
{
    fprintf(stderr, "FAIL case %d: %s\n", round, what);
    return 1;
}

int main(void)
{
    const uint64_t chunks[] = {8192, 16384, 65536, 1u << 20};
    const uint32_t aligns[] = {0, 256, 512, 4096};
    int cases = 0;
    for (int round = 0; round < 400; ++round) {
        uint64_t chunk = chunks[round % 4];
        uint32_t align = aligns[(round / 4) % 4];
        if (align && chunk % align) continue;
        uint32_t n = 1 + (uint32_t)(next_u64() % 300);
        uint64_t *sz = malloc(n * sizeof *sz), *off = malloc(n * sizeof *off), *ooff = malloc(n * sizeof *ooff);
        uint64_t total = 0;
        for (uint32_t i = 0; i < n; ++i) total += (sz[i] = pick_size(chunk));
        if (total == 0) sz[n - 1] = 1;
        uint64_t I = 0, nc = 0, oI = 0, onc = 0;
        if (ckpt_plan(sz, n, chunk, align, off, &I, &nc) != CKPT_OK) return fail(round, "ckpt_plan");
        if (oracle_layout(n, sz, align ? align : 256, chunk, ooff, &oI, &onc) != 0) return fail(round, "oracle");
        if (I != oI || nc != onc || memcmp(off, ooff, n * sizeof *off)) return fail(round, "layout differs");

        uint64_t tb = 0, nt = 0;
        if (ckpt_debug_tile_plan(sz, n, chunk, align, &tb, &nt, NULL, NULL) != CKPT_OK) return fail(round, "tiles");
        if (tb == 0 || chunk % tb || nt != (I + tb - 1) / tb) return fail(round, "tile geometry");
        uint32_t *tf = malloc(nt * sizeof *tf), *tl = malloc(nt * sizeof *tl);
        if (ckpt_debug_tile_plan(sz, n, chunk, align, &tb, &nt, tf, tl) != CKPT_OK) return fail(round, "tile table");
        for (uint64_t t = 0; t < nt; ++t) {
            uint64_t lo = t * tb, hi = (t + 1) * tb < I ? (t + 1) * tb : I;
            int64_t first = -1, last = -1;
            for (uint32_t i = 0; i < n; ++i) {
                if (sz[i] == 0) continue;
                if (off[i] < hi && off[i] + sz[i] > lo) {
                    if (first < 0) first = i;
                    last = i;
                }
            }
            if (first < 0) continue; /* padding-only tile: any bracket is allowed */
            if ((int64_t)tf[t] > first || (int64_t)tl[t] < last || tf[t] > tl[t] || tl[t] >= n)
                return fail(round, "tile bracket misses a fragment");
        }
        free(tf);
        free(tl);
        free(sz);
        free(off);
        free(ooff);
        ++cases;
    }
    uint64_t one = 100, I, nc;
    if (ckpt_plan(&one, 1, 0, 0, NULL, &I, &nc) != CKPT_OK) return fail(-1, "defaults");
    if (ckpt_plan(&one, 1, 1000, 0, NULL, &I, &nc) != CKPT_EINVAL) return fail(-1, "chunk not a tile multiple");
    if (ckpt_plan(&one, 1, 65536, 100, NULL, &I, &nc) != CKPT_EINVAL) return fail(-1, "odd alignment");
    if (ckpt_plan(&one, 0, 65536, 0, NULL, &I, &nc) != CKPT_EINVAL) return fail(-1, "no fragments");
    uint64_t zero = 0;
    if (ckpt_plan(&zero, 1, 65536, 0, NULL, &I, &nc) != CKPT_EINVAL) return fail(-1, "all empty");
    printf("OK plan_fuzz: %d layouts\n", cases);
    return 0;
}
