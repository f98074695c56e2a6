// Host-side exercise of libmurmur's C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer (built with g++, linked against the ABI layer and
// a stub of the kernel launchers, no GPU).  It runs every host-only entry point
// on many random inputs and every argument check of the device calls; the
// device calls are all rejected before a launch (the stub aborts if one is
// reached).
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <vector>

#include "murmur.h"

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static int64_t rnd(int64_t lo, int64_t hi) {  // inclusive, splitmix64
    rng_state += 0x9E3779B97F4A7C15ull;
    uint64_t z = rng_state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return lo + (int64_t)(z % (uint64_t)(hi - lo + 1));
}

#define CHECK(c)                                                     \
    do {                                                             \
        if (!(c)) {                                                  \
            fprintf(stderr, "check failed at %d: %s\n", __LINE__, #c); \
            return 1;                                                \
        }                                                            \
    } while (0)

int main() {
    // Sizing, ring layout and workspace planning on random layouts and policies, including invalid ones.
    for (int it = 0; it < 2000; ++it) {
        const int B = (int)rnd(1, 16);
        std::vector<murmur_seg> seg(B);
        std::vector<murmur_policy> pol(B);
        for (int b = 0; b < B; ++b) {
            seg[b] = {(int32_t)rnd(-1, 40), (int32_t)rnd(0, 3000), (int32_t)rnd(0, 10), (int32_t)rnd(0, 3000)};
            pol[b] = {(int32_t)(rnd(0, 4) ? rnd(1, 900) : -1), (int32_t)rnd(-1, 600), (int32_t)rnd(0, 40),
                      (int32_t)(rnd(0, 4) ? rnd(0, 400) : -1), (int32_t)rnd(0, 8)};
        }
        std::vector<int32_t> counts(B), ranges(B * 12), cur(B);
        int32_t mx = 0;
        const int rc = murmur_retained_count_host(seg.data(), pol.data(), 1, B, counts.data(), &mx);
        CHECK(rc == MURMUR_OK || rc == MURMUR_EINVAL);
        const int32_t cap = (int32_t)rnd(-1, 500);
        const int rr = murmur_ring_layout_host(seg.data(), pol.data(), 1, B, cap, ranges.data(), cur.data());
        CHECK(rr == MURMUR_OK || rr == MURMUR_EINVAL);
        if (rc == MURMUR_OK && rr == MURMUR_OK)
            for (int b = 0; b < B; ++b) {
                int64_t total = 0;
                for (int k = 0; k < 6; ++k) total += ranges[b * 12 + 2 * k + 1];
                CHECK(total == counts[b]);
            }
        std::vector<int32_t> blocks(B * 4);
        const int32_t bs = (int32_t)rnd(0, 64);
        const int fr = murmur_freeable_blocks_host(seg.data(), pol.data(), 1, B, bs, blocks.data());
        CHECK(fr == MURMUR_OK || fr == MURMUR_EINVAL);
        if (fr == MURMUR_OK && rc == MURMUR_OK)
            for (int b = 0; b < B; ++b) {  // freed blocks and retained positions never meet
                const int64_t length = (int64_t)seg[b].prompt_pre + seg[b].speech_len + seg[b].prompt_mid + seg[b].out_len;
                int64_t freed = 0;
                for (int k = 0; k < 2; ++k) {
                    CHECK(blocks[b * 4 + 2 * k] >= 0 && blocks[b * 4 + 2 * k + 1] >= 0);
                    CHECK(((int64_t)blocks[b * 4 + 2 * k] + blocks[b * 4 + 2 * k + 1]) * bs <= length);
                    freed += (int64_t)blocks[b * 4 + 2 * k + 1] * bs;
                }
                CHECK(freed + counts[b] <= length);
            }
        size_t bytes = 0;
        const int32_t split = (int32_t)(rnd(0, 3) ? 32 * rnd(0, 40) : -1);
        const int wr = murmur_decode_attn_workspace((int32_t)rnd(1, 28), B, (int32_t)(4 * rnd(1, 7)), 4,
                                                    (int32_t)rnd(1, 40000), split, &bytes);
        CHECK(wr == MURMUR_OK || wr == MURMUR_EINVAL || wr == MURMUR_EUNSUPPORTED);
    }
    // Chunk planning and Equation 4 on random segment lists.
    for (int it = 0; it < 500; ++it) {
        const int n = (int)rnd(0, 200);
        std::vector<double> s0(n), s1(n);
        double t = (double)rnd(0, 50);
        for (int i = 0; i < n; ++i) {
            s0[i] = t;
            t += (double)rnd(1, it % 7 == 0 ? 900 : 60) + rnd(0, 99) / 100.0;
            s1[i] = t;
            t += (double)rnd(0, it % 5 == 0 ? 700 : 30);
        }
        const int cap = (int)rnd(1, 64);
        std::vector<double> cs(cap), cl(cap);
        std::vector<int32_t> tok(cap), of(n > 0 ? n : 1);
        int32_t nc = 0;
        const int rc = murmur_plan_chunks(s0.data(), s1.data(), n, t + 10, 300.0, 7.5, of.data(), cs.data(), cl.data(),
                                          tok.data(), cap, &nc);
        CHECK(rc == MURMUR_OK || rc == MURMUR_ENOSPACE);
        if (rc == MURMUR_OK && nc > 0) {
            std::vector<double> tl(nc), out(nc);
            std::vector<int32_t> ch(nc);
            for (int c = 0; c < nc; ++c) {
                tl[c] = cl[c] / 2;
                ch[c] = c;
            }
            CHECK(murmur_chunk_timestamps(tl.data(), ch.data(), nc, cl.data(), nc, out.data()) == MURMUR_OK);
            for (int c = 0; c < nc; ++c) CHECK(fabs(out[c] - (cs[c] + tl[c])) < 1e-6);
        }
    }
    // Device entry points: argument checks only (every call below is rejected before any launch).
    void *fake = (void *)(uintptr_t)0x100000;
    int32_t *fi = (int32_t *)fake;
    const murmur_seg *fseg = (const murmur_seg *)fake;
    const murmur_policy *fpol = (const murmur_policy *)fake;
    murmur_kv kv{fake, fake, 1, 4096, 4096LL * 128 * 4, 4096LL * 128 * 4, 4096LL * 128, 128};
    CHECK(murmur_decode_attn(fake, &kv, fi, nullptr, fi, 850, 12, 28, 4, 64, 1.f, 0, fake, MURMUR_DTYPE_BF16,
                             nullptr, fake, 1 << 30, nullptr) == MURMUR_EUNSUPPORTED);
    CHECK(murmur_decode_attn(fake, &kv, fi, nullptr, fi, 850, 12, 28, 5, 128, 1.f, 0, fake, MURMUR_DTYPE_BF16,
                             nullptr, fake, 1 << 30, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_decode_attn(fake, &kv, fi, nullptr, fi, 850, 12, 28, 4, 128, NAN, 0, fake, MURMUR_DTYPE_BF16,
                             nullptr, fake, 1 << 30, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_decode_step(fseg, fpol, 4, fake, &kv, nullptr, nullptr, nullptr, 850, 12, 28, 4, 128, 1.f, 0, fake,
                             MURMUR_DTYPE_BF16, nullptr, fake, 1 << 30, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_decode_step_static(fseg, fpol, 4, fake, &kv, nullptr, nullptr, nullptr, 850, 12, 28, 4, 128, 1.f,
                                    0, fake, MURMUR_DTYPE_BF16, nullptr, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_decode_step_static(fseg, fpol, 0, fake, &kv, nullptr, nullptr, nullptr, 850, 12, 28, 4, 128, 1.f,
                                    32, fake, MURMUR_DTYPE_BF16, nullptr, nullptr) == MURMUR_ENOSPACE);
    murmur_ring ring{0, fake, fake};
    CHECK(murmur_decode_step_ring(fseg, fpol, 1, &ring, fake, &kv, nullptr, nullptr, nullptr, 850, 12, 28, 4, 128,
                                  1.f, 0, fake, MURMUR_DTYPE_BF16, nullptr, fake, 1 << 30, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_evict_compact(nullptr, fpol, 0, 12, fi, 10, fi, nullptr, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_evict_compact_paged(fseg, fpol, 0, 12, fi, 8, 12, fi, 10, fi, nullptr, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_read_probe(fake, 1000, 256, 256, 8, MURMUR_PROBE_REGISTERS, (uint32_t *)fake, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_read_probe(fake, 1024, 256, 1024, 8, MURMUR_PROBE_LDS, (uint32_t *)fake, nullptr) == MURMUR_EINVAL);
    CHECK(murmur_paged_step(fseg, fpol, 0, 12, fi, 8, 12, fi, fi, 64, 0, nullptr, 0, nullptr, nullptr, nullptr) ==
          MURMUR_EINVAL);  // block size not a power of two
    CHECK(murmur_paged_step(fseg, fpol, 0, 12, fi, 8, 16, fi, fi, 0, 0, nullptr, 0, nullptr, nullptr, nullptr) ==
          MURMUR_EINVAL);  // no capacity
    CHECK(murmur_paged_step(fseg, fpol, 0, 12, fi, 8, 16, fi, fi, 64, 0, &kv, 4, nullptr, fake, nullptr) ==
          MURMUR_EINVAL);  // a pool without the current K
    CHECK(murmur_last_error()[0] != '\0');
    printf("host driver: ok\n");
    return 0;
}
