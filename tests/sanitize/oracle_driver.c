/* The fp64 oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (gcc, CPU): retained sets of random layouts and policies, and attention over
 * them on small random caches, several thread counts. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_retained(const int32_t *seg, const int32_t *pol, int32_t pol_per_seq, int32_t B, int32_t *idx,
                    int32_t max_keep, int32_t *count);
int oracle_attn(const uint16_t *q, const uint16_t *k, const uint16_t *v, int32_t NL, int32_t B, int32_t Hq,
                int32_t Hkv, int32_t D, int32_t Lmax, const int32_t *idx, const int32_t *count, int32_t max_keep,
                double scale, double *out, double *lse, int32_t n_threads);

static uint64_t st = 12345;
static int64_t rnd(int64_t lo, int64_t hi) {
    st = st * 6364136223846793005ull + 1442695040888963407ull;
    return lo + (int64_t)((st >> 33) % (uint64_t)(hi - lo + 1));
}

int main(void) {
    for (int it = 0; it < 300; ++it) {
        const int B = (int)rnd(1, 4), NL = (int)rnd(1, 2), Hkv = (int)rnd(1, 2), G = (int)rnd(1, 3), D = 8;
        int32_t seg[16], pol[20];
        int64_t Lmax = 1;
        for (int b = 0; b < B; ++b) {
            seg[4 * b] = (int32_t)rnd(0, 5);
            seg[4 * b + 1] = (int32_t)rnd(0, 60);
            seg[4 * b + 2] = (int32_t)rnd(0, 3);
            seg[4 * b + 3] = (int32_t)rnd(1, 40);
            const int64_t L = seg[4 * b] + seg[4 * b + 1] + seg[4 * b + 2] + seg[4 * b + 3];
            if (L > Lmax) Lmax = L;
            pol[5 * b] = rnd(0, 3) ? (int32_t)rnd(1, 50) : -1;
            pol[5 * b + 1] = (int32_t)rnd(0, 30);
            pol[5 * b + 2] = (int32_t)rnd(0, 5);
            pol[5 * b + 3] = rnd(0, 3) ? (int32_t)rnd(1, 30) : -1;
            pol[5 * b + 4] = (int32_t)rnd(0, 3);
        }
        const int32_t max_keep = (int32_t)Lmax;
        int32_t *idx = malloc(sizeof(int32_t) * B * max_keep), count[4];
        if (oracle_retained(seg, pol, 1, B, idx, max_keep, count) != 0) return 1;
        const int Hq = Hkv * G;
        const size_t nq = (size_t)NL * B * Hq * D, nk = (size_t)NL * B * Hkv * Lmax * D;
        uint16_t *q = malloc(2 * nq), *k = malloc(2 * nk), *v = malloc(2 * nk);
        for (size_t i = 0; i < nq; ++i) q[i] = (uint16_t)(0x3c00 + rnd(0, 0x3ff)) ^ (uint16_t)(rnd(0, 1) << 15);
        for (size_t i = 0; i < nk; ++i) {
            k[i] = (uint16_t)(0x3c00 + rnd(0, 0x3ff)) ^ (uint16_t)(rnd(0, 1) << 15);
            v[i] = (uint16_t)(0x3c00 + rnd(0, 0x3ff)) ^ (uint16_t)(rnd(0, 1) << 15);
        }
        double *out = malloc(sizeof(double) * nq), *lse = malloc(sizeof(double) * NL * B * Hq);
        if (oracle_attn(q, k, v, NL, B, Hq, Hkv, D, (int32_t)Lmax, idx, count, max_keep, 0.5, out, lse,
                        (int32_t)rnd(1, 4)) != 0)
            return 2;
        free(idx);
        free(q);
        free(k);
        free(v);
        free(out);
        free(lse);
    }
    printf("oracle driver: ok\n");
    return 0;
}
