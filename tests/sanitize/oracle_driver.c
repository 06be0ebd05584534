/*
 * Drives every entry of oracle/nmm_oracle.c on small seeded inputs, edge cases included, for the
 * AddressSanitizer / UndefinedBehaviorSanitizer build that tests/test_sanitizers.py makes.  Every
 * buffer is allocated at exactly the size the function's contract states, so an access outside
 * it is a sanitizer finding.  Exits non-zero if a call rejects valid arguments or accepts bad ones.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int nmmo_gemv(int64_t, int64_t, int64_t, int, const uint16_t*, int64_t, const uint16_t*, int64_t, double*, double*,
              int64_t, int);
int nmmo_batched_gemv(int64_t, int64_t, int64_t, int64_t, int, const uint16_t*, int64_t, int64_t, const uint16_t*,
                      int64_t, int64_t, double*, double*, int64_t, int64_t, int);
int nmmo_latent_attention(int64_t, int64_t, int64_t, int64_t, const uint16_t*, int64_t, const uint16_t*, int64_t,
                          double, double*, double*, int64_t, int);
int nmmo_mla_chain(int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, int64_t, const uint16_t*, const uint16_t*,
                   const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*, double*, int);
int nmmo_kv_entry(int64_t, int64_t, const double*, const uint16_t*, double, double, int64_t, int, double*,
                  uint16_t*);
int nmmo_mla_kv_update(int64_t, int64_t, int64_t, const uint16_t*, const uint16_t*, int64_t, const uint16_t*, double,
                       double, int64_t, int, double*, double*, double*, uint16_t*, int);
uint16_t nmmo_round_bf16(double, int);
void nmmo_round_bf16_array(const double*, uint16_t*, int64_t, int);
void nmmo_decode_array(int, const uint16_t*, double*, int64_t);
double nmmo_dec_f16(uint16_t);
double nmmo_dec_bf16(uint16_t);

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint16_t next_bits(int dt) {
    state = state * 6364136223846793005ull + 1442695040888963407ull;
    uint16_t b = (uint16_t)(state >> 48);
    /* finite values of moderate size: clear the top exponent bits (fp16: 5 bits, bf16: 8) */
    return dt == 1 ? (uint16_t)((b & 0x83FFu) | 0x3800u) : (uint16_t)((b & 0x80FFu) | 0x3E00u);
}
static uint16_t* bits(int64_t n, int dt) {
    uint16_t* p = malloc((size_t)(n > 0 ? n : 1) * 2);
    for (int64_t i = 0; i < n; ++i) p[i] = next_bits(dt);
    return p;
}
static double* doubles(int64_t n) { return malloc((size_t)(n > 0 ? n : 1) * sizeof(double)); }

static int fails = 0;
#define EXPECT(c) do { if (!(c)) { fprintf(stderr, "failed: %s (line %d)\n", #c, __LINE__); ++fails; } } while (0)

int main(void) {
    const int64_t shapes[][3] = {{1, 1, 1}, {1, 7, 3}, {3, 33, 17}, {2, 0, 5}, {0, 4, 4}, {5, 64, 1}};
    for (int dt = 1; dt <= 2; ++dt)
        for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i) {
            const int64_t M = shapes[i][0], K = shapes[i][1], N = shapes[i][2];
            const int64_t ldx = K + 1, ldw = N + 2, ldy = N + 3;
            uint16_t *x = bits(M * ldx, dt), *w = bits(K * ldw, dt);
            double *y = doubles(M * ldy), *a = doubles(M * ldy);
            EXPECT(nmmo_gemv(M, K, N, dt, x, ldx, w, ldw, y, a, ldy, 2) == 0);
            EXPECT(nmmo_gemv(M, K, N, dt, x, ldx, w, ldw, y, NULL, ldy, 1) == 0);
            free(x); free(w); free(y); free(a);
            /* batched, strided: batch 3 with the strides of padded matrices */
            const int64_t B = 3, sx = M * ldx + 8, sw = K * ldw + 8, sy = M * ldy + 8;
            x = bits(B * sx, dt); w = bits(B * sw, dt);
            y = doubles(B * sy); a = doubles(B * sy);
            EXPECT(nmmo_batched_gemv(B, M, K, N, dt, x, ldx, sx, w, ldw, sw, y, a, ldy, sy, 2) == 0);
            free(x); free(w); free(y); free(a);
        }
    EXPECT(nmmo_gemv(1, 4, 4, 3, NULL, 4, NULL, 4, NULL, NULL, 4, 1) == -1);
    EXPECT(nmmo_gemv(1, 4, 4, 2, NULL, 3, NULL, 4, NULL, NULL, 4, 1) == -1);
    {   /* attention: 3 heads, 5 rows, d_qk 12, d_v 8, padded pitches; one row */
        const int64_t H = 3, S = 5, dqk = 12, dv = 8, ldq = 16, ldkv = 20, ldo = 9;
        uint16_t *q = bits(H * ldq, 2), *kv = bits(S * ldkv, 2);
        double *o = doubles(H * ldo), *oa = doubles(H * ldo);
        EXPECT(nmmo_latent_attention(H, S, dqk, dv, q, ldq, kv, ldkv, 0.25, o, oa, ldo, 2) == 0);
        EXPECT(nmmo_latent_attention(H, 1, dqk, dv, q, ldq, kv, ldkv, 0.25, o, NULL, ldo, 1) == 0);
        EXPECT(nmmo_latent_attention(H, 0, dqk, dv, q, ldq, kv, ldkv, 0.25, o, NULL, ldo, 1) == -1);
        free(q); free(kv); free(o); free(oa);
    }
    {   /* the decode chain at a small size */
        const int64_t hid = 40, ql = 24, kvl = 16, rope = 8, heads = 3, nope = 8, vh = 8;
        uint16_t *x = bits(hid, 2), *wd = bits(hid * (ql + kvl + rope), 2), *wuq = bits(ql * heads * (nope + rope), 2);
        uint16_t *wuk = bits(heads * nope * kvl, 2), *wuv = bits(heads * kvl * vh, 2), *wo = bits(heads * vh * hid, 2);
        double* y = doubles(hid);
        EXPECT(nmmo_mla_chain(hid, ql, kvl, rope, heads, nope, vh, x, wd, wuq, wuk, wuv, wo, y, 2) == 0);
        free(x); free(wd); free(wuq); free(wuk); free(wuv); free(wo); free(y);
    }
    {   /* the cache entry, with and without the fp64 row, rope 0 and a bad odd rope */
        const int64_t kvl = 12, rope = 6, hid = 24;
        double* mm = doubles(kvl + rope);
        for (int64_t i = 0; i < kvl + rope; ++i) mm[i] = (double)(i % 5) - 2.0;
        uint16_t *g = bits(kvl, 2), *row_b = bits(kvl + rope, 2);
        double* row = doubles(kvl + rope);
        EXPECT(nmmo_kv_entry(kvl, rope, mm, g, 1e-6, 10000.0, 7, 0, row, row_b) == 0);
        EXPECT(nmmo_kv_entry(kvl, rope, mm, g, 1e-6, 10000.0, 7, 1, NULL, row_b) == 0);
        EXPECT(nmmo_kv_entry(kvl, 0, mm, g, 1e-6, 10000.0, 7, 0, NULL, row_b) == 0);
        EXPECT(nmmo_kv_entry(kvl, 5, mm, g, 1e-6, 10000.0, 7, 0, NULL, row_b) == -1);
        uint16_t *h = bits(hid, 2), *w = bits(hid * (kvl + rope + 2), 2);
        double* ma = doubles(kvl + rope);
        EXPECT(nmmo_mla_kv_update(hid, kvl, rope, h, w, kvl + rope + 2, g, 1e-6, 10000.0, 3, 0, mm, ma, row, row_b, 2) == 0);
        free(mm); free(g); free(row_b); free(row); free(h); free(w); free(ma);
    }
    {   /* rounding and decoding over every 16-bit pattern */
        uint16_t* all = malloc(65536 * 2);
        double* d = doubles(65536);
        for (int i = 0; i < 65536; ++i) all[i] = (uint16_t)i;
        nmmo_decode_array(1, all, d, 65536);
        nmmo_decode_array(2, all, d, 65536);
        uint16_t* back = malloc(65536 * 2);
        nmmo_round_bf16_array(d, back, 65536, 0);
        nmmo_round_bf16_array(d, back, 65536, 1);
        for (int i = 0; i < 65536; ++i) {
            const uint16_t b = (uint16_t)i;
            if ((b & 0x7F80u) == 0x7F80u && (b & 0x7Fu)) continue;      /* NaNs: any NaN back */
            EXPECT(nmmo_round_bf16(nmmo_dec_bf16(b), 0) == b);
        }
        (void)nmmo_dec_f16(0x7C00u);
        free(all); free(d); free(back);
    }
    printf("oracle driver: %d failures\n", fails);
    return fails ? 1 : 0;
}
