/*
 * nmm_oracle.c -- the CPU oracle for narrow MatMul.  TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the package's smoke check and the benchmark's CPU-baseline leg may load this
 * library.  The HIP product path never calls, links or includes it, and it shares no code,
 * header, table or helper with that path.
 *
 * What it computes (plain definitions, fp64, no blocking, no fusion, no reordering):
 *
 *  - Narrow MatMul, the paper's problem statement C = A x B with A in R^{MxK}, B in R^{KxN}
 *    (Section II-E "Problem Statement"; Section III-A, Condition 2 "Narrow Dimension"; the
 *    ENSURE clause of Algorithm 1) and its specialisation C = T x W (Section IV-B, eq. 4):
 *        y[m,n]   = sum_{k=0}^{K-1} dec(x[m,k]) * dec(W[k,n])        (ascending k)
 *        abs[m,n] = sum_{k=0}^{K-1} |dec(x[m,k]) * dec(W[k,n])|
 *    The paper's vector kernel keeps the accuracy of the matrix unit (Section IV-D "Data Type
 *    Issue") and computes the same product, so the plain product is the reference.  A product
 *    of two 16-bit floats is exact in fp64; only the K-term summation rounds, at ~K*2^-53.
 *  - The same per batch index (the per-head absorbed MLA matmuls).
 *  - The output narrowing to bf16 (Algorithm 2's final cast, Section IV-E).  The paper names
 *    the mode CAST_ROUND without defining it, so both nearest modes are provided: ties to even
 *    (the default reading, used between the chain's steps) and ties away from zero.
 *  - The vector work the paper places behind MatMul 2 (Section IV-A, eq. 1-3: c^KV = W^DKV h,
 *    k^R = RoPE(W^KR h), computed as one product, followed by RMSNorm, RoPE and caching):
 *        c' = c / sqrt(mean(c^2) + eps) * gamma      RMSNorm (Zhang and Sennrich, 2019)
 *        k' = RoPE(k, t)                             RoPE (Su et al., RoFormer), adjacent pairs
 *        cache[t] = bf16(c' | k')
 *    The paper gives neither formula in full; these are the cited methods' own definitions.
 *  - Latent attention for the decode step's independent stream: fp64 scores, softmax with
 *    the maximum subtracted, then times V.  Not a formula of the paper (its MLA figure is
 *    lost); the plain textbook definition.
 *
 * The 16-bit decoders below take the bit fields apart and rebuild the value with ldexp(), so
 * they depend on no hardware conversion instruction.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (no fast-math, no FMA contraction).
 * OpenMP only splits independent outputs across threads; each output's summation order is
 * fixed, so results are identical for any thread count.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define NMMO_F16 1
#define NMMO_BF16 2

/* ------------------------------------------------------------------ 16-bit decoders */

/* IEEE binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
double nmmo_dec_f16(uint16_t b) {
    int sign = (b >> 15) & 1;
    int e = (b >> 10) & 0x1F;
    int f = b & 0x3FF;
    double v;
    if (e == 0x1F) {
        v = (f == 0) ? INFINITY : NAN;
    } else if (e == 0) {
        v = ldexp((double)f, -24);              /* subnormal: f * 2^-10 * 2^-14 */
    } else {
        v = ldexp((double)(1024 + f), e - 25);  /* (1 + f/2^10) * 2^(e-15) */
    }
    return sign ? -v : v;
}

/* bfloat16: 1 sign, 8 exponent (bias 127), 7 fraction bits. */
double nmmo_dec_bf16(uint16_t b) {
    int sign = (b >> 15) & 1;
    int e = (b >> 7) & 0xFF;
    int f = b & 0x7F;
    double v;
    if (e == 0xFF) {
        v = (f == 0) ? INFINITY : NAN;
    } else if (e == 0) {
        v = ldexp((double)f, -133);             /* subnormal: f * 2^-7 * 2^-126 */
    } else {
        v = ldexp((double)(128 + f), e - 134);  /* (1 + f/2^7) * 2^(e-127) */
    }
    return sign ? -v : v;
}

static double dec(int dt, uint16_t b) { return dt == NMMO_F16 ? nmmo_dec_f16(b) : nmmo_dec_bf16(b); }

/* ------------------------------------------------------------------ rounding to bf16 */

#define NMMO_ROUND_EVEN 0
#define NMMO_ROUND_AWAY 1

/* Round a non-negative double s < 2^53 to an integer, nearest, ties to even or away from 0. */
static double round_nonneg(double s, int mode) {
    double fl = floor(s);
    double frac = s - fl;                 /* exact: s < 2^53 here */
    if (frac > 0.5) return fl + 1.0;
    if (frac < 0.5) return fl;
    if (mode == NMMO_ROUND_AWAY) return fl + 1.0;
    return (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
}

/* Nearest bf16 to the double a (one rounding), ties per mode.  Returns the bit pattern.  NaN
 * maps to a quiet NaN with a's sign; results beyond the largest finite bf16 (after rounding)
 * become inf. */
uint16_t nmmo_round_bf16(double a, int mode) {
    uint16_t sign = signbit(a) ? 0x8000u : 0u;
    if (isnan(a)) return (uint16_t)(sign | 0x7FC0u);
    a = fabs(a);
    if (isinf(a)) return (uint16_t)(sign | 0x7F80u);
    if (a == 0.0) return sign;
    int e;
    (void)frexp(a, &e);                   /* a = mant * 2^e, mant in [0.5, 1) */
    int unb = e - 1;                      /* a in [2^unb, 2^(unb+1)) */
    if (unb < -126) {
        /* subnormal range: the grid step is 2^-133 */
        double r = round_nonneg(ldexp(a, 133), mode);   /* 0..128 */
        if (r >= 128.0) return (uint16_t)(sign | (1u << 7));   /* rounds up to 2^-126 */
        return (uint16_t)(sign | (uint16_t)r);
    }
    /* normal: 8 significant bits; the grid step is 2^(unb-7) */
    double r = round_nonneg(ldexp(a, 7 - unb), mode);   /* in [128, 256] */
    if (r >= 256.0) { r = 128.0; unb += 1; }
    if (unb > 127) return (uint16_t)(sign | 0x7F80u);
    uint16_t ebits = (uint16_t)(unb + 127);
    uint16_t fbits = (uint16_t)((int)r - 128);
    return (uint16_t)(sign | (ebits << 7) | fbits);
}

/* The float v to bf16, ties to even (exact widening, then one rounding). */
uint16_t nmmo_round_bf16_rne(float v) { return nmmo_round_bf16((double)v, NMMO_ROUND_EVEN); }

void nmmo_round_bf16_rne_array(const float* v, uint16_t* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = nmmo_round_bf16_rne(v[i]);
}

void nmmo_round_bf16_array(const double* v, uint16_t* out, int64_t n, int mode) {
    for (int64_t i = 0; i < n; ++i) out[i] = nmmo_round_bf16(v[i], mode);
}

void nmmo_decode_array(int dt, const uint16_t* b, double* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = dec(dt, b[i]);
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

int nmmo_max_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------ narrow MatMul */

/*
 * y[m*ldy + n] and abs_y[m*ldy + n] for m < M, n < N.  x[m*ldx + k], W[k*ldw + n].
 * abs_y may be NULL.  Returns 0, or -1 on a bad argument.
 */
int nmmo_gemv(int64_t M, int64_t K, int64_t N, int dt,
              const uint16_t* x, int64_t ldx, const uint16_t* W, int64_t ldw,
              double* y, double* abs_y, int64_t ldy, int nthreads) {
    if (M < 0 || K < 0 || N < 0 || ldx < K || ldw < N || ldy < N) return -1;
    if (dt != NMMO_F16 && dt != NMMO_BF16) return -1;
    set_threads(nthreads);
    int64_t total = M * N;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < total; ++t) {
        int64_t m = t / N, n = t % N;
        double s = 0.0, sa = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            double p = dec(dt, x[m * ldx + k]) * dec(dt, W[k * ldw + n]);
            s += p;
            sa += fabs(p);
        }
        y[m * ldy + n] = s;
        if (abs_y) abs_y[m * ldy + n] = sa;
    }
    return 0;
}

/* The same product for each batch index b: x + b*stride_x, W + b*stride_w, y + b*stride_y. */
int nmmo_batched_gemv(int64_t batch, int64_t M, int64_t K, int64_t N, int dt,
                      const uint16_t* x, int64_t ldx, int64_t stride_x,
                      const uint16_t* W, int64_t ldw, int64_t stride_w,
                      double* y, double* abs_y, int64_t ldy, int64_t stride_y, int nthreads) {
    if (batch < 0) return -1;
    for (int64_t b = 0; b < batch; ++b) {
        int rc = nmmo_gemv(M, K, N, dt, x + b * stride_x, ldx, W + b * stride_w, ldw,
                           y + b * stride_y, abs_y ? abs_y + b * stride_y : NULL, ldy, nthreads);
        if (rc) return rc;
    }
    return 0;
}

/* ------------------------------------------------------------------ latent attention */

/*
 * For each head h:  s_j = scale * sum_d q[h,d] * kv[j,d]   (d < dqk, j < seq)
 *                   p_j = exp(s_j - max_i s_i) / sum_i exp(s_i - max_i s_i)
 *                   out[h,n] = sum_j p_j * kv[j,n]          (n < dv: V is kv's first dv columns)
 *                   out_abs[h,n] = sum_j p_j * |kv[j,n]|
 * q[h*ldq + d], kv[j*ldkv + d], out[h*ldo + n].  Inputs are bf16 bit patterns.
 */
int nmmo_latent_attention(int64_t heads, int64_t seq, int64_t dqk, int64_t dv,
                          const uint16_t* q, int64_t ldq, const uint16_t* kv, int64_t ldkv,
                          double scale, double* out, double* out_abs, int64_t ldo, int nthreads) {
    if (heads < 0 || seq < 1 || dqk < 0 || dv < 0 || dv > ldkv || dqk > ldkv || ldq < dqk || ldo < dv)
        return -1;
    set_threads(nthreads);
    int bad = 0;
#pragma omp parallel
    {
        double* s = (double*)malloc((size_t)seq * sizeof(double));
        if (!s) {
#pragma omp atomic write
            bad = 1;
        }
#pragma omp for schedule(static)
        for (int64_t h = 0; h < heads; ++h) {
            if (!s) continue;
            double mx = -INFINITY;
            for (int64_t j = 0; j < seq; ++j) {
                double acc = 0.0;
                for (int64_t d = 0; d < dqk; ++d)
                    acc += nmmo_dec_bf16(q[h * ldq + d]) * nmmo_dec_bf16(kv[j * ldkv + d]);
                s[j] = scale * acc;
                if (s[j] > mx) mx = s[j];
            }
            double l = 0.0;
            for (int64_t j = 0; j < seq; ++j) {
                s[j] = exp(s[j] - mx);
                l += s[j];
            }
            for (int64_t n = 0; n < dv; ++n) {
                double o = 0.0, oa = 0.0;
                for (int64_t j = 0; j < seq; ++j) {
                    double v = nmmo_dec_bf16(kv[j * ldkv + n]);
                    o += s[j] * v;
                    oa += s[j] * fabs(v);
                }
                out[h * ldo + n] = o / l;
                if (out_abs) out_abs[h * ldo + n] = oa / l;
            }
        }
        free(s);
    }
    return bad ? -2 : 0;
}

/* ------------------------------------------------------------------ the decode chain */

/*
 * The narrow-MatMul chain of one MLA single-token decode step, composed from the functions
 * above.  Every step's fp64 result is rounded to fp32 and then to bf16 (ties to even) before it
 * feeds the next step:
 *   down = x . w_down                       [1,hidden]  -> [1, q_lora+kv_lora+rope]
 *   c_q  = bf16(down[:q_lora])
 *   q    = c_q . w_uq                       -> [heads, nope+rope]
 *   qn   = bf16(q[:, :nope])
 *   lat  = qn[h] . w_uk[h]  per head        -> [heads, kv_lora]
 *   lat' = bf16(lat)
 *   o    = lat'[h] . w_uv[h]  per head      -> [heads, v_head]
 *   o'   = bf16(o)
 *   y    = o' . w_o                         -> [1, hidden]
 * y is written as double.  Scratch is allocated here.  Returns 0 or a negative error.
 */
int nmmo_mla_chain(int64_t hidden, int64_t q_lora, int64_t kv_lora, int64_t rope, int64_t heads,
                   int64_t nope, int64_t v_head,
                   const uint16_t* x, const uint16_t* w_down, const uint16_t* w_uq,
                   const uint16_t* w_uk, const uint16_t* w_uv, const uint16_t* w_o,
                   double* y, int nthreads) {
    int64_t n_down = q_lora + kv_lora + rope, n_q = heads * (nope + rope);
    int64_t big = n_down > n_q ? n_down : n_q;
    if (heads * kv_lora > big) big = heads * kv_lora;
    double* buf = (double*)malloc((size_t)big * sizeof(double));
    uint16_t* a = (uint16_t*)malloc((size_t)big * sizeof(uint16_t));
    uint16_t* b = (uint16_t*)malloc((size_t)big * sizeof(uint16_t));
    int rc = 0;
    if (!buf || !a || !b) { rc = -2; goto done; }

    rc = nmmo_gemv(1, hidden, n_down, NMMO_BF16, x, hidden, w_down, n_down, buf, NULL, n_down, nthreads);
    if (rc) goto done;
    for (int64_t i = 0; i < q_lora; ++i) a[i] = nmmo_round_bf16_rne((float)buf[i]);

    rc = nmmo_gemv(1, q_lora, n_q, NMMO_BF16, a, q_lora, w_uq, n_q, buf, NULL, n_q, nthreads);
    if (rc) goto done;
    for (int64_t h = 0; h < heads; ++h)
        for (int64_t d = 0; d < nope; ++d)
            b[h * nope + d] = nmmo_round_bf16_rne((float)buf[h * (nope + rope) + d]);

    rc = nmmo_batched_gemv(heads, 1, nope, kv_lora, NMMO_BF16, b, nope, nope, w_uk, kv_lora,
                           nope * kv_lora, buf, NULL, kv_lora, kv_lora, nthreads);
    if (rc) goto done;
    for (int64_t i = 0; i < heads * kv_lora; ++i) a[i] = nmmo_round_bf16_rne((float)buf[i]);

    rc = nmmo_batched_gemv(heads, 1, kv_lora, v_head, NMMO_BF16, a, kv_lora, kv_lora, w_uv, v_head,
                           kv_lora * v_head, buf, NULL, v_head, v_head, nthreads);
    if (rc) goto done;
    for (int64_t i = 0; i < heads * v_head; ++i) b[i] = nmmo_round_bf16_rne((float)buf[i]);

    rc = nmmo_gemv(1, heads * v_head, hidden, NMMO_BF16, b, heads * v_head, w_o, hidden, y, NULL,
                   hidden, nthreads);
done:
    free(buf); free(a); free(b);
    return rc;
}

/* ------------------------------------------------------------------ behind MatMul 2 */

/*
 * RMSNorm of the compressed latent c (Section IV-A names it among the vector work fed by
 * MatMul 2; the definition is Zhang and Sennrich's root-mean-square layer normalisation):
 *   out[i] = c[i] / sqrt((1/n) * sum_j c[j]^2 + eps) * gamma[i]          (gamma bf16)
 */
void nmmo_rmsnorm(int64_t n, const double* c, const uint16_t* gamma, double eps, double* out) {
    double ss = 0.0;
    for (int64_t j = 0; j < n; ++j) ss += c[j] * c[j];
    double inv = 1.0 / sqrt(ss / (double)n + eps);
    for (int64_t i = 0; i < n; ++i) out[i] = c[i] * inv * nmmo_dec_bf16(gamma[i]);
}

/*
 * Rotary position embedding of the decoupled key k^R at position t (eq. 2 of Section IV-A; the
 * definition is RoFormer's, Su et al.): the d values form d/2 adjacent pairs (k[2i], k[2i+1]),
 * and pair i turns by the angle t * theta^(-2i/d):
 *   out[2i]   = k[2i] cos(a_i) - k[2i+1] sin(a_i)
 *   out[2i+1] = k[2i] sin(a_i) + k[2i+1] cos(a_i)
 */
void nmmo_rope(int64_t d, const double* k, int64_t t, double theta, double* out) {
    for (int64_t i = 0; i < d / 2; ++i) {
        double a = (double)t * pow(theta, -2.0 * (double)i / (double)d);
        double cs = cos(a), sn = sin(a);
        out[2 * i] = k[2 * i] * cs - k[2 * i + 1] * sn;
        out[2 * i + 1] = k[2 * i] * sn + k[2 * i + 1] * cs;
    }
}

/*
 * The cache entry built from MatMul 2's product mm = [c^KV | k^R] (kv_lora + rope values):
 *   row[:kv_lora] = RMSNorm(mm[:kv_lora]),  row[kv_lora:] = RoPE(mm[kv_lora:], t),
 *   row_bf16 = bf16(row) (one rounding, ties per mode).
 * row may be NULL.  Returns 0 or a negative error.
 */
int nmmo_kv_entry(int64_t kv_lora, int64_t rope, const double* mm, const uint16_t* gamma, double eps,
                  double theta, int64_t t, int mode, double* row, uint16_t* row_bf16) {
    if (kv_lora < 1 || rope < 0 || (rope & 1) || !mm || !gamma || !row_bf16) return -1;
    double* r = row ? row : (double*)malloc((size_t)(kv_lora + rope) * sizeof(double));
    if (!r) return -2;
    nmmo_rmsnorm(kv_lora, mm, gamma, eps, r);
    nmmo_rope(rope, mm + kv_lora, t, theta, r + kv_lora);
    nmmo_round_bf16_array(r, row_bf16, kv_lora + rope, mode);
    if (!row) free(r);
    return 0;
}

/*
 * MatMul 2 for one token and the cache entry behind it (Section IV-A, eq. 3 and 4):
 *   mm = h . W,  W = (W^DKV | W^KR)^T  [hidden, kv_lora + rope] (row pitch ldw),
 * then nmmo_kv_entry.  mm (fp64, kv_lora + rope values) is an output too, and mm_abs (may be
 * NULL) receives sum_k |h_k W_kn|.
 */
int nmmo_mla_kv_update(int64_t hidden, int64_t kv_lora, int64_t rope, const uint16_t* h, const uint16_t* w,
                       int64_t ldw, const uint16_t* gamma, double eps, double theta, int64_t t, int mode,
                       double* mm, double* mm_abs, double* row, uint16_t* row_bf16, int nthreads) {
    int64_t n = kv_lora + rope;
    int rc = nmmo_gemv(1, hidden, n, NMMO_BF16, h, hidden, w, ldw, mm, mm_abs, n, nthreads);
    if (rc) return rc;
    return nmmo_kv_entry(kv_lora, rope, mm, gamma, eps, theta, t, mode, row, row_bf16);
}
