/*
 * moe_oracle.c -- plain fp64 CPU reference of the sparse Mixture-of-Experts
 * FFN layer (Mixtral-8x7B shape) served by the engine in the paper.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that the GPU library is
 * checked against.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load it.  It shares no code, header, table or helper with
 * the HIP library, and the HIP library never loads it.
 *
 * What is computed.  The paper (Sec. 4.1, "Optimize Inference Engine") states
 * that the engine work targets Mixture-of-Experts LLMs, citing Mixtral, and
 * serves Mixtral-8x7B (Sec. 5, experimental settings).  The Mixtral layer it
 * cites is, per token x (a row of d values):
 *
 *   logits  l_e = sum_i x_i Wr[e,i] (+ b_e)                      router GEMM
 *   S       = the k experts with the largest logits; exactly equal logits
 *             rank the lower expert index first                   top-k
 *   g_j     = exp(l_{S_j}) / sum_{m<k} exp(l_{S_m})               softmax over S
 *   FFN_e(x)= W2[e] ( silu(W1[e] x) * (W3[e] x) ),
 *             silu(z) = z / (1 + exp(-z))                         SwiGLU expert
 *   out     = sum_{j<k} g_j FFN_{S_j}(x)                           weighted combine
 *
 * plus, for a stack, a pre-norm residual block around every layer:
 *   a = RMSNorm(h) * gamma,  h' = h + MoE(a).
 *
 * Every value is carried in double.  bf16 inputs are widened exactly (a bf16
 * bit pattern is the top half of an IEEE float).  Nothing is rounded back to
 * bf16 or float.  Loops are plain and run in index order, so results do not
 * depend on the OpenMP thread count.  Work is arranged expert-major (each
 * expert's weight row is widened once and used for all of its tokens); this is
 * a loop order, not a change to any sum.
 *
 * Weight layout (row-major, reduction index contiguous):
 *   x [T,d], Wr [E,d], W1 [E,ffn,d], W3 [E,ffn,d], W2 [E,d,ffn], b [E] float.
 *
 * 8-bit expert weights.  The paper's engine section (Sec. 4.1, "Model
 * Quantization") stores weights as 8-bit floats, and its parallelism
 * experiment (Sec. 5) serves an 8-bit quantized Mixtral-8x7B.  The format read
 * here is OCP FP8 E4M3 with one float scale per weight row (output channel):
 *   W[e,n,i] = E4M3(q[e,n,i]) * s[e,n]
 * where E4M3(b) has sign bit 7, exponent bits 6..3 (bias 7) and mantissa bits
 * 2..0; exponent 0 is subnormal (m/8 * 2^-6); exponent 15 with mantissa 7 is
 * NaN; there is no infinity (largest finite 448).  The router stays bf16.
 *
 * Pins: tests compare this file against a pure-Python brute force on tiny
 * shapes (subset enumeration for top-k, dense all-expert evaluation), against
 * torch fp64 dense SwiGLU for E=1,k=1 and against a dense softmax mixture for
 * k=E, against closed forms for one-hot inputs, and against the layer's
 * invariants (gate weights sum to one, token-permutation equivariance, a
 * zeroed expert contributes nothing).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORACLE_OK = 0, ORACLE_BAD_ARG = 1, ORACLE_NONFINITE = 2, ORACLE_NO_MEMORY = 3 };

static double widen(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* OCP FP8 E4M3 byte -> double (exact); NaN for S.1111.111. */
static double fp8_e4m3(uint8_t b)
{
    const int sign = b >> 7, e = (b >> 3) & 15, m = b & 7;
    double v;
    if (e == 15 && m == 7)
        v = NAN;
    else if (e == 0)
        v = ldexp((double)m / 8.0, -6);
    else
        v = ldexp(1.0 + (double)m / 8.0, e - 7);
    return sign ? -v : v;
}

/* An expert weight tensor [E, rows, cols]: bf16 bits, or E4M3 bytes with one
 * float scale per row. */
typedef struct {
    const uint16_t* bf16;
    const uint8_t* q;
    const float* s;
} wmat_t;

/* Row r (counted over all experts) of a weight tensor, widened to double.
 * Returns 0 if any value is not finite. */
static int widen_row(wmat_t w, int64_t r, int64_t cols, double* out)
{
    int ok = 1;
    if (w.bf16) {
        for (int64_t i = 0; i < cols; ++i) out[i] = widen(w.bf16[r * cols + i]);
    } else {
        const double s = (double)w.s[r];
        for (int64_t i = 0; i < cols; ++i) out[i] = fp8_e4m3(w.q[r * cols + i]) * s;
    }
    for (int64_t i = 0; i < cols; ++i)
        if (!isfinite(out[i])) ok = 0;
    return ok;
}

/* Decodes n E4M3 bytes (for the tests' pins of the format). */
int oracle_fp8_e4m3(const uint8_t* q, int64_t n, double* out)
{
    if (n < 0) return ORACLE_BAD_ARG;
    for (int64_t i = 0; i < n; ++i) out[i] = fp8_e4m3(q[i]);
    return ORACLE_OK;
}

int oracle_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* Inputs must be finite: the layer is undefined otherwise. */
static int all_finite_bf16(const uint16_t* p, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        if ((p[i] & 0x7f80u) == 0x7f80u) return 0;
    return 1;
}

/* ---- router GEMM ------------------------------------------------------- */

/* logits[t,e] = sum_i x[t,i] * Wr[e,i]  (+ bias[e] when bias != NULL) */
int oracle_router_logits(const uint16_t* x, const uint16_t* wr, const float* bias,
                         int64_t T, int64_t d, int64_t E, double* logits)
{
    if (T < 0 || d <= 0 || E <= 0) return ORACLE_BAD_ARG;
    if (!all_finite_bf16(x, T * d) || !all_finite_bf16(wr, E * d)) return ORACLE_NONFINITE;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t e = 0; e < E; ++e) {
            double s = 0.0;
            for (int64_t i = 0; i < d; ++i)
                s += widen(x[t * d + i]) * widen(wr[e * d + i]);
            if (bias) s += (double)bias[e];
            logits[t * E + e] = s;
        }
    }
    return ORACLE_OK;
}

/* ---- top-k gating -------------------------------------------------------- */

/* Expert a ranks ahead of expert b: larger logit, or an equal logit and a
 * lower index.  (+0 and -0 compare equal.) */
static int ranks_ahead(double la, int a, double lb, int b)
{
    return la > lb || (la == lb && a < b);
}

/* ids[t,j]: the j-th ranked expert of token t, j < k.
 * gates[t,j] = exp(l_{ids[t,j]} - l_{ids[t,0]}) / sum_m exp(l_{ids[t,m]} - l_{ids[t,0]}),
 * i.e. a softmax over the selected logits (shifted by the largest one, which
 * leaves the ratio unchanged). */
int oracle_topk_gate(const double* logits, int64_t T, int E, int k, int32_t* ids, double* gates)
{
    if (T < 0 || E <= 0 || k <= 0 || k > E) return ORACLE_BAD_ARG;
    for (int64_t t = 0; t < T; ++t) {
        const double* l = logits + t * E;
        int32_t* s = ids + t * k;
        for (int j = 0; j < k; ++j) {
            int best = -1;
            for (int e = 0; e < E; ++e) {
                int taken = 0;
                for (int m = 0; m < j; ++m) taken |= (s[m] == e);
                if (taken) continue;
                if (best < 0 || ranks_ahead(l[e], e, l[best], best)) best = e;
            }
            s[j] = best;
        }
        double top = l[s[0]], denom = 0.0;
        for (int j = 0; j < k; ++j) denom += exp(l[s[j]] - top);
        for (int j = 0; j < k; ++j) gates[t * k + j] = exp(l[s[j]] - top) / denom;
    }
    return ORACLE_OK;
}

/* Gate weights of a given expert choice (e.g. one made elsewhere):
 * gates[t,j] = exp(l[t,ids[t,j]] - l[t,ids[t,0]]) / sum_m exp(l[t,ids[t,m]] - l[t,ids[t,0]]). */
int oracle_gates_for_ids(const double* logits, const int32_t* ids, int64_t T, int E, int k,
                         double* gates)
{
    if (T < 0 || E <= 0 || k <= 0 || k > E) return ORACLE_BAD_ARG;
    for (int64_t t = 0; t < T; ++t) {
        const double* l = logits + t * E;
        const int32_t* s = ids + t * k;
        for (int j = 0; j < k; ++j)
            if (s[j] < 0 || s[j] >= E) return ORACLE_BAD_ARG;
        double top = l[s[0]], denom = 0.0;
        for (int j = 0; j < k; ++j) denom += exp(l[s[j]] - top);
        for (int j = 0; j < k; ++j) gates[t * k + j] = exp(l[s[j]] - top) / denom;
    }
    return ORACLE_OK;
}

/* ---- dispatch: histogram, offsets, permutation ---------------------------- */

/* Assignment a = t*k + j goes to expert ids[a].
 * counts[e]   = number of assignments to e
 * offsets[e]  = sum_{e' < e} counts[e'],  offsets[E] = T*k
 * perm[r]     = the r-th assignment in (expert ascending, a ascending) order,
 *               so rows offsets[e] .. offsets[e+1]-1 hold expert e's tokens
 *               in ascending token order. */
int oracle_dispatch(const int32_t* ids, int64_t T, int E, int k,
                    int32_t* counts, int32_t* offsets, int32_t* perm)
{
    if (T < 0 || E <= 0 || k <= 0) return ORACLE_BAD_ARG;
    const int64_t A = T * k;
    for (int64_t a = 0; a < A; ++a)
        if (ids[a] < 0 || ids[a] >= E) return ORACLE_BAD_ARG;
    for (int e = 0; e < E; ++e) {
        int32_t c = 0;
        for (int64_t a = 0; a < A; ++a) c += (ids[a] == e);
        counts[e] = c;
    }
    offsets[0] = 0;
    for (int e = 0; e < E; ++e) offsets[e + 1] = offsets[e] + counts[e];
    int64_t r = 0;
    for (int e = 0; e < E; ++e)
        for (int64_t a = 0; a < A; ++a)
            if (ids[a] == e) perm[r++] = (int32_t)a;
    return ORACLE_OK;
}

/* ---- expert FFN and combine ---------------------------------------------- */

static double silu(double z) { return z / (1.0 + exp(-z)); }

/* out[t,:] = sum_j gates[t,j] * FFN_{ids[t,j]}(x[t,:]), slots summed in
 * ascending j.  Optional diagnostics (NULL to skip):
 *   h_slots [T*k, ffn]: silu(W1 x) * (W3 x) of assignment a = t*k+j
 *   y_slots [T*k, d]  : W2 h of assignment a (not gate-weighted) */
static int moe_apply(const uint16_t* x, wmat_t w1, wmat_t w3, wmat_t w2, const int32_t* ids,
                     const double* gates, int64_t T, int64_t d, int64_t ffn, int E, int k,
                     double* out, double* h_slots, double* y_slots)
{
    if (T < 0 || d <= 0 || ffn <= 0 || E <= 0 || k <= 0 || k > E) return ORACLE_BAD_ARG;
    const int64_t A = T * k;
    for (int64_t a = 0; a < A; ++a)
        if (ids[a] < 0 || ids[a] >= E) return ORACLE_BAD_ARG;
    if (!all_finite_bf16(x, T * d)) return ORACLE_NONFINITE;

    double* xd = (double*)malloc(sizeof(double) * (size_t)(T * d + 1));
    double* h = (double*)malloc(sizeof(double) * (size_t)(A * ffn + 1));
    double* y = (double*)malloc(sizeof(double) * (size_t)(A * d + 1));
    int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(A + 1));
    if (!xd || !h || !y || !rows) {
        free(xd); free(h); free(y); free(rows);
        return ORACLE_NO_MEMORY;
    }
    for (int64_t i = 0; i < T * d; ++i) xd[i] = widen(x[i]);
    int bad = 0;  /* a weight row used below holds a non-finite value */

    for (int e = 0; e < E; ++e) {
        /* the assignments routed to expert e, ascending */
        int64_t n_rows = 0;
        for (int64_t a = 0; a < A; ++a)
            if (ids[a] == e) rows[n_rows++] = a;
        if (n_rows == 0) continue;

        /* h[a,n] = silu(sum_i W1[n,i] x[t,i]) * (sum_i W3[n,i] x[t,i]) */
#pragma omp parallel
        {
            double* r1 = (double*)malloc(sizeof(double) * (size_t)d);
            double* r3 = (double*)malloc(sizeof(double) * (size_t)d);
#pragma omp for schedule(static)
            for (int64_t n = 0; n < ffn; ++n) {
                if (!widen_row(w1, (int64_t)e * ffn + n, d, r1) |
                    !widen_row(w3, (int64_t)e * ffn + n, d, r3)) {
#pragma omp atomic write
                    bad = 1;
                }
                for (int64_t q = 0; q < n_rows; ++q) {
                    const double* xt = xd + (rows[q] / k) * d;
                    double u = 0.0, v = 0.0;
                    for (int64_t i = 0; i < d; ++i) {
                        u += r1[i] * xt[i];
                        v += r3[i] * xt[i];
                    }
                    h[rows[q] * ffn + n] = silu(u) * v;
                }
            }
            free(r1);
            free(r3);
        }

        /* y[a,i] = sum_n W2[i,n] h[a,n] */
#pragma omp parallel
        {
            double* r2 = (double*)malloc(sizeof(double) * (size_t)ffn);
#pragma omp for schedule(static)
            for (int64_t i = 0; i < d; ++i) {
                if (!widen_row(w2, (int64_t)e * d + i, ffn, r2)) {
#pragma omp atomic write
                    bad = 1;
                }
                for (int64_t q = 0; q < n_rows; ++q) {
                    const double* ha = h + rows[q] * ffn;
                    double s = 0.0;
                    for (int64_t n = 0; n < ffn; ++n) s += r2[n] * ha[n];
                    y[rows[q] * d + i] = s;
                }
            }
            free(r2);
        }
    }

    if (bad) {
        free(xd); free(h); free(y); free(rows);
        return ORACLE_NONFINITE;
    }

    /* out[t,i] = sum_{j ascending} gates[t,j] * y[t*k+j, i] */
    for (int64_t t = 0; t < T; ++t) {
        for (int64_t i = 0; i < d; ++i) {
            double s = 0.0;
            for (int j = 0; j < k; ++j) s += gates[t * k + j] * y[(t * k + j) * d + i];
            out[t * d + i] = s;
        }
    }
    if (h_slots) memcpy(h_slots, h, sizeof(double) * (size_t)(A * ffn));
    if (y_slots) memcpy(y_slots, y, sizeof(double) * (size_t)(A * d));
    free(xd); free(h); free(y); free(rows);
    return ORACLE_OK;
}

int oracle_moe_apply(const uint16_t* x, const uint16_t* w1, const uint16_t* w3,
                     const uint16_t* w2, const int32_t* ids, const double* gates,
                     int64_t T, int64_t d, int64_t ffn, int E, int k,
                     double* out, double* h_slots, double* y_slots)
{
    const wmat_t m1 = {w1, NULL, NULL}, m3 = {w3, NULL, NULL}, m2 = {w2, NULL, NULL};
    return moe_apply(x, m1, m3, m2, ids, gates, T, d, ffn, E, k, out, h_slots, y_slots);
}

/* As oracle_moe_apply with E4M3 expert weights and per-row scales:
 * w1q/w3q [E,ffn,d] bytes, w1s/w3s [E,ffn]; w2q [E,d,ffn], w2s [E,d]. */
int oracle_moe_apply_fp8(const uint16_t* x, const uint8_t* w1q, const float* w1s,
                         const uint8_t* w3q, const float* w3s, const uint8_t* w2q,
                         const float* w2s, const int32_t* ids, const double* gates,
                         int64_t T, int64_t d, int64_t ffn, int E, int k,
                         double* out, double* h_slots, double* y_slots)
{
    const wmat_t m1 = {NULL, w1q, w1s}, m3 = {NULL, w3q, w3s}, m2 = {NULL, w2q, w2s};
    return moe_apply(x, m1, m3, m2, ids, gates, T, d, ffn, E, k, out, h_slots, y_slots);
}

/* The whole layer: router GEMM, top-k gating, experts, combine.  ids, gates
 * and logits are outputs (logits [T,E], ids/gates [T,k]). */
int oracle_moe_layer(const uint16_t* x, const uint16_t* wr, const float* bias,
                     const uint16_t* w1, const uint16_t* w3, const uint16_t* w2,
                     int64_t T, int64_t d, int64_t ffn, int E, int k,
                     double* out, double* logits, int32_t* ids, double* gates)
{
    int rc = oracle_router_logits(x, wr, bias, T, d, E, logits);
    if (rc) return rc;
    rc = oracle_topk_gate(logits, T, E, k, ids, gates);
    if (rc) return rc;
    return oracle_moe_apply(x, w1, w3, w2, ids, gates, T, d, ffn, E, k, out, NULL, NULL);
}

/* The whole layer with E4M3 expert weights (router in bf16). */
int oracle_moe_layer_fp8(const uint16_t* x, const uint16_t* wr, const float* bias,
                         const uint8_t* w1q, const float* w1s, const uint8_t* w3q,
                         const float* w3s, const uint8_t* w2q, const float* w2s,
                         int64_t T, int64_t d, int64_t ffn, int E, int k,
                         double* out, double* logits, int32_t* ids, double* gates)
{
    int rc = oracle_router_logits(x, wr, bias, T, d, E, logits);
    if (rc) return rc;
    rc = oracle_topk_gate(logits, T, E, k, ids, gates);
    if (rc) return rc;
    return oracle_moe_apply_fp8(x, w1q, w1s, w3q, w3s, w2q, w2s, ids, gates, T, d, ffn, E, k,
                                out, NULL, NULL);
}

/* ---- RMSNorm for the residual stack -------------------------------------- */

/* a[t,i] = h[t,i] / sqrt(mean_i h[t,i]^2 + eps) * gamma[i]; h is the float
 * residual stream, gamma bf16. */
int oracle_rmsnorm(const float* h, const uint16_t* gamma, int64_t T, int64_t d, double eps,
                   double* a)
{
    if (T < 0 || d <= 0 || !(eps >= 0.0)) return ORACLE_BAD_ARG;
    for (int64_t t = 0; t < T; ++t) {
        double ss = 0.0;
        for (int64_t i = 0; i < d; ++i) ss += (double)h[t * d + i] * (double)h[t * d + i];
        double inv = 1.0 / sqrt(ss / (double)d + eps);
        for (int64_t i = 0; i < d; ++i) a[t * d + i] = (double)h[t * d + i] * inv * widen(gamma[i]);
    }
    return ORACLE_OK;
}

/* ==========================================================================
 * The decoder layer around the MoE block, for one decode step.
 *
 * The paper's engine serves the whole Mixtral model with FlashAttention- and
 * PagedAttention-style attention kernels (Sec. 2 and Sec. 4.1).  One decoder
 * layer of the model is, per decode token (the request's next position p):
 *
 *   a   = bf16( RMSNorm(h) * gamma_attn )
 *   q   = Wq a, k = Wk a, v = Wv a            Hq query heads, Hkv key/value
 *                                             heads of hd values (Hq/Hkv
 *                                             query heads share one KV head)
 *   q, k rotated by position p (RoPE)
 *   the KV cache stores k, v (bf16) at position p of the request
 *   o_h = sum_{s <= p} softmax_s( q_h . k_s / sqrt(hd) ) v_s   (KV head of h)
 *   h   = h + Wo [o_0 .. o_{Hq-1}]
 *   h   = h + MoE( bf16( RMSNorm(h) * gamma_moe ) )
 *
 * The functions below are the steps that are not already above: RoPE,
 * attention over a paged cache, and rounding to bf16 (the cache's storage
 * precision).  The projections are plain matrix products.
 * ========================================================================== */

/* Round to the nearest bf16 value, ties to even, straight from double (no
 * intermediate float rounding).  Finite inputs within the bf16 range. */
static uint16_t round_to_bf16(double x)
{
    const uint16_t sign = signbit(x) ? 0x8000 : 0;
    if (x == 0.0) return sign;
    int e;
    const double f = frexp(fabs(x), &e); /* |x| = f * 2^e, f in [0.5, 1) */
    /* 8 significant bits for normals (exponent e - 1 >= -126), fewer below */
    int bits = 8;
    if (e - 1 < -126) bits = 8 - (-126 - (e - 1));
    /* bits = 0: |x| in [2^-134, 2^-133), rounds to 0 or the smallest subnormal */
    double v = 0.0;
    if (bits >= 0) v = ldexp(nearbyint(ldexp(f, bits)), e - bits); /* nearbyint: ties to even */
    const float fv = (float)v; /* exact: v has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &fv, sizeof u);
    return (uint16_t)(u >> 16) | sign;
}

int oracle_round_bf16(const double* x, int64_t n, uint16_t* out)
{
    if (n < 0) return ORACLE_BAD_ARG;
    for (int64_t i = 0; i < n; ++i) {
        if (!isfinite(x[i])) return ORACLE_NONFINITE;
        out[i] = round_to_bf16(x[i]);
    }
    return ORACLE_OK;
}

/* RoPE, the rotate-half pairing of the Mixtral checkpoints: element i pairs
 * with element i + hd/2 of the same head, rotated by the angle
 * pos * base^(-2i/hd), i < hd/2:
 *   y[i]        = x[i] cos - x[i + hd/2] sin
 *   y[i + hd/2] = x[i + hd/2] cos + x[i] sin
 * In place on x [T, H, hd]; token t has position pos[t]. */
int oracle_rope(double* x, int64_t T, int H, int hd, const int32_t* pos, double base)
{
    if (T < 0 || H <= 0 || hd <= 0 || hd % 2 || !(base > 0.0)) return ORACLE_BAD_ARG;
    const int half = hd / 2;
    for (int64_t t = 0; t < T; ++t) {
        if (pos[t] < 0) return ORACLE_BAD_ARG;
        for (int h = 0; h < H; ++h) {
            double* v = x + (t * H + h) * hd;
            for (int i = 0; i < half; ++i) {
                const double ang = (double)pos[t] * pow(base, -2.0 * i / hd);
                const double c = cos(ang), s = sin(ang);
                const double a = v[i], b = v[i + half];
                v[i] = a * c - b * s;
                v[i + half] = b * c + a * s;
            }
        }
    }
    return ORACLE_OK;
}

/* Decode attention over a paged KV cache.
 *   cache layout: kc, vc [pages, Hkv, page, hd] bf16 bits;
 *   token t attends to its request's positions s = 0 .. ctx[t]-1, position s
 *   stored in physical page page_table[t * maxp + s / page], slot s % page;
 *   query head h reads KV head h / (Hq / Hkv);
 *   out[t, h, :] = sum_s w_s V_s / sum_s w_s,
 *   w_s = exp(scale * q[t,h,:] . K_s - max_s'(scale * q . K_s'))
 * (the usual shift by the largest score; it leaves the softmax unchanged). */
int oracle_attention_decode(const double* q, const uint16_t* kc, const uint16_t* vc,
                            const int32_t* page_table, int64_t maxp, int64_t npages,
                            const int32_t* ctx, int64_t T, int Hq, int Hkv, int hd, int page,
                            double scale, double* out)
{
    if (T < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || hd <= 0 || page <= 0 || maxp <= 0 ||
        npages <= 0)
        return ORACLE_BAD_ARG;
    for (int64_t t = 0; t < T; ++t) {
        if (ctx[t] < 1 || ctx[t] > maxp * page) return ORACLE_BAD_ARG;
        for (int64_t j = 0; j < (ctx[t] + page - 1) / page; ++j) {
            const int32_t pg = page_table[t * maxp + j];
            if (pg < 0 || pg >= npages) return ORACLE_BAD_ARG;
        }
    }
    const int group = Hq / Hkv;
    int bad = 0;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int64_t t = 0; t < T; ++t) {
        for (int h = 0; h < Hq; ++h) {
            const int g = h / group;
            const int L = ctx[t];
            const double* qv = q + (t * Hq + h) * hd;
            double* sc = (double*)malloc(sizeof(double) * (size_t)L);
            double* acc = out + (t * Hq + h) * hd;
            if (!sc) {
#pragma omp atomic write
                bad = 1;
                continue;
            }
            double mx = -INFINITY;
            for (int s = 0; s < L; ++s) {
                const int64_t pg = page_table[t * maxp + s / page];
                const uint16_t* kr = kc + ((pg * Hkv + g) * page + s % page) * hd;
                double dot = 0.0;
                for (int i = 0; i < hd; ++i) dot += qv[i] * widen(kr[i]);
                sc[s] = scale * dot;
                if (sc[s] > mx) mx = sc[s];
            }
            double den = 0.0;
            for (int i = 0; i < hd; ++i) acc[i] = 0.0;
            for (int s = 0; s < L; ++s) {
                const int64_t pg = page_table[t * maxp + s / page];
                const uint16_t* vr = vc + ((pg * Hkv + g) * page + s % page) * hd;
                const double w = exp(sc[s] - mx);
                den += w;
                for (int i = 0; i < hd; ++i) acc[i] += w * widen(vr[i]);
            }
            for (int i = 0; i < hd; ++i) acc[i] /= den;
            free(sc);
        }
    }
    return bad ? ORACLE_NO_MEMORY : ORACLE_OK;
}
