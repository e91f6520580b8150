/*
 * oracle.c -- plain CPU oracle for the Prox sparse SwiGLU FFN decode step.
 *
 * TEST INFRASTRUCTURE ONLY.  This is the slow, obviously-correct reference
 * that the HIP path is checked against.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it; the product library never
 * does, and this file shares no code, header or table with it.
 *
 * Arithmetic is IEEE binary64 throughout.  16-bit inputs (bf16 or fp16 bit
 * patterns) are converted to double exactly.  The file is compiled with
 * -ffp-contract=off so no multiply-add is fused.  OpenMP only splits
 * independent output channels / columns across threads; every individual sum
 * is taken in the ascending index order written below.
 *
 * Notation (Sec. 2.1): W_gate, W_up in R^{d x f}; W_down in R^{f x d};
 * u = x W_up, h = SiLU(x W_gate), s = u (.) h.  Storage is channel-major:
 *   wg[j*d + i] = W_gate[i, j],  wu[j*d + i] = W_up[i, j],
 *   wd[j*d + c] = W_down[j, c];  x[b*d + i] for batch row b.
 * Proxy codes use the same [f][d] layout; scales are [f][d/group].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define DT_F16 0
#define DT_BF16 1

/* ------------------------------------------------------------------ */
/* Exact 16-bit -> double conversions, and double -> fp16 rounding      */
/* ------------------------------------------------------------------ */

static double bf16_to_double(uint16_t h)
{
    /* bf16 is the top half of an IEEE binary32. */
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double f16_to_double(uint16_t h)
{
    /* IEEE binary16: 1 sign, 5 exponent (bias 15), 10 fraction bits. */
    int sign = h >> 15, e = (h >> 10) & 31, m = h & 1023;
    double v;
    if (e == 0)
        v = ldexp((double)m, -24);               /* subnormal: m * 2^-24 */
    else if (e == 31)
        v = m ? NAN : INFINITY;
    else
        v = ldexp((double)(m + 1024), e - 25);   /* (1 + m/1024) * 2^(e-15) */
    return sign ? -v : v;
}

double oracle_half_to_double(uint16_t h, int dtype)
{
    return dtype == DT_BF16 ? bf16_to_double(h) : f16_to_double(h);
}

/* Round a double to IEEE binary16, round-to-nearest ties-to-even. */
uint16_t oracle_double_to_f16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isnan(v))
        return 0x7E00;
    if (a == 0.0)
        return sign;
    int e2;
    frexp(a, &e2);                 /* a in [2^(e2-1), 2^e2) */
    int E = e2 - 1;                /* unbiased exponent of a */
    if (E < -14)
        E = -14;                   /* subnormal binade shares the 2^-24 quantum */
    double quantum = ldexp(1.0, E - 10);
    double r = nearbyint(a / quantum) * quantum;   /* default mode: ties to even */
    if (r >= 65536.0)
        return sign | 0x7C00;      /* overflow to infinity */
    if (r < ldexp(1.0, -14))
        return sign | (uint16_t)(r / ldexp(1.0, -24));
    int er;
    double fr = frexp(r, &er);     /* r = fr * 2^er, fr in [0.5, 1) */
    uint16_t biased = (uint16_t)(er - 1 + 15);
    uint16_t mant = (uint16_t)((fr * 2.0 - 1.0) * 1024.0);
    return sign | (uint16_t)(biased << 10) | mant;
}

/* Round a double to bfloat16 (8 exponent bits as binary32, 7 fraction bits),
 * round-to-nearest ties-to-even; returns the bit pattern. */
uint16_t oracle_double_to_bf16(double v)
{
    uint16_t sign = signbit(v) ? 0x8000 : 0;
    double a = fabs(v);
    if (isnan(v))
        return 0x7FC0;
    if (a == 0.0)
        return sign;
    int e2;
    frexp(a, &e2);
    int E = e2 - 1;
    if (E < -126)
        E = -126;                  /* subnormals share the 2^-133 quantum */
    double quantum = ldexp(1.0, E - 7);
    double r = nearbyint(a / quantum) * quantum;
    if (r >= ldexp(1.0, 128))
        return sign | 0x7F80;
    float fr = (float)r;           /* exact: r has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &fr, sizeof u);
    return sign | (uint16_t)(u >> 16);
}

/* out[i] = the exact value of the 16-bit pattern h[i]. */
void oracle_halves_to_double(const uint16_t *h, int n, int dtype, double *out)
{
    for (int i = 0; i < n; ++i)
        out[i] = oracle_half_to_double(h[i], dtype);
}

/* out[i] = v[i] rounded to the 16-bit dtype (RNE), as bit patterns. */
void oracle_round_to_dtype(const double *v, int n, int dtype, uint16_t *out)
{
    for (int i = 0; i < n; ++i)
        out[i] = dtype == DT_BF16 ? oracle_double_to_bf16(v[i]) : oracle_double_to_f16(v[i]);
}

static double silu(double z)
{
    /* SiLU(z) = z * sigmoid(z) = z / (1 + e^{-z})  (Sec. 2.1). */
    return z / (1.0 + exp(-z));
}

/* GELU(z) = z * Phi(z), Phi the standard normal CDF = erfc(-z / sqrt 2) / 2
 * (= (1 + erf(z / sqrt 2)) / 2, without the cancellation for z << 0): the
 * gate of a GeGLU FFN. */
static double gelu(double z)
{
    return 0.5 * z * erfc(-z / sqrt(2.0));
}

/* Gate activation of the gated FFN: 0 SiLU (SwiGLU), 1 GELU (GeGLU). */
double oracle_gate_act(double z, int act)
{
    return act == 0 ? silu(z) : gelu(z);
}

#define XV(b, i) oracle_half_to_double(x[(size_t)(b) * d + (i)], dtype)
#define WV(w, j, i) oracle_half_to_double((w)[(size_t)(j) * d + (i)], dtype)

/* ------------------------------------------------------------------ */
/* Step 1 -- proxy quantisation (Sec. 4.3)                              */
/* ------------------------------------------------------------------ */
/*
 * Symmetric quantisation of one matrix W (channel-major [f][d]).  For each
 * output channel j and each group of `group` consecutive input channels:
 *   amax  = max |W[i,j]| over the group
 *   sigma = fp16_RNE(amax / qmax),  qmax = 2^(bits-1) - 1   (7 or 127)
 *   q     = clamp(round_half_even(W[i,j] / sigma), -qmax, qmax), q = 0 if sigma == 0
 * group == d gives one scale per output channel (per-row quantisation).
 * codes: int8 [f][d]; scales: fp16 bits [f][d/group].
 */
void oracle_quantize(const uint16_t *w, int dtype, int d, int f, int bits, int group,
                     int8_t *codes, uint16_t *scales)
{
    const int qmax = (1 << (bits - 1)) - 1;
    const int ng = d / group;
#pragma omp parallel for schedule(static)
    for (int j = 0; j < f; ++j) {
        for (int g = 0; g < ng; ++g) {
            double amax = 0.0;
            for (int i = g * group; i < (g + 1) * group; ++i) {
                double a = fabs(WV(w, j, i));
                if (a > amax)
                    amax = a;
            }
            uint16_t sbits = oracle_double_to_f16(amax / (double)qmax);
            scales[(size_t)j * ng + g] = sbits;
            double sigma = f16_to_double(sbits);
            for (int i = g * group; i < (g + 1) * group; ++i) {
                double q = 0.0;
                if (sigma != 0.0) {
                    q = nearbyint(WV(w, j, i) / sigma);
                    if (q > qmax)
                        q = qmax;
                    if (q < -qmax)
                        q = -qmax;
                }
                codes[(size_t)j * d + i] = (int8_t)q;
            }
        }
    }
}

/* ------------------------------------------------------------------ */
/* Stage 2 on INT4 base weights (W4A16)                                 */
/* ------------------------------------------------------------------ */

/*
 * Low-bit base weights combined with the sparse step, which the paper leaves
 * to future work (Sec. 5.1, compatibility with model quantization).  Each of
 * W_gate, W_up, W_down is stored as the symmetric 4-bit group quantisation of
 * Sec. 4.3 (oracle_quantize with bits = 4): entry (j, i) stands for
 * sigma_{j,g(i)} * q_{j,i}, g(i) = i / group.
 * Gate and up sum x_i q_{j,i} over each group and scale each group sum once;
 * the down row j scales q_{j,c} by the sigma of output column c's group.
 * Codes are int8 [f][d], scales fp16 bits [f][d/group].  Otherwise the step
 * is oracle_stage2: s_{b,j} = act(g_{b,j}) u_{b,j}, y_b = sum_j s_{b,j} W_down[j, :].
 */
void oracle_stage2_w4(const uint16_t *x, int dtype, int B, int d, int group,
                      const int8_t *cg, const uint16_t *sg, const int8_t *cu,
                      const uint16_t *su, const int8_t *cd, const uint16_t *sd,
                      const int32_t *ff_idx, int k_ff, double *s_out, double *y, int act)
{
    const int ng = d / group;
    double *s = (double *)malloc(sizeof(double) * (size_t)B * (size_t)(k_ff > 0 ? k_ff : 1));
#pragma omp parallel for schedule(static)
    for (int t = 0; t < k_ff; ++t) {
        int j = ff_idx[t];
        for (int b = 0; b < B; ++b) {
            double g = 0.0, u = 0.0;
            for (int gr = 0; gr < ng; ++gr) {
                double gq = 0.0, uq = 0.0;   /* sum of x_i q_{j,i} over the group */
                for (int i = gr * group; i < (gr + 1) * group; ++i) {
                    double xi = XV(b, i);
                    gq += xi * (double)cg[(size_t)j * d + i];
                    uq += xi * (double)cu[(size_t)j * d + i];
                }
                g += f16_to_double(sg[(size_t)j * ng + gr]) * gq;
                u += f16_to_double(su[(size_t)j * ng + gr]) * uq;
            }
            s[(size_t)b * k_ff + t] = oracle_gate_act(g, act) * u;
        }
    }
    const int cblk = 256;
#pragma omp parallel for schedule(static)
    for (int c0 = 0; c0 < d; c0 += cblk) {
        int c1 = c0 + cblk < d ? c0 + cblk : d;
        for (int b = 0; b < B; ++b) {
            double *yb = y + (size_t)b * d;
            for (int c = c0; c < c1; ++c)
                yb[c] = 0.0;
            for (int t = 0; t < k_ff; ++t) {
                int j = ff_idx[t];
                double sj = s[(size_t)b * k_ff + t];
                for (int c = c0; c < c1; ++c)
                    yb[c] += sj * f16_to_double(sd[(size_t)j * ng + c / group]) *
                             (double)cd[(size_t)j * d + c];
            }
        }
    }
    if (s_out)
        memcpy(s_out, s, sizeof(double) * (size_t)B * (size_t)k_ff);
    free(s);
}

/* ------------------------------------------------------------------ */
/* Top-k selection (App. A.6, per-token top-k rule)                     */
/* ------------------------------------------------------------------ */

typedef struct {
    double key;
    int idx;
} keyed;

static int by_key_desc_then_index(const void *pa, const void *pb)
{
    const keyed *a = (const keyed *)pa, *b = (const keyed *)pb;
    if (a->key > b->key)
        return -1;
    if (a->key < b->key)
        return 1;
    return (a->idx > b->idx) - (a->idx < b->idx);
}

static int int_asc(const void *pa, const void *pb)
{
    int a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

/* Indices of the k largest keys, ties going to the lower index; the result
 * is returned in ascending index order. */
void oracle_topk(const double *key, int n, int k, int32_t *idx_out)
{
    keyed *arr = (keyed *)malloc(sizeof(keyed) * (size_t)(n > 0 ? n : 1));
    for (int i = 0; i < n; ++i) {
        arr[i].key = key[i];
        arr[i].idx = i;
    }
    qsort(arr, (size_t)n, sizeof(keyed), by_key_desc_then_index);
    for (int t = 0; t < k; ++t)
        idx_out[t] = arr[t].idx;
    qsort(idx_out, (size_t)k, sizeof(int32_t), int_asc);
    free(arr);
}

/* Step 2 -- input mask m_x (Sec. 4.1) read as a per-token top-k: keep the
 * k_in input channels with the largest a_i = max_b |x_{b,i}| (one set shared
 * by the batch rows). */
void oracle_select_inputs(const uint16_t *x, int dtype, int B, int d, int k_in,
                          int32_t *in_idx)
{
    double *a = (double *)malloc(sizeof(double) * (size_t)d);
    for (int i = 0; i < d; ++i) {
        double m = 0.0;
        for (int b = 0; b < B; ++b) {
            double v = fabs(XV(b, i));
            if (v > m)
                m = v;
        }
        a[i] = m;
    }
    oracle_topk(a, d, k_in, in_idx);
    free(a);
}

/* ------------------------------------------------------------------ */
/* Step 3 -- proxy intermediate state (Sec. 4.1, Stage 1)               */
/* ------------------------------------------------------------------ */
/*
 * g~ = Pi_in(x, W~_gate, m_x),  u~ = Pi_in(x, W~_up, m_x),
 * s~ = SiLU(g~) (.) u~,  score_j = max_b |s~_{b,j}|.
 * proxy_kind 0: W~[i,j] = q[i,j] * sigma[g(i), j] from codes/scales.
 * proxy_kind 1: W~ = W itself (unquantised proxy).
 * gt, ut, st are [B][f] (may be NULL); score is [f].
 */
void oracle_proxy(const uint16_t *x, int dtype, int B, int d, int f,
                  const int32_t *in_idx, int k_in, int proxy_kind,
                  const int8_t *cg, const uint16_t *sg,
                  const int8_t *cu, const uint16_t *su, int group,
                  const uint16_t *wg, const uint16_t *wu,
                  double *gt, double *ut, double *st, double *score, int act)
{
    const int ng = group > 0 ? d / group : 0;
#pragma omp parallel for schedule(static)
    for (int j = 0; j < f; ++j) {
        double best = 0.0;
        for (int b = 0; b < B; ++b) {
            double g = 0.0, u = 0.0;
            for (int t = 0; t < k_in; ++t) {
                int i = in_idx[t];
                double xi = XV(b, i), wgt, wut;
                if (proxy_kind == 0) {
                    size_t sidx = (size_t)j * ng + i / group;
                    wgt = (double)cg[(size_t)j * d + i] * f16_to_double(sg[sidx]);
                    wut = (double)cu[(size_t)j * d + i] * f16_to_double(su[sidx]);
                } else {
                    wgt = WV(wg, j, i);
                    wut = WV(wu, j, i);
                }
                g += xi * wgt;
                u += xi * wut;
            }
            double s = oracle_gate_act(g, act) * u;
            if (gt)
                gt[(size_t)b * f + j] = g;
            if (ut)
                ut[(size_t)b * f + j] = u;
            if (st)
                st[(size_t)b * f + j] = s;
            if (fabs(s) > best)
                best = fabs(s);
        }
        score[j] = best;
    }
}

/* Step 4 -- channel mask m_s (Sec. 4.1) read as top-k over the proxy score,
 * shared by the batch. */
void oracle_select_channels(const double *score, int f, int k_ff, int32_t *ff_idx)
{
    oracle_topk(score, f, k_ff, ff_idx);
}

/* ------------------------------------------------------------------ */
/* Step 5 -- exact sparse computation (Sec. 4.1, Stage 2)               */
/* ------------------------------------------------------------------ */
/*
 * For the selected channels j (ascending), over ALL d inputs:
 *   g_j = x . W_gate[:, j],  u_j = x . W_up[:, j],  s_j = SiLU(g_j) u_j
 *   y   = sum_{j in M, ascending} s_j W_down[j, :]
 * s_out is [B][k_ff] (may be NULL), y is [B][d].
 */
void oracle_stage2(const uint16_t *x, int dtype, int B, int d, int f,
                   const uint16_t *wg, const uint16_t *wu, const uint16_t *wd,
                   const int32_t *ff_idx, int k_ff, double *s_out, double *y, int act)
{
    (void)f;
    double *s = (double *)malloc(sizeof(double) * (size_t)B * (size_t)(k_ff > 0 ? k_ff : 1));
#pragma omp parallel for schedule(static)
    for (int t = 0; t < k_ff; ++t) {
        int j = ff_idx[t];
        for (int b = 0; b < B; ++b) {
            double g = 0.0, u = 0.0;
            for (int i = 0; i < d; ++i) {
                double xi = XV(b, i);
                g += xi * WV(wg, j, i);
                u += xi * WV(wu, j, i);
            }
            s[(size_t)b * k_ff + t] = oracle_gate_act(g, act) * u;
        }
    }
    const int cblk = 256;
#pragma omp parallel for schedule(static)
    for (int c0 = 0; c0 < d; c0 += cblk) {
        int c1 = c0 + cblk < d ? c0 + cblk : d;
        for (int b = 0; b < B; ++b) {
            double *yb = y + (size_t)b * d;
            for (int c = c0; c < c1; ++c)
                yb[c] = 0.0;
            for (int t = 0; t < k_ff; ++t) {
                int j = ff_idx[t];
                double sj = s[(size_t)b * k_ff + t];
                for (int c = c0; c < c1; ++c)
                    yb[c] += sj * WV(wd, j, c);
            }
        }
    }
    if (s_out)
        memcpy(s_out, s, sizeof(double) * (size_t)B * (size_t)k_ff);
    free(s);
}

/* ------------------------------------------------------------------ */
/* Dense SwiGLU FFN (Sec. 2.1): y = (x W_up (.) SiLU(x W_gate)) W_down   */
/* ------------------------------------------------------------------ */
void oracle_ffn_dense(const uint16_t *x, int dtype, int B, int d, int f,
                      const uint16_t *wg, const uint16_t *wu, const uint16_t *wd,
                      double *y, int act)
{
    double *s = (double *)malloc(sizeof(double) * (size_t)B * (size_t)f);
#pragma omp parallel for schedule(static)
    for (int j = 0; j < f; ++j) {
        for (int b = 0; b < B; ++b) {
            double g = 0.0, u = 0.0;
            for (int i = 0; i < d; ++i) {
                double xi = XV(b, i);
                g += xi * WV(wg, j, i);
                u += xi * WV(wu, j, i);
            }
            s[(size_t)b * f + j] = u * oracle_gate_act(g, act);
        }
    }
    const int cblk = 256;
#pragma omp parallel for schedule(static)
    for (int c0 = 0; c0 < d; c0 += cblk) {
        int c1 = c0 + cblk < d ? c0 + cblk : d;
        for (int b = 0; b < B; ++b) {
            double *yb = y + (size_t)b * d;
            for (int c = c0; c < c1; ++c)
                yb[c] = 0.0;
            for (int j = 0; j < f; ++j) {
                double sj = s[(size_t)b * f + j];
                for (int c = c0; c < c1; ++c)
                    yb[c] += sj * WV(wd, j, c);
            }
        }
    }
    free(s);
}

/* ------------------------------------------------------------------ */
/* The whole sparse decode step: Stage 1 then Stage 2 (Sec. 4.1)        */
/* ------------------------------------------------------------------ */
/*
 * mask_override: NULL, or an ascending list of k_ff channels used instead of
 * the proxy's selection (to evaluate Stage 2 on another implementation's
 * mask).  Optional outputs (NULL to skip): in_idx_out [k_in], score_out [f],
 * ff_idx_out [k_ff].  y is [B][d].
 */
void oracle_ffn_sparse(const uint16_t *x, int dtype, int B, int d, int f,
                       const uint16_t *wg, const uint16_t *wu, const uint16_t *wd,
                       int proxy_kind, const int8_t *cg, const uint16_t *sg,
                       const int8_t *cu, const uint16_t *su, int group,
                       int k_in, int k_ff, const int32_t *mask_override,
                       int32_t *in_idx_out, double *score_out, int32_t *ff_idx_out,
                       double *y, int act)
{
    int32_t *in_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)k_in);
    int32_t *ff_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)k_ff);
    double *score = (double *)malloc(sizeof(double) * (size_t)f);
    if (mask_override) {
        memcpy(ff_idx, mask_override, sizeof(int32_t) * (size_t)k_ff);
        if (in_idx_out || score_out) {
            oracle_select_inputs(x, dtype, B, d, k_in, in_idx);
            oracle_proxy(x, dtype, B, d, f, in_idx, k_in, proxy_kind, cg, sg, cu, su, group,
                         wg, wu, NULL, NULL, NULL, score, act);
        }
    } else {
        oracle_select_inputs(x, dtype, B, d, k_in, in_idx);
        oracle_proxy(x, dtype, B, d, f, in_idx, k_in, proxy_kind, cg, sg, cu, su, group,
                     wg, wu, NULL, NULL, NULL, score, act);
        oracle_select_channels(score, f, k_ff, ff_idx);
    }
    oracle_stage2(x, dtype, B, d, f, wg, wu, wd, ff_idx, k_ff, NULL, y, act);
    if (in_idx_out)
        memcpy(in_idx_out, in_idx, sizeof(int32_t) * (size_t)k_in);
    if (score_out)
        memcpy(score_out, score, sizeof(double) * (size_t)f);
    if (ff_idx_out)
        memcpy(ff_idx_out, ff_idx, sizeof(int32_t) * (size_t)k_ff);
    free(in_idx);
    free(ff_idx);
    free(score);
}

/* ------------------------------------------------------------------ */
/* Threshold-mode selection (Sec. 4.1 masks with layer-wise thresholds,  */
/* App. A.6)                                                            */
/* ------------------------------------------------------------------ */
/* The indices i (ascending) whose key is at least tau; returns how many. */
int oracle_select_threshold(const double *key, int n, double tau, int32_t *idx_out)
{
    int c = 0;
    for (int i = 0; i < n; ++i)
        if (key[i] >= tau)
            idx_out[c++] = i;
    return c;
}

/* Input mask m_x with a threshold: keep channel i when a_i = max_b |x_{b,i}|
 * is at least tau_x (one set shared by the batch; for one row this is
 * |x_i| >= tau_x).  in_idx must hold d entries; returns k_in. */
int oracle_select_inputs_tau(const uint16_t *x, int dtype, int B, int d, double tau_x,
                             int32_t *in_idx)
{
    double *a = (double *)malloc(sizeof(double) * (size_t)d);
    for (int i = 0; i < d; ++i) {
        double m = 0.0;
        for (int b = 0; b < B; ++b) {
            double v = fabs(XV(b, i));
            if (v > m)
                m = v;
        }
        a[i] = m;
    }
    int k = oracle_select_threshold(a, d, tau_x, in_idx);
    free(a);
    return k;
}

/*
 * The decode step with thresholds instead of counts: m_x from tau_x, the
 * proxy on m_x, m_s = {j : score_j >= tau_s}, Stage 2 on m_s.  The counts
 * k_in and k_ff follow from the data.  mask_override (n_override entries,
 * ascending) replaces m_s as in oracle_ffn_sparse.  Outputs: in_idx_out [d],
 * score_out [f], ff_idx_out [f] (each may be NULL), counts[0] = k_in,
 * counts[1] = k_ff, y [B][d].
 */
void oracle_ffn_sparse_tau(const uint16_t *x, int dtype, int B, int d, int f,
                           const uint16_t *wg, const uint16_t *wu, const uint16_t *wd,
                           int proxy_kind, const int8_t *cg, const uint16_t *sg,
                           const int8_t *cu, const uint16_t *su, int group,
                           double tau_x, double tau_s,
                           const int32_t *mask_override, int n_override,
                           int32_t *in_idx_out, double *score_out, int32_t *ff_idx_out,
                           int32_t *counts, double *y, int act)
{
    int32_t *in_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)d);
    int32_t *ff_idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)f);
    double *score = (double *)malloc(sizeof(double) * (size_t)f);
    int k_in = oracle_select_inputs_tau(x, dtype, B, d, tau_x, in_idx);
    oracle_proxy(x, dtype, B, d, f, in_idx, k_in, proxy_kind, cg, sg, cu, su, group,
                 wg, wu, NULL, NULL, NULL, score, act);
    int k_ff;
    if (mask_override) {
        memcpy(ff_idx, mask_override, sizeof(int32_t) * (size_t)n_override);
        k_ff = n_override;
    } else {
        k_ff = oracle_select_threshold(score, f, tau_s, ff_idx);
    }
    oracle_stage2(x, dtype, B, d, f, wg, wu, wd, ff_idx, k_ff, NULL, y, act);
    if (in_idx_out)
        memcpy(in_idx_out, in_idx, sizeof(int32_t) * (size_t)k_in);
    if (score_out)
        memcpy(score_out, score, sizeof(double) * (size_t)f);
    if (ff_idx_out)
        memcpy(ff_idx_out, ff_idx, sizeof(int32_t) * (size_t)k_ff);
    counts[0] = k_in;
    counts[1] = k_ff;
    free(in_idx);
    free(ff_idx);
    free(score);
}

/* ------------------------------------------------------------------ */
/* Threshold calibration (App. A.7): a bounded sample per signal and    */
/* its empirical quantile                                               */
/* ------------------------------------------------------------------ */
/*
 * Reservoir of at most cap samples over a stream (Algorithm R).  The stream
 * item numbered t (0-based, *seen items came before this call) fills slot t
 * while t < cap; after that it replaces slot (r mod (t + 1)) when that index
 * is below cap.  r holds one uniform 64-bit random number per item, in
 * stream order (the caller draws them).  *seen grows by n.
 */
void oracle_reservoir_add(double *res, int cap, long long *seen, const double *v, int n,
                          const uint64_t *r)
{
    for (int i = 0; i < n; ++i) {
        long long t = *seen + i;
        if (t < cap) {
            res[t] = v[i];
        } else {
            uint64_t j = r[i] % (uint64_t)(t + 1);
            if (j < (uint64_t)cap)
                res[j] = v[i];
        }
    }
    *seen += n;
}

static int double_asc(const void *pa, const void *pb)
{
    double a = *(const double *)pa, b = *(const double *)pb;
    return (a > b) - (a < b);
}

/* Threshold for a target sparsity s (0 <= s < 1) of the rule |z| >= tau:
 * the sample value at 0-based position min(n - 1, floor(s n)) in ascending
 * order, so that about s n of the n samples fall below it. */
double oracle_quantile_threshold(const double *v, int n, double s)
{
    double *t = (double *)malloc(sizeof(double) * (size_t)n);
    memcpy(t, v, sizeof(double) * (size_t)n);
    qsort(t, (size_t)n, sizeof(double), double_asc);
    long long pos = (long long)floor(s * (double)n);
    if (pos > n - 1)
        pos = n - 1;
    if (pos < 0)
        pos = 0;
    double tau = t[pos];
    free(t);
    return tau;
}

/* ------------------------------------------------------------------ */
/* Cost model and sparsity allocation (Sec. 4.2)                        */
/* ------------------------------------------------------------------ */
/* Normalised cost: each dense projection costs 1 (a dense FFN costs 3); a
 * proxy projection costs alpha.  Stage 1 runs two proxy projections on a
 * (1 - s1) share of the inputs, Stage 2 three exact projections on a
 * (1 - s2) share of the channels. */
double oracle_prox_cost(double s1, double s2, double alpha)
{
    return 2.0 * alpha * (1.0 - s1) + 3.0 * (1.0 - s2);
}

/* Effective sparsity against the dense cost of 3. */
double oracle_effective_sparsity(double s1, double s2, double alpha)
{
    return 1.0 - oracle_prox_cost(s1, s2, alpha) / 3.0;
}

/* Allocation for a target effective sparsity e: s2 starts at s_ref and s1
 * takes the rest of the budget; when that s1 leaves [s1_min, s1_max] it is
 * clamped to the nearer bound and s2 is solved again from e. */
void oracle_allocate(double e, double alpha, double s_ref, double s1_min, double s1_max,
                     double *s1_out, double *s2_out)
{
    double s2 = s_ref;
    /* e = s2 - 2 alpha (1 - s1) / 3  =>  s1 = 1 - 3 (s2 - e) / (2 alpha) */
    double s1 = 1.0 - 3.0 * (s2 - e) / (2.0 * alpha);
    if (s1 < s1_min || s1 > s1_max) {
        s1 = s1 < s1_min ? s1_min : s1_max;
        s2 = e + 2.0 * alpha * (1.0 - s1) / 3.0;
    }
    *s1_out = s1;
    *s2_out = s2;
}

/* ------------------------------------------------------------------ */
/* Residual + RMSNorm between stacked layers (unit gain)                */
/* ------------------------------------------------------------------ */
/* out_b = r_b / sqrt(mean(r_b^2) + eps),  r_b = x_b + y_b.  out is [B][d]. */
void oracle_add_rmsnorm(const uint16_t *x, const uint16_t *y, int dtype, int B, int d,
                        double eps, double *out)
{
    for (int b = 0; b < B; ++b) {
        double ss = 0.0;
        for (int i = 0; i < d; ++i) {
            double r = XV(b, i) + oracle_half_to_double(y[(size_t)b * d + i], dtype);
            ss += r * r;
        }
        double inv = 1.0 / sqrt(ss / d + eps);
        for (int i = 0; i < d; ++i) {
            double r = XV(b, i) + oracle_half_to_double(y[(size_t)b * d + i], dtype);
            out[(size_t)b * d + i] = r * inv;
        }
    }
}

int oracle_max_threads(void)
{
#ifdef _OPENMP
    extern int omp_get_max_threads(void);
    return omp_get_max_threads();
#else
    return 1;
#endif
}
