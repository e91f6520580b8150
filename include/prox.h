/*
 * prox.h -- C-ABI of libprox.so: the Prox sparse SwiGLU FFN decode step
 * (two-stage, training-free activation sparsity; arxiv 2607.27591) on AMD
 * MI355X (gfx950).
 *
 * Notation follows the paper (Sec. 2.1): W_gate, W_up in R^{d x f},
 * W_down in R^{f x d}, u = x W_up, h = SiLU(x W_gate), s = u (.) h.
 * d = d_model, f = d_ff, B = batch rows decoded together.
 *
 * Conventions shared by every entry point:
 *  - Pointers named as device pointers must point to device memory that the
 *    caller allocated and owns; the library never allocates, frees or
 *    synchronises inside prox_ffn_* / prox_pack_proxy / prox_add_rmsnorm.
 *    All work is enqueued on the given HIP stream (0 = the null stream) and
 *    completes asynchronously.
 *  - Arguments are validated on the host before any HIP call; on failure
 *    nothing is enqueued and a status other than PROX_OK is returned.  No
 *    entry point aborts or throws.
 *  - Calls are reentrant when they use distinct workspaces.  Two calls that
 *    share a workspace must be ordered on one stream.
 *  - 16-bit tensors are IEEE fp16 or bf16 bit patterns (prox_dtype).  Inputs
 *    must be finite.
 */
#ifndef PROX_H
#define PROX_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* The enums are int-sized.  In C++ they get int as their fixed underlying
 * type, so any int a C caller passes is a valid value there too (the entry
 * points reject the ones outside the enumerators). */
#ifdef __cplusplus
#define PROX_ENUM_INT : int
#else
#define PROX_ENUM_INT
#endif

typedef enum PROX_ENUM_INT {
    PROX_OK = 0,
    PROX_ERR_INVALID = 1,     /* null pointer, size out of range, misalignment */
    PROX_ERR_UNSUPPORTED = 2, /* well-formed but outside the supported shapes */
    PROX_ERR_WORKSPACE = 3,   /* workspace (or proxy blob) smaller than required */
    PROX_ERR_HIP = 4          /* a HIP launch or runtime call failed */
} prox_status;

typedef enum PROX_ENUM_INT { PROX_F16 = 0, PROX_BF16 = 1 } prox_dtype;

/* Gate activation: SwiGLU (SiLU(z) = z / (1 + e^-z), Sec. 2.1) or GeGLU
 * (GELU(z) = z * Phi(z) = z (1 + erf(z / sqrt 2)) / 2, the gated FFN of the
 * Gemma models the paper mentions).  Applied to the proxy (Stage 1) and to
 * the exact gate (Stage 2) alike. */
typedef enum PROX_ENUM_INT { PROX_ACT_SILU = 0, PROX_ACT_GELU = 1 } prox_act;

/* Proxy formats.  PROX_Q_NONE keeps W_gate, W_up themselves, in the weights'
 * 16-bit dtype (the unquantised-proxy ablation, W~ = W; also the reference
 * point of the proxy-cost ratio alpha of Sec. 4.2); it takes group = d_model
 * and has no codes to unpack. */
typedef enum PROX_ENUM_INT { PROX_Q_INT8 = 0, PROX_Q_INT4 = 1, PROX_Q_NONE = 2 } prox_qfmt;

/* Supported sizes.  Batches past the rows one launch takes (Stage 1: 4 on the
 * dot-product kernel, 8 or 16 on the matrix cores; Stage 2: 16 per chunk on
 * the matrix-core path, see prox_stage2_rows, else 8, fewer for INT4 base
 * weights on wide d_model) run as several launches on the same stream:
 * Stage 1 takes the max of the scores over them, Stage 2 writes disjoint rows
 * of the partial sums, so the result does not depend on the split.  Each
 * Stage 2 launch or chunk reads the kept rows again. */
#define PROX_MAX_BATCH 64
#define PROX_MIN_D_MODEL 128
#define PROX_MAX_D_MODEL 16384   /* multiple of 128 */
#define PROX_MAX_D_FF 65536
#define PROX_SPARSE_STAGES 3     /* events recorded by prox_ffn_sparse_staged */

/*
 * Original FFN weights (Sec. 2.1), all three channel-major: row j holds the
 * d entries that meet intermediate channel j, so a kept channel reads three
 * contiguous rows.
 *   w_gate[j*d + i] = W_gate[i, j]   (nn.Linear gate_proj.weight)
 *   w_up  [j*d + i] = W_up[i, j]     (nn.Linear up_proj.weight)
 *   w_down[j*d + c] = W_down[j, c]   (nn.Linear down_proj.weight, transposed)
 * Device pointers, 16-byte aligned, read-only, owned by the caller.
 */
typedef struct {
    int d_model;
    int d_ff;
    prox_dtype dtype;
    const void *w_gate;
    const void *w_up;
    const void *w_down;
    prox_act act;   /* PROX_ACT_SILU unless the FFN is a GeGLU */
} prox_weights;

/*
 * Quantised proxy copies W~_gate, W~_up of Stage 1 (Sec. 4.3): symmetric
 * quantisation, one fp16 scale per (output channel, group of `group`
 * consecutive input channels); group == d_model is one scale per channel.
 *   sigma = fp16_RNE(amax / qmax), q = clamp(round_half_even(w / sigma),
 *   -qmax, qmax), qmax = 7 (INT4) or 127 (INT8), q = 0 when sigma == 0.
 * `blob` is an opaque, device-resident, caller-allocated buffer of at least
 * prox_proxy_bytes() bytes (16-byte aligned).  It starts with a 256-byte
 * header (magic "PRXB", version, fmt, group, d_model, d_ff, tile width) so a
 * saved blob describes itself.  group must be a multiple of 128 dividing
 * d_model.
 */
typedef struct {
    prox_qfmt fmt;
    int group;
    void *blob;
    size_t bytes;
} prox_proxy;

/* Bytes of the proxy blob for this shape; 0 if the shape is unsupported. */
size_t prox_proxy_bytes(int d_model, int d_ff, prox_qfmt fmt, int group);

/*
 * Offline preparation (Sec. 4.3): quantise w->w_gate and w->w_up into
 * p->blob.  Bit-exact and deterministic.  p->fmt, p->group, p->blob and
 * p->bytes are inputs.
 */
prox_status prox_pack_proxy(const prox_weights *w, prox_proxy *p, hipStream_t stream);

/*
 * Inverse view of a packed blob, for inspection and tests: writes the integer
 * codes q (int8, [d_ff][d_model], channel-major like the weights) and the
 * fp16 scale bit patterns ([d_ff][d_model/group]) of both proxies.  All four
 * outputs are device pointers.
 */
prox_status prox_unpack_proxy(const prox_proxy *p, int d_model, int d_ff, int8_t *codes_gate,
                              uint16_t *scales_gate, int8_t *codes_up, uint16_t *scales_up,
                              hipStream_t stream);

/* Workspace bytes needed by prox_ffn_sparse / prox_ffn_dense (16-bit
 * weights) for this shape and batch; 0 if unsupported.  The workspace needs
 * no initialisation.  It holds the proxy scores, the kept-channel list and
 * the partial y of Stage 2: one row set per Stage 2 workgroup (256), or, for
 * more than 8 batch rows at d_model >= 4096, per kept-channel group of the
 * matrix-core down projection (64) plus s of the kept channels.  INT4 base
 * weights always take the 256 row sets: see prox_w4_workspace_bytes. */
size_t prox_workspace_bytes(int d_model, int d_ff, int batch);

/*
 * Which Stage-1 kernel a sparse call takes (for inspection and tests): the
 * batch rows one launch of the matrix-core kernel covers for this shape, or 0
 * when Stage 1 runs on the dot-product kernel (an INT8 or unquantised proxy,
 * fewer than three batch rows up to d_model 4096 or fewer than five above, a
 * kept-input list too long for the LDS, or an unsupported shape).  k_in is the kept-input count; the threshold entry
 * point sizes its list for k_in = d_model.  Host only, no HIP calls.  The two
 * kernels compute the same proxy in a different fp32 summation order.
 */
int prox_stage1_mfma_rows(int d_model, prox_qfmt fmt, int group, int batch, int k_in);

/*
 * Which Stage-2 path a call takes (for inspection and tests): the batch rows
 * one Stage-2 pass covers.  16 means the matrix-core path (more than eight
 * batch rows of 16-bit weights with d_model >= 4096): every chunk of up to 16
 * rows, the batch tail included, runs gate/up as 16x16x16 MFMAs and then the
 * down projection as a second launch, so the three matrices are read once per
 * 16 rows.  Otherwise one fused VALU launch per up to 8 rows (fewer for INT4
 * weights, w4 != 0, at wide d_model).  0 for an unsupported shape or batch.
 * Host only, no HIP calls.  Both paths give the same kept set; y differs only
 * in fp32 summation order.
 */
int prox_stage2_rows(int d_model, int d_ff, int w4, int batch);

/*
 * Dense SwiGLU FFN (Sec. 2.1):  y = (x W_up (.) SiLU(x W_gate)) W_down.
 *   x: device [batch][d_model], w->dtype;  y: device [batch][d_model], same
 *   dtype, rounded once (round-to-nearest-even) from fp32 accumulation.
 *   ws: device workspace of ws_bytes >= prox_workspace_bytes(), 256-byte
 *   aligned.  1 <= batch <= PROX_MAX_BATCH.
 */
prox_status prox_ffn_dense(const prox_weights *w, const void *x, int batch, void *y, void *ws,
                           size_t ws_bytes, hipStream_t stream);

/*
 * The Prox sparse decode step (Sec. 4.1), with the per-token top-k rule of
 * App. A.6 for both masks:
 *  Stage 1  m_x = the k_in input channels with the largest a_i = max_b |x_{b,i}|
 *           (one set shared by the batch; ties go to the lower index);
 *           g~ = Pi_in(x, W~_gate, m_x), u~ = Pi_in(x, W~_up, m_x) in fp32;
 *           score_j = max_b |SiLU(g~_{b,j}) u~_{b,j}|;
 *           m_s = the k_ff channels with the largest score (ties to the lower
 *           index), shared by the batch.
 *  Stage 2  for j in m_s, over all d inputs: g_j, u_j exact (fp32 accumulation
 *           of the original weights), s_j = SiLU(g_j) u_j kept in fp32;
 *           y = sum_{j in m_s} s_j W_down[j, :], rounded once to the dtype.
 * Arguments:
 *   x      device [batch][d_model] (w->dtype), 16-byte aligned
 *   y      device [batch][d_model] output (w->dtype), 16-byte aligned
 *   mask   device uint8 [d_ff] output: 1 for channels in m_s, else 0
 *   in_mask  device uint8 [d_model] output for m_x, or NULL
 *   scores device float [d_ff] output of score_j, or NULL
 *   1 <= k_in <= d_model, 1 <= k_ff <= d_ff, 1 <= batch <= PROX_MAX_BATCH.
 */
prox_status prox_ffn_sparse(const prox_weights *w, const prox_proxy *p, const void *x, int batch,
                            int k_in, int k_ff, void *y, uint8_t *mask, uint8_t *in_mask,
                            float *scores, void *ws, size_t ws_bytes, hipStream_t stream);

/*
 * prox_ffn_sparse without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The call allocates nothing and calls no
 * allocating routine: it runs the same kernels as prox_ffn_sparse on the
 * library's own device scratch, a file-scope array of
 * PROX_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU, created with the library's code
 * object and held until the process ends.
 *   Arguments: as prox_ffn_sparse, without ws / ws_bytes.
 *   Limit: prox_workspace_bytes(d_model, d_ff, batch) must not exceed
 *   PROX_NOALLOC_SCRATCH_BYTES (e.g. 8192 x 28672 up to batch 2, d_model
 *   16384 at batch 1), else PROX_ERR_WORKSPACE before any HIP call.
 *   The first call on a device looks up that device's copy of the scratch
 *   (hipGetSymbolAddress); a failure there returns PROX_ERR_HIP.
 *   Every call on one GPU shares that GPU's scratch, which keeps the last
 *   call's contents (the kernels need none of it initialised): calls that
 *   overlap on one GPU (other streams, other host threads) race, so order
 *   them, e.g. on one stream.
 * Results are bitwise those of prox_ffn_sparse for the same arguments.
 */
#define PROX_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
prox_status prox_ffn_sparse_noalloc(const prox_weights *w, const prox_proxy *p, const void *x,
                                    int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                                    uint8_t *in_mask, float *scores, hipStream_t stream);

/* PROX_NOALLOC_SCRATCH_BYTES of the built library (host only). */
size_t prox_noalloc_max_bytes(void);

/*
 * The decode step with the paper's layer-wise thresholds in place of counts
 * (Sec. 4.1 masks, App. A.6 rule; thresholds calibrated offline, App. A.7):
 *   m_x = { i : max_b |x_{b,i}| >= tau_x }   (one set shared by the batch)
 *   m_s = { j : score_j >= tau_s },  score_j = max_b |SiLU(g~_{b,j}) u~_{b,j}|
 * Stage 1 and Stage 2 otherwise as prox_ffn_sparse.  The kept counts follow
 * from the data and may be 0 (then y = 0) up to d_model and d_ff.
 *   tau_x, tau_s  fp32 thresholds, not NaN (+inf keeps nothing, <= 0 keeps all)
 *   counts   device int32 [2] output (4-byte aligned), or NULL:
 *            counts[0] = |m_x|, counts[1] = |m_s| of this call
 *   x, y, mask, in_mask, scores, ws, ws_bytes, stream: as prox_ffn_sparse.
 * Comparisons are fp32: |x| exactly, the scores as the fp32 proxy computes
 * them.  Returns PROX_ERR_INVALID for a NaN threshold or a misaligned counts.
 */
prox_status prox_ffn_sparse_tau(const prox_weights *w, const prox_proxy *p, const void *x,
                                int batch, float tau_x, float tau_s, void *y, uint8_t *mask,
                                uint8_t *in_mask, float *scores, int32_t *counts, void *ws,
                                size_t ws_bytes, hipStream_t stream);

/*
 * prox_ffn_sparse with timing: `events` holds PROX_SPARSE_STAGES + 1 caller-
 * created HIP events, recorded on `stream` before the first stage and after
 * each stage: (0) input top-k + proxy GEMV + score, (1) channel top-k +
 * gate/up + down partial sums, (2) reduction of the partial sums into y.
 * Same kernels and launch configuration as prox_ffn_sparse.
 */
prox_status prox_ffn_sparse_staged(const prox_weights *w, const prox_proxy *p, const void *x,
                                   int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                                   uint8_t *in_mask, float *scores, void *ws, size_t ws_bytes,
                                   hipEvent_t *events, hipStream_t stream);

/* Name of stage i of prox_ffn_sparse_staged (static string), or NULL. */
const char *prox_sparse_stage_name(int i);

/*
 * Low-bit base weights combined with the sparse step (W4A16): Sec. 5.1 finds
 * the two complementary and leaves kernels that do both to future work.
 * Stage 2 reads an INT4 copy of W_gate, W_up and W_down instead of the 16-bit
 * rows; Stage 1 is unchanged (the proxy is packed from the 16-bit weights as
 * usual).  Each matrix is quantised like the proxy (Sec. 4.3): per (channel,
 * group of `group` consecutive inputs along d_model) a scale sigma = amax / 7
 * rounded to fp16, codes q = round-half-even(w / sigma) clamped to [-7, 7],
 * so the weight (j, i) stands for sigma_{j,g(i)} q_{j,i}.  Stage 2 computes
 *   g_j = sum_g sigma^gate_{j,g} sum_{i in g} x_i q^gate_{j,i}   (u_j alike),
 *   y   = sum_{j in m_s} s_j sum_c sigma^down_{j,g(c)} q^down_{j,c} e_c,
 * with fp32 accumulation, y rounded once to the dtype.
 * The blob (device, 256-byte aligned, prox_w4_bytes() bytes) holds, for
 * gate, up and down in turn, the codes [d_ff][d_model / 2] (input i of
 * channel j in byte i / 2: the low nibble when i is even, as q + 8), then the
 * three scale arrays [d_ff][d_model / group] of fp16 bit patterns; every
 * array starts on a 256-byte boundary.  All fields are inputs.
 */
typedef struct {
    int dtype;     /* prox_dtype of x and y (and of the weights packed from) */
    int d_model;
    int d_ff;
    int group;     /* a multiple of 128 that divides d_model */
    int act;       /* prox_act */
    void *blob;
    size_t bytes;
} prox_w4_weights;

/* Bytes of the W4 blob for this shape; 0 if unsupported. */
size_t prox_w4_bytes(int d_model, int d_ff, int group);

/* Quantise w's three matrices into q->blob (bit-exact, deterministic).
 * q->dtype, d_model, d_ff must equal w's. */
prox_status prox_pack_w4(const prox_weights *w, const prox_w4_weights *q, hipStream_t stream);

/* Inverse view of matrix 0 (gate), 1 (up) or 2 (down), for inspection and
 * tests: codes int8 [d_ff][d_model] and scales [d_ff][d_model / group],
 * both device pointers. */
prox_status prox_unpack_w4(const prox_w4_weights *q, int matrix, int8_t *codes,
                           uint16_t *scales, hipStream_t stream);

/* Workspace bytes needed by the calls on INT4 base weights (the *_w4 calls)
 * for this shape and batch (>= prox_workspace_bytes; equal up to 8 rows);
 * 0 if unsupported.  No initialisation needed. */
size_t prox_w4_workspace_bytes(int d_model, int d_ff, int batch);

/* The dense FFN on the INT4 weights (every channel; the W4 baseline).
 * x, y, batch as prox_ffn_dense; ws: ws_bytes >= prox_w4_workspace_bytes(),
 * 256-byte aligned. */
prox_status prox_ffn_dense_w4(const prox_w4_weights *q, const void *x, int batch, void *y,
                              void *ws, size_t ws_bytes, hipStream_t stream);

/* The sparse decode step of prox_ffn_sparse with Stage 2 on the INT4 weights.
 * p is the proxy of the same FFN.  events: NULL, or PROX_SPARSE_STAGES + 1
 * caller-created events recorded as in prox_ffn_sparse_staged.  ws: ws_bytes
 * >= prox_w4_workspace_bytes().  Other arguments as prox_ffn_sparse. */
prox_status prox_ffn_sparse_w4(const prox_w4_weights *q, const prox_proxy *p, const void *x,
                               int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                               uint8_t *in_mask, float *scores, void *ws, size_t ws_bytes,
                               hipEvent_t *events, hipStream_t stream);

/* The threshold-mode step of prox_ffn_sparse_tau with Stage 2 on the INT4
 * weights.  Arguments as prox_ffn_sparse_tau, with q in place of w and ws_bytes
 * >= prox_w4_workspace_bytes(). */
prox_status prox_ffn_sparse_tau_w4(const prox_w4_weights *q, const prox_proxy *p, const void *x,
                                   int batch, float tau_x, float tau_s, void *y, uint8_t *mask,
                                   uint8_t *in_mask, float *scores, int32_t *counts, void *ws,
                                   size_t ws_bytes, hipStream_t stream);

/*
 * Threshold calibration (App. A.7), host code only (no HIP calls; all
 * pointers are host memory).  Offline, a layer's thresholds come from
 * calibration activations run through the earlier layers with their final
 * thresholds (Alg. 1): each signal (|x| for tau_x, |s~| = the proxy scores
 * of one token for tau_s) is kept in a bounded sample, and the threshold is
 * that sample's empirical quantile at the target sparsity.
 *
 * prox_reservoir_add: offers values[0..n) to a reservoir of capacity cap
 * (Algorithm R).  *seen counts the values offered before this call and grows
 * by n; the reservoir holds min(cap, *seen) values.  Offer number t fills
 * slot t while t < cap, then replaces slot (draws[i] mod (t + 1)) when that
 * index is below cap.  draws: one uniform 64-bit random number per value,
 * drawn by the caller.  PROX_ERR_INVALID for NULL pointers (values/draws may
 * be NULL when n == 0) or cap == 0.
 *
 * prox_quantile_threshold: *tau = the sample value at ascending position
 * min(n - 1, floor(sparsity * n)), so that about sparsity * n of the n
 * samples lie below it and the rule |z| >= tau keeps the rest.
 * PROX_ERR_INVALID for n == 0, sparsity outside [0, 1), a NaN sample or NULL
 * pointers.
 */
prox_status prox_reservoir_add(float *reservoir, size_t cap, uint64_t *seen, const float *values,
                               size_t n, const uint64_t *draws);
prox_status prox_quantile_threshold(const float *samples, size_t n, double sparsity, float *tau);

/*
 * Sparsity allocation between the two stages (Sec. 4.2), host code only.
 * A dense FFN costs 3 (one per projection); a proxy projection costs alpha
 * (the paper rounds its measured ratios to 1/3).
 *
 * prox_effective_sparsity: e = 1 - (2 alpha (1 - s1) + 3 (1 - s2)) / 3.
 *
 * prox_allocate_sparsity: (s1, s2) for a target e.  s2 = s_ref (the paper
 * uses 0.7) and s1 takes the remaining budget; if that s1 leaves
 * [s1_min, s1_max] (the paper uses [0, 0.7]) it is clamped to the nearer
 * bound and s2 is solved again from e.  PROX_ERR_INVALID for alpha <= 0,
 * s1_min > s1_max, a NaN argument or a NULL output.
 */
double prox_effective_sparsity(double s1, double s2, double alpha);
prox_status prox_allocate_sparsity(double e, double alpha, double s_ref, double s1_min,
                                   double s1_max, double *s1, double *s2);

/*
 * Residual + unit-gain RMSNorm between stacked FFN layers:
 *   out_b = r_b / sqrt(mean(r_b^2) + eps),  r_b = x_b + y_b  (fp32),
 * rounded once to the dtype.  x, y, out: device [batch][d_model]; out may
 * alias x.
 */
prox_status prox_add_rmsnorm(const void *x, const void *y, int batch, int d_model,
                             prox_dtype dtype, float eps, void *out, hipStream_t stream);

/* Static description of a status code. */
const char *prox_strerror(prox_status status);

#ifdef __cplusplus
}
#endif

#endif /* PROX_H */
