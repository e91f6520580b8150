// C-ABI of libprox (declared in include/prox.h): argument validation on the
// host, workspace carving, and the launch sequence of each entry point.
#include <prox.h>

#include <cmath>
#include <mutex>

#include "kernels.hpp"

using namespace prox;

namespace {

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool dtype_ok(int dt) { return dt == PROX_F16 || dt == PROX_BF16; }

bool shape_ok(int d, int f) {
    return d >= PROX_MIN_D_MODEL && d <= PROX_MAX_D_MODEL && d % 128 == 0 && f >= 1 &&
           f <= PROX_MAX_D_FF;
}

int qbits_of(int fmt) {
    return fmt == PROX_Q_INT4 ? 4 : fmt == PROX_Q_INT8 ? 8 : fmt == PROX_Q_NONE ? 16 : 0;
}

bool proxy_shape_ok(int d, int fmt, int group) {
    if (fmt == PROX_Q_NONE) return group == d;   // one unit scale per channel
    return qbits_of(fmt) != 0 && group >= 128 && group % 128 == 0 && d % group == 0;
}

prox_status check_weights(const prox_weights *w) {
    if (!w || !w->w_gate || !w->w_up || !w->w_down) return PROX_ERR_INVALID;
    if (!dtype_ok(w->dtype)) return PROX_ERR_INVALID;
    if (w->act != PROX_ACT_SILU && w->act != PROX_ACT_GELU) return PROX_ERR_INVALID;
    if (!aligned(w->w_gate, 16) || !aligned(w->w_up, 16) || !aligned(w->w_down, 16))
        return PROX_ERR_INVALID;
    if (w->d_model < 1 || w->d_ff < 1) return PROX_ERR_INVALID;
    if (!shape_ok(w->d_model, w->d_ff)) return PROX_ERR_UNSUPPORTED;
    return PROX_OK;
}

bool w4_group_ok(int d, int group) { return group >= 128 && group % 128 == 0 && d % group == 0; }

prox_status check_w4(const prox_w4_weights *q) {
    if (!q || !q->blob || !aligned(q->blob, 256)) return PROX_ERR_INVALID;
    if (!dtype_ok(q->dtype)) return PROX_ERR_INVALID;
    if (q->act != PROX_ACT_SILU && q->act != PROX_ACT_GELU) return PROX_ERR_INVALID;
    if (q->d_model < 1 || q->d_ff < 1) return PROX_ERR_INVALID;
    if (!shape_ok(q->d_model, q->d_ff) || !w4_group_ok(q->d_model, q->group))
        return PROX_ERR_UNSUPPORTED;
    if (q->bytes < W4Layout(q->d_model, q->d_ff, q->group).total) return PROX_ERR_WORKSPACE;
    return PROX_OK;
}

// What the launch sequence needs of either weight format.
struct Model {
    int dtype, d, f, act;
    Stage2Weights s2;
};

Model model_of(const prox_weights *w) {
    return Model{w->dtype, w->d_model, w->d_ff, w->act,
                 Stage2Weights{w->w_gate, w->w_up, w->w_down, nullptr, nullptr, nullptr, 16, 0}};
}

Model model_of(const prox_w4_weights *q) {
    const W4Layout L(q->d_model, q->d_ff, q->group);
    const uint8_t *b = static_cast<const uint8_t *>(q->blob);
    auto sc = [&](int m) { return reinterpret_cast<const uint16_t *>(b + L.scales[m]); };
    return Model{q->dtype, q->d_model, q->d_ff, q->act,
                 Stage2Weights{b + L.codes[0], b + L.codes[1], b + L.codes[2], sc(0), sc(1), sc(2), 4,
                               q->group}};
}

prox_status hip_status(hipError_t e) { return e == hipSuccess ? PROX_OK : PROX_ERR_HIP; }

#define PROX_TRY(expr)                                \
    do {                                              \
        prox_status st_ = hip_status(expr);           \
        if (st_ != PROX_OK) return st_;               \
    } while (0)

struct Ws {
    float *scores, *ypart, *sbuf;
    int32_t *klist;
};

Ws carve(void *ws, int d, int f, int batch, int wq) {
    const WsLayout L(d, f, batch, wq);
    char *b = static_cast<char *>(ws);
    Ws w;
    w.scores = reinterpret_cast<float *>(b + L.scores);
    w.ypart = reinterpret_cast<float *>(b + L.ypart);
    w.klist = reinterpret_cast<int32_t *>(b + L.klist);
    w.sbuf = reinterpret_cast<float *>(b + L.sbuf);
    return w;
}

const char *const kStageNames[PROX_SPARSE_STAGES] = {"proxy_gemv_score",
                                                     "stage2_select_gate_up_down", "reduce_y"};

// Batch rows per Stage 2 launch for a call of `batch` rows.
int stage2_launch_rows(int d, int wq, int batch) {
    return batch > kStage2MaxNB && stage2_mfma_ok(d, wq) ? kStage2MfmaRows : stage2_rows(d, wq);
}

// Stage 2 and the final reduction, shared by the sparse and the dense FFN
// (scores == NULL: every channel).
prox_status stage2_and_reduce(const Model &m, const void *x, int batch, int k_ff,
                              const float *scores, uint8_t *mask, float *scores_copy, void *y,
                              const Ws &W, Select sel, hipEvent_t *events, hipStream_t stream) {
    const int d = m.d, f = m.f, dt = m.dtype;
    const uint16_t *xb = static_cast<const uint16_t *>(x);
    // With the threshold rule the kept count is found on the device: size the
    // grid for every channel (workgroups past the count get no channels).
    const int nwg = stage2_wgs(scores && !sel.tau_mode ? k_ff : f);
    const int ystride = ypart_rows(batch);
    // More than eight rows of 16-bit weights: the matrix-core path, 16 rows
    // per chunk (its tail too).
    const int rows = stage2_launch_rows(d, m.s2.wq, batch);
    if (rows == kStage2MfmaRows) {
        // Every 16-row chunk: gate/up on the matrix cores (s to the
        // workspace, kept list written by the first chunk), then the down
        // projection over kStage2DownGroups channel groups; the reduction
        // sums those groups' partial y.
        const int n_max = scores && !sel.tau_mode ? k_ff : f;
        for (int c0 = 0; c0 < batch; c0 += rows) {
            const int nb = batch - c0 < rows ? batch - c0 : rows;
            const int list_mode = !scores ? kListNone : c0 == 0 ? kListWrite : kListRead;
            PROX_TRY(launch_stage2_mfma(dt, xb + (size_t)c0 * d, nb, d, f, m.s2, scores, k_ff,
                                        mask, c0 == 0 ? scores_copy : nullptr, W.sbuf, nwg,
                                        c0 == 0 ? sel : Select{sel.tau_mode, sel.tau, nullptr},
                                        m.act, W.klist, list_mode, stream));
            PROX_TRY(launch_stage2_down(dt, nb, d, f, m.s2.wd, W.sbuf, scores ? W.klist : nullptr,
                                        n_max, W.ypart + (size_t)c0 * d, ystride, stream));
        }
        if (events) PROX_TRY(hipEventRecord(events[2], stream));
        PROX_TRY(launch_reduce(dt, W.ypart, kStage2DownGroups, batch, d, y, stream));
        if (events) PROX_TRY(hipEventRecord(events[3], stream));
        return PROX_OK;
    }
    for (int c0 = 0; c0 < batch; c0 += rows) {
        const int nb = batch - c0 < rows ? batch - c0 : rows;
        const int list_mode = !scores || rows >= batch ? kListNone
                              : c0 == 0             ? kListWrite
                                                    : kListRead;
        PROX_TRY(launch_stage2(dt, xb + (size_t)c0 * d, nb, d, f, m.s2, scores, k_ff, mask,
                               c0 == 0 ? scores_copy : nullptr, W.ypart + (size_t)c0 * d, ystride,
                               nwg, c0 == 0 ? sel : Select{sel.tau_mode, sel.tau, nullptr}, m.act,
                               W.klist, list_mode, stream));
    }
    if (events) PROX_TRY(hipEventRecord(events[2], stream));
    PROX_TRY(launch_reduce(dt, W.ypart, nwg, batch, d, y, stream));
    if (events) PROX_TRY(hipEventRecord(events[3], stream));
    return PROX_OK;
}

// Batch rows per matrix-core Stage-1 launch, or 0 for the dot-product kernel.
int stage1_mfma_rows(int d, int qbits, int group, int batch, int k_in) {
    return qbits == 4 && batch >= proxy_mfma_min_rows(d) ? proxy_mfma_rows(d, group, k_in) : 0;
}

// The selection of each stage: counts (k_in, k_ff) or thresholds.
struct Rules {
    int tau_mode;
    float tau_x, tau_s;
    int32_t *counts;   // threshold mode: [k_in, k_ff] realised, or NULL
};

// Host-side checks of a sparse call, workspace aside (no HIP call).  In
// threshold mode k_in becomes the proxy's list capacity (d) and k_ff 0.
prox_status sparse_check(const Model &m, const prox_proxy *p, const void *x, int batch,
                         int &k_in, int &k_ff, const Rules &rules, void *y, uint8_t *mask,
                         float *scores, hipEvent_t *events) {
    if (!p || !p->blob || !x || !y || !mask) return PROX_ERR_INVALID;
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(p->blob, 16) ||
        (scores && !aligned(scores, 4)))
        return PROX_ERR_INVALID;
    const int d = m.d, f = m.f;
    if (batch < 1 || batch > PROX_MAX_BATCH) return PROX_ERR_INVALID;
    if (rules.tau_mode) {
        if (std::isnan(rules.tau_x) || std::isnan(rules.tau_s)) return PROX_ERR_INVALID;
        if (rules.counts && !aligned(rules.counts, 4)) return PROX_ERR_INVALID;
        k_in = d;   // the proxy's list capacity
        k_ff = 0;
    } else if (k_in < 1 || k_in > d || k_ff < 1 || k_ff > f) {
        return PROX_ERR_INVALID;
    }
    if (!proxy_shape_ok(d, p->fmt, p->group)) return PROX_ERR_UNSUPPORTED;
    if (p->bytes < BlobLayout(d, f, qbits_of(p->fmt), p->group).total) return PROX_ERR_WORKSPACE;
    if (events)
        for (int i = 0; i <= PROX_SPARSE_STAGES; ++i)
            if (!events[i]) return PROX_ERR_INVALID;
    return PROX_OK;
}

// The launch sequence of a checked sparse call on a workspace of at least
// WsLayout(d, f, batch).total bytes.
prox_status sparse_run(const Model &m, const prox_proxy *p, const void *x, int batch, int k_in,
                       int k_ff, const Rules &rules, void *y, uint8_t *mask, uint8_t *in_mask,
                       float *scores, void *ws, hipEvent_t *events, hipStream_t stream) {
    const int d = m.d, f = m.f;
    const int qbits = qbits_of(p->fmt);
    const Ws W = carve(ws, d, f, batch, m.s2.wq);
    const int dt = m.dtype;
    if (events) PROX_TRY(hipEventRecord(events[0], stream));
    // Several batch rows with an INT4 proxy: the matrix-core kernel, which
    // reads the codes once for up to 16 rows; else the dot-product kernel.
    const int mfma_rows = stage1_mfma_rows(d, qbits, p->group, batch, k_in);
    const int pnb = mfma_rows ? mfma_rows : proxy_max_nb(d);
    for (int c0 = 0; c0 < batch; c0 += pnb) {
        const int nb = batch - c0 < pnb ? batch - c0 : pnb;
        const Select in_sel{rules.tau_mode, rules.tau_x, rules.counts};
        // With several matrix-core launches only the first selects; its list
        // of kept rows goes to the partial-y area, which Stage 2 writes only
        // after the last Stage 1 launch.
        const int list_mode = batch <= pnb ? kListNone : c0 == 0 ? kListWrite : kListRead;
        if (mfma_rows)
            PROX_TRY(launch_proxy_mfma(dt, x, batch, c0, nb, d, f, p->group, k_in, p->blob,
                                       c0 == 0 ? in_mask : nullptr, W.scores, c0 > 0, in_sel,
                                       m.act, reinterpret_cast<int32_t *>(W.ypart), list_mode,
                                       stream));
        else
            PROX_TRY(launch_proxy(dt, qbits, x, batch, c0, nb, d, f, p->group, k_in, p->blob,
                                  c0 == 0 ? in_mask : nullptr, W.scores, c0 > 0, in_sel, m.act,
                                  stream));
    }
    if (events) PROX_TRY(hipEventRecord(events[1], stream));
    const Select ff_sel{rules.tau_mode, rules.tau_s, rules.counts ? rules.counts + 1 : nullptr};
    return stage2_and_reduce(m, x, batch, k_ff, W.scores, mask, scores, y, W, ff_sel, events,
                             stream);
}

prox_status sparse_impl(const Model &m, const prox_proxy *p, const void *x, int batch,
                        int k_in, int k_ff, const Rules &rules, void *y, uint8_t *mask,
                        uint8_t *in_mask, float *scores, void *ws, size_t ws_bytes,
                        hipEvent_t *events, hipStream_t stream) {
    prox_status st = sparse_check(m, p, x, batch, k_in, k_ff, rules, y, mask, scores, events);
    if (st != PROX_OK) return st;
    if (!ws || !aligned(ws, 256)) return PROX_ERR_INVALID;
    if (ws_bytes < WsLayout(m.d, m.f, batch, m.s2.wq).total) return PROX_ERR_WORKSPACE;
    return sparse_run(m, p, x, batch, k_in, k_ff, rules, y, mask, in_mask, scores, ws, events,
                      stream);
}

prox_status dense_impl(const Model &m, const void *x, int batch, void *y, void *ws,
                       size_t ws_bytes, hipStream_t stream) {
    if (!x || !y || !ws) return PROX_ERR_INVALID;
    if (!aligned(x, 16) || !aligned(y, 16) || !aligned(ws, 256)) return PROX_ERR_INVALID;
    if (batch < 1 || batch > PROX_MAX_BATCH) return PROX_ERR_INVALID;
    if (ws_bytes < WsLayout(m.d, m.f, batch, m.s2.wq).total) return PROX_ERR_WORKSPACE;
    const Ws W = carve(ws, m.d, m.f, batch, m.s2.wq);
    return stage2_and_reduce(m, x, batch, m.f, nullptr, nullptr, nullptr, y, W,
                             Select{0, 0.0f, nullptr}, nullptr, stream);
}

}  // namespace

// Device scratch of prox_ffn_sparse_noalloc, one copy per GPU the library runs
// on, held until the process ends.  In host code `scratch` names a host-side
// stand-in: the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[PROX_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch[kMaxDevices];   // device address of `scratch` per device, or NULL

// The current device's copy of `scratch` (looked up on its first use).
prox_status scratch_of_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PROX_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return PROX_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return PROX_ERR_HIP;
        g_scratch[dev] = ptr;
    }
    *out = g_scratch[dev];
    return PROX_OK;
}

}  // namespace

extern "C" {

const char *prox_strerror(prox_status s) {
    switch (s) {
        case PROX_OK: return "ok";
        case PROX_ERR_INVALID: return "invalid argument";
        case PROX_ERR_UNSUPPORTED: return "unsupported shape or format";
        case PROX_ERR_WORKSPACE: return "workspace or proxy buffer too small";
        case PROX_ERR_HIP: return "HIP runtime or launch error";
    }
    return "unknown status";
}

const char *prox_sparse_stage_name(int i) {
    return i >= 0 && i < PROX_SPARSE_STAGES ? kStageNames[i] : nullptr;
}

int prox_stage1_mfma_rows(int d_model, prox_qfmt fmt, int group, int batch, int k_in) {
    if (d_model < 1 || d_model > kMaxDModel || !proxy_shape_ok(d_model, fmt, group) ||
        batch < 1 || batch > PROX_MAX_BATCH || k_in < 1 || k_in > d_model)
        return 0;
    return stage1_mfma_rows(d_model, qbits_of(fmt), group, batch, k_in);
}

int prox_stage2_rows(int d_model, int d_ff, int w4, int batch) {
    if (!shape_ok(d_model, d_ff) || batch < 1 || batch > PROX_MAX_BATCH) return 0;
    return stage2_launch_rows(d_model, w4 ? 4 : 16, batch);
}

size_t prox_proxy_bytes(int d_model, int d_ff, prox_qfmt fmt, int group) {
    if (!shape_ok(d_model, d_ff) || !proxy_shape_ok(d_model, fmt, group)) return 0;
    return BlobLayout(d_model, d_ff, qbits_of(fmt), group).total;
}

size_t prox_workspace_bytes(int d_model, int d_ff, int batch) {
    if (!shape_ok(d_model, d_ff) || batch < 1 || batch > PROX_MAX_BATCH) return 0;
    return WsLayout(d_model, d_ff, batch, 16).total;
}

size_t prox_w4_workspace_bytes(int d_model, int d_ff, int batch) {
    if (!shape_ok(d_model, d_ff) || batch < 1 || batch > PROX_MAX_BATCH) return 0;
    return WsLayout(d_model, d_ff, batch, 4).total;
}

prox_status prox_pack_proxy(const prox_weights *w, prox_proxy *p, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    if (!p || !p->blob || !aligned(p->blob, 16)) return PROX_ERR_INVALID;
    if (!proxy_shape_ok(w->d_model, p->fmt, p->group)) return PROX_ERR_UNSUPPORTED;
    const int qbits = qbits_of(p->fmt);
    if (p->bytes < BlobLayout(w->d_model, w->d_ff, qbits, p->group).total)
        return PROX_ERR_WORKSPACE;
    return hip_status(launch_pack(w->dtype, qbits, w->w_gate, w->w_up, w->d_model, w->d_ff,
                                  p->group, p->blob, stream));
}

prox_status prox_unpack_proxy(const prox_proxy *p, int d_model, int d_ff, int8_t *codes_gate,
                              uint16_t *scales_gate, int8_t *codes_up, uint16_t *scales_up,
                              hipStream_t stream) {
    if (!p || !p->blob || !codes_gate || !scales_gate || !codes_up || !scales_up)
        return PROX_ERR_INVALID;
    if (!aligned(p->blob, 16) || !aligned(scales_gate, 2) || !aligned(scales_up, 2))
        return PROX_ERR_INVALID;
    if (!shape_ok(d_model, d_ff) || !proxy_shape_ok(d_model, p->fmt, p->group) ||
        p->fmt == PROX_Q_NONE)
        return PROX_ERR_UNSUPPORTED;
    const int qbits = qbits_of(p->fmt);
    if (p->bytes < BlobLayout(d_model, d_ff, qbits, p->group).total) return PROX_ERR_WORKSPACE;
    return hip_status(launch_unpack(qbits, p->blob, d_model, d_ff, p->group, codes_gate,
                                    scales_gate, codes_up, scales_up, stream));
}

prox_status prox_ffn_dense(const prox_weights *w, const void *x, int batch, void *y, void *ws,
                           size_t ws_bytes, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    return dense_impl(model_of(w), x, batch, y, ws, ws_bytes, stream);
}

prox_status prox_ffn_sparse(const prox_weights *w, const prox_proxy *p, const void *x, int batch,
                            int k_in, int k_ff, void *y, uint8_t *mask, uint8_t *in_mask,
                            float *scores, void *ws, size_t ws_bytes, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    return sparse_impl(model_of(w), p, x, batch, k_in, k_ff, Rules{0, 0.0f, 0.0f, nullptr}, y,
                       mask, in_mask, scores, ws, ws_bytes, nullptr, stream);
}

prox_status prox_ffn_sparse_noalloc(const prox_weights *w, const prox_proxy *p, const void *x,
                                    int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                                    uint8_t *in_mask, float *scores, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    const Model m = model_of(w);
    const Rules rules{0, 0.0f, 0.0f, nullptr};
    st = sparse_check(m, p, x, batch, k_in, k_ff, rules, y, mask, scores, nullptr);
    if (st != PROX_OK) return st;
    if (WsLayout(m.d, m.f, batch, m.s2.wq).total > PROX_NOALLOC_SCRATCH_BYTES) return PROX_ERR_WORKSPACE;
    void *ws = nullptr;
    st = scratch_of_current_device(&ws);
    if (st != PROX_OK) return st;
    return sparse_run(m, p, x, batch, k_in, k_ff, rules, y, mask, in_mask, scores, ws, nullptr,
                      stream);
}

size_t prox_noalloc_max_bytes(void) { return PROX_NOALLOC_SCRATCH_BYTES; }

prox_status prox_ffn_sparse_tau(const prox_weights *w, const prox_proxy *p, const void *x,
                                int batch, float tau_x, float tau_s, void *y, uint8_t *mask,
                                uint8_t *in_mask, float *scores, int32_t *counts, void *ws,
                                size_t ws_bytes, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    return sparse_impl(model_of(w), p, x, batch, 0, 0, Rules{1, tau_x, tau_s, counts}, y, mask,
                       in_mask, scores, ws, ws_bytes, nullptr, stream);
}

prox_status prox_ffn_sparse_staged(const prox_weights *w, const prox_proxy *p, const void *x,
                                   int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                                   uint8_t *in_mask, float *scores, void *ws, size_t ws_bytes,
                                   hipEvent_t *events, hipStream_t stream) {
    if (!events) return PROX_ERR_INVALID;
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    return sparse_impl(model_of(w), p, x, batch, k_in, k_ff, Rules{0, 0.0f, 0.0f, nullptr}, y,
                       mask, in_mask, scores, ws, ws_bytes, events, stream);
}

size_t prox_w4_bytes(int d_model, int d_ff, int group) {
    if (!shape_ok(d_model, d_ff) || !w4_group_ok(d_model, group)) return 0;
    return W4Layout(d_model, d_ff, group).total;
}

prox_status prox_pack_w4(const prox_weights *w, const prox_w4_weights *q, hipStream_t stream) {
    prox_status st = check_weights(w);
    if (st != PROX_OK) return st;
    st = check_w4(q);
    if (st != PROX_OK) return st;
    if (q->dtype != w->dtype || q->d_model != w->d_model || q->d_ff != w->d_ff)
        return PROX_ERR_INVALID;
    return hip_status(launch_pack_w4(w->dtype, w->w_gate, w->w_up, w->w_down, w->d_model,
                                     w->d_ff, q->group, q->blob, stream));
}

prox_status prox_unpack_w4(const prox_w4_weights *q, int matrix, int8_t *codes,
                           uint16_t *scales, hipStream_t stream) {
    prox_status st = check_w4(q);
    if (st != PROX_OK) return st;
    if (matrix < 0 || matrix > 2 || !codes || !scales || !aligned(scales, 2))
        return PROX_ERR_INVALID;
    return hip_status(launch_unpack_w4(q->blob, q->d_model, q->d_ff, q->group, matrix, codes,
                                       scales, stream));
}

prox_status prox_ffn_dense_w4(const prox_w4_weights *q, const void *x, int batch, void *y,
                              void *ws, size_t ws_bytes, hipStream_t stream) {
    prox_status st = check_w4(q);
    if (st != PROX_OK) return st;
    return dense_impl(model_of(q), x, batch, y, ws, ws_bytes, stream);
}

prox_status prox_ffn_sparse_tau_w4(const prox_w4_weights *q, const prox_proxy *p, const void *x,
                                   int batch, float tau_x, float tau_s, void *y, uint8_t *mask,
                                   uint8_t *in_mask, float *scores, int32_t *counts, void *ws,
                                   size_t ws_bytes, hipStream_t stream) {
    prox_status st = check_w4(q);
    if (st != PROX_OK) return st;
    return sparse_impl(model_of(q), p, x, batch, 0, 0, Rules{1, tau_x, tau_s, counts}, y, mask,
                       in_mask, scores, ws, ws_bytes, nullptr, stream);
}

prox_status prox_ffn_sparse_w4(const prox_w4_weights *q, const prox_proxy *p, const void *x,
                               int batch, int k_in, int k_ff, void *y, uint8_t *mask,
                               uint8_t *in_mask, float *scores, void *ws, size_t ws_bytes,
                               hipEvent_t *events, hipStream_t stream) {
    prox_status st = check_w4(q);
    if (st != PROX_OK) return st;
    return sparse_impl(model_of(q), p, x, batch, k_in, k_ff, Rules{0, 0.0f, 0.0f, nullptr}, y,
                       mask, in_mask, scores, ws, ws_bytes, events, stream);
}

prox_status prox_add_rmsnorm(const void *x, const void *y, int batch, int d_model,
                             prox_dtype dtype, float eps, void *out, hipStream_t stream) {
    if (!x || !y || !out || !dtype_ok(dtype)) return PROX_ERR_INVALID;
    if (!aligned(x, 2) || !aligned(y, 2) || !aligned(out, 2)) return PROX_ERR_INVALID;
    if (batch < 1 || batch > PROX_MAX_BATCH || d_model < 1) return PROX_ERR_INVALID;
    if (d_model > PROX_MAX_D_MODEL) return PROX_ERR_UNSUPPORTED;
    if (!(eps >= 0.0f)) return PROX_ERR_INVALID;
    return hip_status(launch_add_rmsnorm(dtype, x, y, batch, d_model, eps, out, stream));
}

}  // extern "C"
