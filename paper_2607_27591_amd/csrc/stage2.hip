// Stage 2 exact sparse computation (Sec. 4.1 Stage 2) and the dense FFN
// (Sec. 2.1), which runs the same kernels over every channel.
//
//  gate/up : for each kept channel j (one wave per channel), the contiguous
//            rows W_gate[:, j] and W_up[:, j] are streamed with 16-byte loads
//            and dotted with x (staged in LDS) by dot2 instructions in fp32;
//            s_j = SiLU(g_j) u_j is kept in fp32.
//  down    : y = sum_j s_j W_down[j, :] as a split-K GEMV.  A workgroup owns
//            kDownCols output columns and one slice of the kept channels; its
//            8 waves split the slice and are summed in LDS in wave order, the
//            slices are summed by the last workgroup to arrive in slice order,
//            and y is rounded once.  Deterministic: no floating-point atomics.
#include "common.hpp"
#include "kernels.hpp"

namespace prox {

constexpr int kGuThreads = 512;
constexpr int kDownThreads = kDownWaves * kWave;

template <int NB, int DT>
__global__ __launch_bounds__(kGuThreads) void gateup_kernel(
    const uint16_t *__restrict__ x, int nb, int d, const uint16_t *__restrict__ wg,
    const uint16_t *__restrict__ wu, const int *__restrict__ ff_idx, int n_ch,
    float *__restrict__ s_out, int s_stride, Ctrl *__restrict__ ctrl_reset) {
    extern __shared__ uint4 xs_vec[];   // [NB][d / 8] 16-byte vectors of x
    const int nvec = d / 8;
    for (int e = threadIdx.x; e < NB * nvec; e += kGuThreads) {
        const int b = e / nvec, vv = e % nvec;
        xs_vec[e] = b < nb ? reinterpret_cast<const uint4 *>(x + (size_t)b * d)[vv]
                           : make_uint4(0, 0, 0, 0);
    }
    if (ctrl_reset && blockIdx.x == 0)
        for (int i = threadIdx.x; i < 256; i += kGuThreads) ctrl_reset->down_count[i] = 0;
    __syncthreads();

    const int lane = lane_id();
    const int waves = gridDim.x * (kGuThreads / kWave);
    constexpr int U = 4;
    for (int t = blockIdx.x * (kGuThreads / kWave) + threadIdx.x / kWave; t < n_ch; t += waves) {
        const int j = ff_idx ? ff_idx[t] : t;
        const uint4 *rg = reinterpret_cast<const uint4 *>(wg + (size_t)j * d);
        const uint4 *ru = reinterpret_cast<const uint4 *>(wu + (size_t)j * d);
        float ag[NB], au[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) ag[b] = au[b] = 0.0f;
        for (int v0 = lane; v0 < nvec; v0 += kWave * U) {
            uint4 gv[U], uv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (v0 + u * kWave < nvec) {
                    gv[u] = load_stream16(rg + v0 + u * kWave);
                    uv[u] = load_stream16(ru + v0 + u * kWave);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (v0 + u * kWave < nvec) {
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const uint4 xv = xs_vec[b * nvec + v0 + u * kWave];
                        ag[b] = dot2<DT>(xv.x, gv[u].x, ag[b]);
                        ag[b] = dot2<DT>(xv.y, gv[u].y, ag[b]);
                        ag[b] = dot2<DT>(xv.z, gv[u].z, ag[b]);
                        ag[b] = dot2<DT>(xv.w, gv[u].w, ag[b]);
                        au[b] = dot2<DT>(xv.x, uv[u].x, au[b]);
                        au[b] = dot2<DT>(xv.y, uv[u].y, au[b]);
                        au[b] = dot2<DT>(xv.z, uv[u].z, au[b]);
                        au[b] = dot2<DT>(xv.w, uv[u].w, au[b]);
                    }
                }
            }
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const float gs = wave_sum(ag[b]);
            const float us = wave_sum(au[b]);
            if (lane == 0 && b < nb) s_out[(size_t)b * s_stride + t] = silu(gs) * us;
        }
    }
}

template <int NB, int DT>
__global__ __launch_bounds__(kDownThreads) void down_kernel(
    const uint16_t *__restrict__ wd, int d, const int *__restrict__ ff_idx, int n_ch,
    const float *__restrict__ s, int s_stride, int nb, int ch_per_split,
    float *__restrict__ ypart, Ctrl *__restrict__ ctrl, uint16_t *__restrict__ y) {
    extern __shared__ float dsh[];   // idx[cps] | s[NB][cps] | red[NB][kDownCols]
    int *idx_sh = reinterpret_cast<int *>(dsh);
    float *s_sh = dsh + ch_per_split;
    float *red_sh = s_sh + NB * ch_per_split;
    __shared__ int last_sh;

    const int tile = blockIdx.x, split = blockIdx.y, n_splits = gridDim.y;
    const int t0 = split * ch_per_split;
    const int n = max(0, min(n_ch - t0, ch_per_split));
    for (int e = threadIdx.x; e < n; e += kDownThreads) {
        idx_sh[e] = ff_idx ? ff_idx[t0 + e] : t0 + e;
#pragma unroll
        for (int b = 0; b < NB; ++b) s_sh[b * ch_per_split + e] = b < nb ? s[(size_t)b * s_stride + t0 + e] : 0.0f;
    }
    __syncthreads();

    const int wid = threadIdx.x / kWave, lane = lane_id();
    const int c0 = tile * kDownCols + lane * 8;
    const bool active = c0 < d;
    float acc[NB][8];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[b][e] = 0.0f;
    constexpr int U = 4;
    if (active) {
        for (int e0 = wid; e0 < n; e0 += kDownWaves * U) {
            uint4 wv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u * kDownWaves;
                if (e < n)
                    wv[u] = load_stream16(wd + (size_t)idx_sh[e] * d + c0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int e = e0 + u * kDownWaves;
                if (e < n) {
                    const uint32_t w4[4] = {wv[u].x, wv[u].y, wv[u].z, wv[u].w};
                    float wf[8];
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        wf[2 * q] = lo_to_float<DT>(w4[q]);
                        wf[2 * q + 1] = hi_to_float<DT>(w4[q]);
                    }
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const float sv = s_sh[b * ch_per_split + e];
#pragma unroll
                        for (int q = 0; q < 8; ++q) acc[b][q] = fmaf(sv, wf[q], acc[b][q]);
                    }
                }
            }
        }
    }
    // Sum the 8 waves in wave order through one LDS tile.
    for (int w = 0; w < kDownWaves; ++w) {
        if (wid == w) {
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    float *dst = &red_sh[b * kDownCols + lane * 8 + q];
                    *dst = w == 0 ? acc[b][q] : *dst + acc[b][q];
                }
        }
        __syncthreads();
    }
    for (int e = threadIdx.x; e < nb * kDownCols; e += kDownThreads) {
        const int b = e / kDownCols, c = e % kDownCols;
        const int col = tile * kDownCols + c;
        if (col < d) ypart[((size_t)split * NB + b) * d + col] = red_sh[b * kDownCols + c];
    }

    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = atomicAdd(&ctrl->down_count[tile], 1u);
        last_sh = prev == (uint32_t)(n_splits - 1);
    }
    __syncthreads();
    if (!last_sh) return;
    __threadfence();
    for (int e = threadIdx.x; e < nb * kDownCols; e += kDownThreads) {
        const int b = e / kDownCols, c = e % kDownCols;
        const int col = tile * kDownCols + c;
        if (col >= d) continue;
        float acc_y = 0.0f;
        for (int sp = 0; sp < n_splits; ++sp)
            acc_y += __builtin_nontemporal_load(&ypart[((size_t)sp * NB + b) * d + col]);
        y[(size_t)b * d + col] = float_to_half<DT>(acc_y);
    }
    if (threadIdx.x == 0) ctrl->down_count[tile] = 0;
}

template <int DT>
__global__ __launch_bounds__(1024) void add_rmsnorm_kernel(const uint16_t *__restrict__ x,
                                                           const uint16_t *__restrict__ y, int d,
                                                           float eps, uint16_t *out) {
    __shared__ float wsum[1024 / kWave];
    const int b = blockIdx.x;
    const uint16_t *xb = x + (size_t)b * d, *yb = y + (size_t)b * d;
    float ss = 0.0f;
    for (int i = threadIdx.x; i < d; i += 1024) {
        const float r = half_to_float<DT>(xb[i]) + half_to_float<DT>(yb[i]);
        ss = fmaf(r, r, ss);
    }
    ss = wave_sum(ss);
    if (lane_id() == 0) wsum[threadIdx.x / kWave] = ss;
    __syncthreads();
    float tot = 0.0f;
    for (int w = 0; w < 1024 / kWave; ++w) tot += wsum[w];
    const float inv = 1.0f / sqrtf(tot / (float)d + eps);
    __syncthreads();   // every thread has read x, y before out (which may alias x) is written
    for (int i = threadIdx.x; i < d; i += 1024) {
        const float r = half_to_float<DT>(xb[i]) + half_to_float<DT>(yb[i]);
        out[(size_t)b * d + i] = float_to_half<DT>(r * inv);
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

// Dynamic LDS above 64 KiB must be allowed per kernel (gfx950 has 160 KiB).
template <typename K>
static hipError_t allow_lds(K kernel, size_t bytes) {
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

int gateup_grid(int n_ch) {
    // Enough waves to cover the channels, at most 4 workgroups per CU.
    const int waves_per_wg = kGuThreads / kWave;
    int wgs = (n_ch + waves_per_wg - 1) / waves_per_wg;
    return wgs < 1024 ? (wgs < 1 ? 1 : wgs) : 1024;
}

template <int NB, int DT>
static void launch_gateup_t(const void *x, int nb, int d, const void *wg, const void *wu,
                            const int *ff_idx, int n_ch, float *s_out, int s_stride,
                            Ctrl *ctrl_reset, hipStream_t st) {
    const size_t lds = (size_t)NB * d * sizeof(uint16_t);
    if (allow_lds(gateup_kernel<NB, DT>, lds) != hipSuccess) return;
    gateup_kernel<NB, DT><<<gateup_grid(n_ch), kGuThreads, lds, st>>>(
        static_cast<const uint16_t *>(x), nb, d, static_cast<const uint16_t *>(wg),
        static_cast<const uint16_t *>(wu), ff_idx, n_ch, s_out, s_stride, ctrl_reset);
}

hipError_t launch_gateup(int dtype, const void *x, int nb, int d, const void *wg, const void *wu,
                         const int *ff_idx, int n_ch, float *s_out, int s_stride,
                         Ctrl *ctrl_reset, hipStream_t st) {
#define GU(NB_)                                                                                    \
    (dtype == kBF16 ? launch_gateup_t<NB_, kBF16>(x, nb, d, wg, wu, ff_idx, n_ch, s_out, s_stride, \
                                                   ctrl_reset, st)                                 \
                    : launch_gateup_t<NB_, kF16>(x, nb, d, wg, wu, ff_idx, n_ch, s_out, s_stride,  \
                                                  ctrl_reset, st))
    if (nb == 1) GU(1);
    else if (nb == 2) GU(2);
    else GU(4);
#undef GU
    return hipGetLastError();
}

void down_geometry(int d, int n_ch, int &tiles, int &splits, int &ch_per_split) {
    tiles = (d + kDownCols - 1) / kDownCols;
    // About 16 channels per wave, at most kDownMaxSplits slices.
    int sp = n_ch / (kDownWaves * 16);
    sp = sp < 1 ? 1 : (sp > kDownMaxSplits ? kDownMaxSplits : sp);
    ch_per_split = (n_ch + sp - 1) / sp;
    splits = (n_ch + ch_per_split - 1) / ch_per_split;
}

size_t down_lds_bytes(int nbt, int ch_per_split) {
    return (size_t)ch_per_split * sizeof(int) + (size_t)nbt * ch_per_split * sizeof(float) +
           (size_t)nbt * kDownCols * sizeof(float);
}

template <int NB, int DT>
static void launch_down_t(const void *wd, int d, const int *ff_idx, int n_ch, const float *s,
                          int s_stride, int nb, float *ypart, Ctrl *ctrl, void *y, hipStream_t st) {
    int tiles, splits, cps;
    down_geometry(d, n_ch, tiles, splits, cps);
    if (allow_lds(down_kernel<NB, DT>, down_lds_bytes(NB, cps)) != hipSuccess) return;
    down_kernel<NB, DT><<<dim3(tiles, splits), kDownThreads, down_lds_bytes(NB, cps), st>>>(
        static_cast<const uint16_t *>(wd), d, ff_idx, n_ch, s, s_stride, nb, cps, ypart, ctrl,
        static_cast<uint16_t *>(y));
}

hipError_t launch_down(int dtype, const void *wd, int d, const int *ff_idx, int n_ch,
                       const float *s, int s_stride, int nb, float *ypart, Ctrl *ctrl, void *y,
                       hipStream_t st) {
#define DN(NB_)                                                                                 \
    (dtype == kBF16 ? launch_down_t<NB_, kBF16>(wd, d, ff_idx, n_ch, s, s_stride, nb, ypart, ctrl, y, st) \
                    : launch_down_t<NB_, kF16>(wd, d, ff_idx, n_ch, s, s_stride, nb, ypart, ctrl, y, st))
    switch (down_nb_t(nb)) {
        case 1: DN(1); break;
        case 2: DN(2); break;
        case 4: DN(4); break;
        case 8: DN(8); break;
        default: DN(16); break;
    }
#undef DN
    return hipGetLastError();
}

hipError_t launch_add_rmsnorm(int dtype, const void *x, const void *y, int batch, int d, float eps,
                              void *out, hipStream_t st) {
    auto *xp = static_cast<const uint16_t *>(x);
    auto *yp = static_cast<const uint16_t *>(y);
    auto *op = static_cast<uint16_t *>(out);
    if (dtype == kBF16) add_rmsnorm_kernel<kBF16><<<batch, 1024, 0, st>>>(xp, yp, d, eps, op);
    else add_rmsnorm_kernel<kF16><<<batch, 1024, 0, st>>>(xp, yp, d, eps, op);
    return hipGetLastError();
}

}  // namespace prox
