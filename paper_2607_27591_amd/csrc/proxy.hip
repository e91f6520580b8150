// Stage 1 proxy GEMV and score (Sec. 4.1 Stage 1, Sec. 4.3).
//
//   g~_{b,j} = sum_{i in m_x} x_{b,i} q^g_{ij} sigma^g_{g(i),j}   (u~ alike)
//   score_j  = max_b |SiLU(g~_{b,j}) u~_{b,j}|
//
// Decomposition: grid = (column tile of kTile proxy columns) x (split of
// kProxyRowsPerSplit input rows).  Each wave owns 64 consecutive input rows,
// all inside one quantisation group (group is a multiple of 128).  The wave
// ballots which of its rows the input top-k kept, compacts them into an LDS
// list, and walks the kept rows two at a time: every lane reads 8 bytes (INT4)
// or 16 bytes (INT8) of both rows' contiguous segments, i.e. 16 columns of the
// gate (lanes 0-31) or up (lanes 32-63) proxy.
//
// INT4 dequantisation without per-element conversions: the two rows' bytes
// are interleaved with v_perm, each nibble pair is OR-ed under the exponent of
// 128.0 (bf16) or 1024.0 (fp16), giving the exact 16-bit values M + n with
// n = q + 8, and a single dot2 instruction accumulates x_a (M + n_a) +
// x_b (M + n_b) in fp32.  The constant (M + 8) * sum(x) is subtracted once per
// wave, and the group scale is applied once per column.
//
// The partial sums of all row splits of a tile are combined by the last
// workgroup to arrive (arrival counter per tile), in split order, which then
// evaluates SiLU(g~) u~ and the batch-max magnitude.
#include "common.hpp"
#include "kernels.hpp"

namespace prox {

constexpr int kProxyThreads = kProxyWaves * kWave;
constexpr int kListCap = kProxyRowsPerWave + 2;   // kept rows + odd padding

template <int DT>
struct Magic;
template <>
struct Magic<kBF16> {   // 0x4300 = 128.0 in bf16; 128 + n exact for n < 128
    static constexpr uint32_t pair = 0x43004300u;
    static constexpr float offset = 136.0f;   // 128 + 8 (code bias)
};
template <>
struct Magic<kF16> {    // 0x6400 = 1024.0 in fp16; 1024 + n exact for n < 1024
    static constexpr uint32_t pair = 0x64006400u;
    static constexpr float offset = 1032.0f;
};

// acc[c] += x_a * (M + n_a[c]) + x_b * (M + n_b[c]) for the 8 columns of one
// 32-bit word of each row.
template <int DT>
__device__ __forceinline__ void int4_pair_dot8(uint32_t a, uint32_t b, uint32_t xpair,
                                               float *acc) {
    constexpr uint32_t M = Magic<DT>::pair;
    const uint32_t p = __builtin_amdgcn_perm(b, a, 0x05040100u);  // a.b0 a.b1 b.b0 b.b1
    const uint32_t q = __builtin_amdgcn_perm(b, a, 0x07060302u);  // a.b2 a.b3 b.b2 b.b3
    acc[0] = dot2<DT>(xpair, (p & 0x000F000Fu) | M, acc[0]);
    acc[1] = dot2<DT>(xpair, ((p >> 4) & 0x000F000Fu) | M, acc[1]);
    acc[2] = dot2<DT>(xpair, ((p >> 8) & 0x000F000Fu) | M, acc[2]);
    acc[3] = dot2<DT>(xpair, ((p >> 12) & 0x000F000Fu) | M, acc[3]);
    acc[4] = dot2<DT>(xpair, (q & 0x000F000Fu) | M, acc[4]);
    acc[5] = dot2<DT>(xpair, ((q >> 4) & 0x000F000Fu) | M, acc[5]);
    acc[6] = dot2<DT>(xpair, ((q >> 8) & 0x000F000Fu) | M, acc[6]);
    acc[7] = dot2<DT>(xpair, ((q >> 12) & 0x000F000Fu) | M, acc[7]);
}

template <int NB, int DT, int QB>
__global__ __launch_bounds__(kProxyThreads) void proxy_kernel(
    const uint16_t *__restrict__ x,      // rows of this launch, [nb][d]
    int nb,
    const uint16_t *__restrict__ x_all,  // all batch rows, for the selection test
    int B_all, int d, int f, int group, const uint8_t *__restrict__ blob,
    Ctrl *__restrict__ ctrl, float *__restrict__ part, float *__restrict__ scores,
    int accumulate) {
    const BlobLayout L(d, f, QB, group);
    const int tile = blockIdx.x, split = blockIdx.y, n_splits = gridDim.y;
    const int wid = threadIdx.x / kWave, lane = lane_id();
    const int r0 = split * kProxyRowsPerSplit + wid * kProxyRowsPerWave;

    __shared__ __align__(4) uint16_t rows_sh[kProxyWaves][kListCap];
    __shared__ __align__(4) uint16_t xs_sh[kProxyWaves][NB][kListCap];
    __shared__ float red_sh[4][NB][2 * kTile];
    __shared__ int last_sh;

    // ---- which of this wave's 64 rows did the input top-k keep ----
    const uint32_t v = ctrl->in_v, cut = ctrl->in_cut;
    const int i = r0 + lane;
    bool sel = false;
    if (i < d) {
        uint32_t key = 0;
        for (int b = 0; b < B_all; ++b) key = max(key, (uint32_t)(x_all[(size_t)b * d + i] & 0x7FFFu));
        sel = key > v || (key == v && (uint32_t)i <= cut);
    }
    const uint64_t m = __ballot(sel);
    const int cnt = __popcll(m);
    if (sel) {
        const int pos = (int)lanes_below(m);
        rows_sh[wid][pos] = (uint16_t)i;
#pragma unroll
        for (int b = 0; b < NB; ++b) xs_sh[wid][b][pos] = b < nb ? x[(size_t)b * d + i] : 0;
    }
    if (lane == 0 && (cnt & 1)) {   // pad to an even count with a zero-weight row
        rows_sh[wid][cnt] = (uint16_t)r0;
#pragma unroll
        for (int b = 0; b < NB; ++b) xs_sh[wid][b][cnt] = 0;
    }
    __syncthreads();

    // ---- accumulate over the kept rows, two at a time ----
    const int mat = lane >> 5;                 // 0: gate, 1: up
    const int lc = (lane & 31) * 16;           // first of this lane's 16 columns
    constexpr int kSegBytes = kTile * QB / 8;  // one matrix's part of a row segment
    const uint8_t *base = blob + L.codes_offset + (size_t)tile * d * L.row_bytes + mat * kSegBytes +
                          lc * QB / 8;
    float acc[NB][16];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int c = 0; c < 16; ++c) acc[b][c] = 0.0f;

    const int npairs = (cnt + 1) >> 1;
    const uint32_t *rows32 = reinterpret_cast<const uint32_t *>(rows_sh[wid]);
    constexpr int U = 4;   // row pairs in flight
    for (int p0 = 0; p0 < npairs; p0 += U) {
        if constexpr (QB == 4) {
            uint2 wa[U], wb[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p0 + u < npairs) {
                    const uint32_t rr = rows32[p0 + u];
                    wa[u] = *reinterpret_cast<const uint2 *>(base + (size_t)(rr & 0xFFFFu) * L.row_bytes);
                    wb[u] = *reinterpret_cast<const uint2 *>(base + (size_t)(rr >> 16) * L.row_bytes);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p0 + u < npairs) {
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const uint32_t xp = reinterpret_cast<const uint32_t *>(xs_sh[wid][b])[p0 + u];
                        int4_pair_dot8<DT>(wa[u].x, wb[u].x, xp, &acc[b][0]);
                        int4_pair_dot8<DT>(wa[u].y, wb[u].y, xp, &acc[b][8]);
                    }
                }
            }
        } else {
            uint4 wa[U], wb[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p0 + u < npairs) {
                    const uint32_t rr = rows32[p0 + u];
                    wa[u] = *reinterpret_cast<const uint4 *>(base + (size_t)(rr & 0xFFFFu) * L.row_bytes);
                    wb[u] = *reinterpret_cast<const uint4 *>(base + (size_t)(rr >> 16) * L.row_bytes);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (p0 + u < npairs) {
                    const uint32_t wa_w[4] = {wa[u].x, wa[u].y, wa[u].z, wa[u].w};
                    const uint32_t wb_w[4] = {wb[u].x, wb[u].y, wb[u].z, wb[u].w};
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const uint32_t xp = reinterpret_cast<const uint32_t *>(xs_sh[wid][b])[p0 + u];
                        const float xa = lo_to_float<DT>(xp), xb = hi_to_float<DT>(xp);
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const float na = (float)((wa_w[e >> 2] >> (8 * (e & 3))) & 255u);
                            const float nbv = (float)((wb_w[e >> 2] >> (8 * (e & 3))) & 255u);
                            acc[b][e] = fmaf(xa, na, acc[b][e]);
                            acc[b][e] = fmaf(xb, nbv, acc[b][e]);
                        }
                    }
                }
            }
        }
    }

    // ---- remove the code bias, apply the group scale ----
    const int ng = d / group;
    const int g = min(r0, d - 1) / group;
    const uint16_t *sc = reinterpret_cast<const uint16_t *>(blob + L.scales_offset) +
                         (((size_t)tile * ng + g) * 2 + mat) * kTile + lc;
    uint4 s01 = reinterpret_cast<const uint4 *>(sc)[0];
    uint4 s23 = reinterpret_cast<const uint4 *>(sc)[1];
    const uint32_t sw[8] = {s01.x, s01.y, s01.z, s01.w, s23.x, s23.y, s23.z, s23.w};
    constexpr float off = QB == 4 ? Magic<DT>::offset : 128.0f;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const float xv = lane < cnt ? half_to_float<DT>(xs_sh[wid][b][lane]) : 0.0f;
        const float xsum = wave_sum(xv);
#pragma unroll
        for (int c = 0; c < 16; ++c) {
            const float sg = f16_bits_to_float((c & 1) ? (sw[c >> 1] >> 16) : (sw[c >> 1] & 0xFFFFu));
            acc[b][c] = cnt > 0 ? sg * (acc[b][c] - off * xsum) : 0.0f;
        }
    }

    // ---- combine the 8 waves in a fixed order: (w0+w4)+(w1+w5)+(w2+w6)+(w3+w7) ----
    const int col = mat * kTile + lc;
    if (wid >= 4) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int c = 0; c < 16; ++c) red_sh[wid - 4][b][col + c] = acc[b][c];
    }
    __syncthreads();
    if (wid < 4) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int c = 0; c < 16; ++c) red_sh[wid][b][col + c] += acc[b][c];
    }
    __syncthreads();
    const int f_pad = L.f_pad;
    for (int e = threadIdx.x; e < NB * 2 * kTile; e += kProxyThreads) {
        const int b = e / (2 * kTile), rem = e % (2 * kTile);
        const float vsum = (red_sh[0][b][rem] + red_sh[1][b][rem]) + (red_sh[2][b][rem] + red_sh[3][b][rem]);
        const int mm = rem / kTile, cc = rem % kTile;
        part[((size_t)(split * NB + b) * 2 + mm) * f_pad + (size_t)tile * kTile + cc] = vsum;
    }

    // ---- last workgroup of this tile: reduce splits, SwiGLU, batch max ----
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = atomicAdd(&ctrl->proxy_count[tile], 1u);
        last_sh = prev == (uint32_t)(n_splits - 1);
    }
    __syncthreads();
    if (!last_sh) return;
    __threadfence();
    for (int c = threadIdx.x; c < kTile; c += kProxyThreads) {
        const int j = tile * kTile + c;
        float best = 0.0f;
        for (int b = 0; b < nb; ++b) {
            float gs = 0.0f, us = 0.0f;
            for (int sp = 0; sp < n_splits; ++sp) {
                gs += __builtin_nontemporal_load(&part[((size_t)(sp * NB + b) * 2 + 0) * f_pad + j]);
                us += __builtin_nontemporal_load(&part[((size_t)(sp * NB + b) * 2 + 1) * f_pad + j]);
            }
            best = fmaxf(best, fabsf(silu(gs) * us));
        }
        if (j < f) scores[j] = accumulate ? fmaxf(scores[j], best) : best;
    }
    if (threadIdx.x == 0) ctrl->proxy_count[tile] = 0;
}

template <int NB, int DT, int QB>
static void launch_proxy_t(const void *x, int nb, const void *x_all, int B_all, int d, int f,
                           int group, const void *blob, Ctrl *ctrl, float *part, float *scores,
                           int accumulate, hipStream_t s) {
    const BlobLayout L(d, f, QB, group);
    dim3 grid(L.n_tiles, proxy_splits(d));
    proxy_kernel<NB, DT, QB><<<grid, kProxyThreads, 0, s>>>(
        static_cast<const uint16_t *>(x), nb, static_cast<const uint16_t *>(x_all), B_all, d, f,
        group, static_cast<const uint8_t *>(blob), ctrl, part, scores, accumulate);
}

template <int DT, int QB>
static void launch_proxy_nb(int nb, const void *x, const void *x_all, int B_all, int d, int f,
                            int group, const void *blob, Ctrl *ctrl, float *part, float *scores,
                            int accumulate, hipStream_t s) {
    if (nb == 1) launch_proxy_t<1, DT, QB>(x, nb, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    else if (nb == 2) launch_proxy_t<2, DT, QB>(x, nb, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    else launch_proxy_t<4, DT, QB>(x, nb, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
}

hipError_t launch_proxy(int dtype, int qbits, const void *x, int nb, const void *x_all, int B_all,
                        int d, int f, int group, const void *blob, Ctrl *ctrl, float *part,
                        float *scores, int accumulate, hipStream_t s) {
    if (dtype == kBF16 && qbits == 4) launch_proxy_nb<kBF16, 4>(nb, x, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    else if (dtype == kBF16) launch_proxy_nb<kBF16, 8>(nb, x, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    else if (qbits == 4) launch_proxy_nb<kF16, 4>(nb, x, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    else launch_proxy_nb<kF16, 8>(nb, x, x_all, B_all, d, f, group, blob, ctrl, part, scores, accumulate, s);
    return hipGetLastError();
}

}  // namespace prox
