// Stage 1 of the sparse decode step (Sec. 4.1 Stage 1; proxies of Sec. 4.3):
//
//   m_x      = top-k_in of a_i = max_b |x_{b,i}|            (App. A.6 rule)
//   g~_{b,j} = sum_{i in m_x} x_{b,i} q^g_{ij} sigma^g_{g(i),j}   (u~ alike)
//   score_j  = max_b |SiLU(g~_{b,j}) u~_{b,j}|
//
// One workgroup per column tile of the proxy blob, so a workgroup owns its
// outputs completely and no partial sums leave it.  Every workgroup first
// finds the input top-k itself (block-local work, cheaper than a separate
// launch) and writes the kept rows, in ascending order, into one LDS list,
// padded per quantisation group to an even count.  Each of the 16 waves then
// streams a contiguous range of row pairs.
//
// A lane reads 4 (INT4) or 8 (INT8) bytes of both rows' contiguous segments,
// i.e. the same 8 proxy columns of two input rows.  For INT4 the two rows'
// bytes are interleaved with v_perm and each nibble pair is OR-ed under the
// exponent of 128.0 (bf16) or 1024.0 (fp16): that is the exact 16-bit pair
// (M + n_a, M + n_b), n = q + 8, and one dot2 accumulates
// x_a (M + n_a) + x_b (M + n_b) in fp32.  (M + 8) * sum(x) is subtracted and
// the group's scale applied once per group and column.  Lane groups and waves
// are summed in a fixed order, so results are deterministic.
#include "common.hpp"
#include "kernels.hpp"
#include "topk.hpp"

#include <type_traits>

namespace prox {

template <int DT>
struct Magic;
template <>
struct Magic<kBF16> {   // 0x4300 = 128.0 in bf16; 128 + n is exact for n < 128
    static constexpr uint32_t pair = 0x43004300u;
    static constexpr float offset = 136.0f;   // 128 + 8 (code bias)
};
template <>
struct Magic<kF16> {    // 0x6400 = 1024.0 in fp16; 1024 + n is exact for n < 1024
    static constexpr uint32_t pair = 0x64006400u;
    static constexpr float offset = 1032.0f;
};

// acc[c] += x_a (M + n_a[c]) + x_b (M + n_b[c]) for the 8 INT4 columns held in
// one 32-bit word of each row.
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

// acc[c] += x_a n_a[c] + x_b n_b[c] for 8 INT8 columns (n = q + 128).
template <int DT>
__device__ __forceinline__ void int8_pair_fma8(uint2 a, uint2 b, uint32_t xpair, float *acc) {
    const float xa = lo_to_float<DT>(xpair), xb = hi_to_float<DT>(xpair);
    const uint32_t aw[2] = {a.x, a.y}, bw[2] = {b.x, b.y};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float na = (float)((aw[e >> 2] >> (8 * (e & 3))) & 255u);
        const float nb = (float)((bw[e >> 2] >> (8 * (e & 3))) & 255u);
        acc[e] = fmaf(xb, nb, fmaf(xa, na, acc[e]));
    }
}

__device__ __forceinline__ uint32_t input_key(const uint16_t *__restrict__ x, int B, int d, int i) {
    // |x| as its 15-bit magnitude pattern: monotone in |x| for fp16 and bf16,
    // with +0 and -0 equal.
    uint32_t k = 0;
    for (int b = 0; b < B; ++b) k = max(k, (uint32_t)(x[(size_t)b * d + i] & 0x7FFFu));
    return k;
}

// Dynamic LDS of the proxy kernel: the kept-row list (row ids, x values per
// batch row, group id per pair), later reused for the cross-wave reduction.
__host__ __device__ inline int proxy_list_cap(int k_in, int ng) {
    return (k_in + ng + 1) / 2 * 2;   // kept rows + one pad per odd group, even
}
__host__ __device__ inline size_t proxy_lds_bytes(int k_in, int ng, int nbt, int T) {
    const size_t cap = (size_t)proxy_list_cap(k_in, ng);
    const size_t list = align_up(cap * 2 * (1 + nbt), 16) + align_up(cap / 2, 16);
    const size_t red = (size_t)kMaxBlockWaves * nbt * 2 * T * 4;
    return list > red ? list : red;
}

template <int NB, int DT, int QB, int T>
__global__ __launch_bounds__(kBlock) void proxy_kernel(
    const uint16_t *__restrict__ x_all, int B_all,  // every batch row (selection keys)
    int row0, int nb,                                 // rows [row0, row0 + nb) are projected
    int d, int f, int group, int k_in, const uint8_t *__restrict__ blob,
    Ctrl *__restrict__ ctrl, uint8_t *__restrict__ in_mask, float *__restrict__ scores,
    int accumulate) {
    constexpr int LPS = T / 4;            // lanes per row segment, 8 columns each
    constexpr int NGRP = kWave / LPS;     // row pairs a wave works on side by side
    constexpr int C = kMaxDModel / kBlock;
    constexpr int U = 8;                  // row pairs in flight per lane group
    const BlobLayout L(d, f, QB, group);
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();
    const int tile = blockIdx.x;
    const int ng = d / group;

    __shared__ TopKScratch tk;
    __shared__ int gcnt[kMaxDModel / 128];     // kept rows per group
    __shared__ int gstart[kMaxDModel / 128];   // padded list position of each group
    __shared__ int n_pairs_sh;
    extern __shared__ __align__(16) unsigned char dsm[];

    const int cap = proxy_list_cap(k_in, ng);
    uint16_t *rows_sh = reinterpret_cast<uint16_t *>(dsm);               // [cap]
    uint16_t *xs_sh = rows_sh + cap;                                      // [NB][cap]
    uint8_t *grp_sh = dsm + align_up((size_t)cap * 2 * (1 + NB), 16);    // [cap / 2]

    // ---- input top-k: thread t owns rows [t*c, t*c + c) ----
    const int c = (d + kBlock - 1) / kBlock;
    uint32_t key[C];
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const int i = tid * c + r;
        key[r] = (r < c && i < d) ? input_key(x_all, B_all, d, i) : 0u;
    }
    for (int g = tid; g < ng; g += kBlock) gcnt[g] = 0;
    uint32_t v;
    int need;
    const RegKeys<C> keys{key};
    topk_threshold<kBlock, C>(keys, c, d, k_in, tk, v, need);
    int rank;
    const int pos0 = topk_positions<kBlock, C>(keys, c, d, v, need, tk, rank);
    // Count the kept rows of each group (integer atomics: order-independent).
    {
        int g_cur = -1, n_cur = 0, rk = rank;
#pragma unroll
        for (int r = 0; r < C; ++r) {
            const int i = tid * c + r;
            if (r >= c || i >= d) continue;
            bool sel = key[r] > v;
            if (key[r] == v) sel = rk++ < need;
            const int g = i / group;
            if (g != g_cur) {
                if (n_cur) atomicAdd(&gcnt[g_cur], n_cur);
                g_cur = g;
                n_cur = 0;
            }
            n_cur += sel;
        }
        if (n_cur) atomicAdd(&gcnt[g_cur], n_cur);
    }
    __syncthreads();
    if (wid == 0) {
        // Padded start of each group: earlier groups' counts rounded up to even.
        int carry = 0;
        for (int g0 = 0; g0 < ng; g0 += kWave) {
            const int g = g0 + lane;
            const int padded = g < ng ? (gcnt[g] + 1) / 2 * 2 : 0;
            const int incl = wave_inclusive_scan(padded);
            if (g < ng) gstart[g] = carry + incl - padded;
            carry += __shfl(incl, kWave - 1, kWave);
        }
        if (lane == 0) n_pairs_sh = carry / 2;
    }
    __syncthreads();
    // Scatter the kept rows to their padded positions, then the pad entries.
    {
        int pos = pos0, rk = rank, g_cur = -1, g_base = 0;
#pragma unroll
        for (int r = 0; r < C; ++r) {
            const int i = tid * c + r;
            if (r >= c || i >= d) continue;
            bool sel = key[r] > v;
            if (key[r] == v) {
                sel = rk < need;
                if (tile == 0 && rk == need - 1) {
                    ctrl->in_v = v;
                    ctrl->in_cut = (uint32_t)i;
                }
                ++rk;
            }
            if (tile == 0 && in_mask) in_mask[i] = sel ? 1 : 0;
            if (!sel) continue;
            const int g = i / group;
            if (g != g_cur) {   // kept rows of all earlier groups
                g_base = 0;
                for (int h = 0; h < g; ++h) g_base += gcnt[h];
                g_cur = g;
            }
            const int p = gstart[g] + (pos - g_base);
            rows_sh[p] = (uint16_t)i;
#pragma unroll
            for (int b = 0; b < NB; ++b)
                xs_sh[b * cap + p] = b < nb ? x_all[(size_t)(row0 + b) * d + i] : 0;
            if ((p & 1) == 0) grp_sh[p >> 1] = (uint8_t)g;
            ++pos;
        }
    }
    for (int g = tid; g < ng; g += kBlock) {
        if (gcnt[g] & 1) {   // zero-weight pad row keeps pairs inside the group
            const int p = gstart[g] + gcnt[g];
            rows_sh[p] = (uint16_t)(g * group);
#pragma unroll
            for (int b = 0; b < NB; ++b) xs_sh[b * cap + p] = 0;
        }
    }
    __syncthreads();

    // ---- stream the kept row pairs: wave w owns a contiguous range ----
    const int npairs = n_pairs_sh;
    const int ps = (int)((long long)wid * npairs / kMaxBlockWaves);
    const int pe = (int)((long long)(wid + 1) * npairs / kMaxBlockWaves);
    const uint32_t *rows32 = reinterpret_cast<const uint32_t *>(rows_sh);
    const int lg = lane / LPS, li = lane % LPS;
    const int mat = li / (LPS / 2);                 // 0: gate, 1: up
    const int col8 = (li % (LPS / 2)) * 8;          // first of this lane's 8 columns
    const uint8_t *cbase = blob + L.codes_offset + (size_t)tile * d * L.row_bytes +
                           (size_t)mat * (T * QB / 8) + (size_t)col8 * QB / 8;
    const uint16_t *sbase = reinterpret_cast<const uint16_t *>(blob + L.scales_offset) +
                            (size_t)tile * ng * 2 * T + (size_t)mat * T + col8;
    constexpr float off = QB == 4 ? Magic<DT>::offset : 128.0f;

    float tot[NB][8], acc[NB][8], xsum[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        xsum[b] = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) tot[b][e] = acc[b][e] = 0.0f;
    }
    int cur_g = ps + lg < pe ? grp_sh[ps + lg] : 0;
    uint4 sc = *reinterpret_cast<const uint4 *>(sbase + (size_t)cur_g * 2 * T);

    auto flush = [&](const uint4 &s4) {
        const uint32_t sw[4] = {s4.x, s4.y, s4.z, s4.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float sg = f16_bits_to_float((e & 1) ? (sw[e >> 1] >> 16) : (sw[e >> 1] & 0xFFFFu));
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                tot[b][e] = fmaf(sg, acc[b][e] - off * xsum[b], tot[b][e]);
                acc[b][e] = 0.0f;
            }
        }
#pragma unroll
        for (int b = 0; b < NB; ++b) xsum[b] = 0.0f;
    };

    using W = typename std::conditional<QB == 4, uint32_t, uint2>::type;
    for (int p0 = ps + lg; p0 < pe; p0 += NGRP * U) {
        W wa[U], wb[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int p = p0 + u * NGRP;
            if (p < pe) {
                const uint32_t rr = rows32[p];
                wa[u] = *reinterpret_cast<const W *>(cbase + (size_t)(rr & 0xFFFFu) * L.row_bytes);
                wb[u] = *reinterpret_cast<const W *>(cbase + (size_t)(rr >> 16) * L.row_bytes);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int p = p0 + u * NGRP;
            if (p < pe) {
                const int g = grp_sh[p];
                if (g != cur_g) {
                    // The new group's scales are fetched here and first used at
                    // its own flush, so the load latency stays hidden.
                    const uint4 nsc = *reinterpret_cast<const uint4 *>(sbase + (size_t)g * 2 * T);
                    flush(sc);
                    sc = nsc;
                    cur_g = g;
                }
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    const uint32_t xp = reinterpret_cast<const uint32_t *>(xs_sh + b * cap)[p];
                    xsum[b] += lo_to_float<DT>(xp) + hi_to_float<DT>(xp);
                    if constexpr (QB == 4) int4_pair_dot8<DT>(wa[u], wb[u], xp, acc[b]);
                    else int8_pair_fma8<DT>(wa[u], wb[u], xp, acc[b]);
                }
            }
        }
    }
    flush(sc);

    // ---- combine lane groups, then waves, in a fixed order ----
#pragma unroll
    for (int o = LPS; o < kWave; o <<= 1)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < 8; ++e) tot[b][e] += __shfl_xor(tot[b][e], o, kWave);
    __syncthreads();   // the list is dead; reuse the LDS for the reduction
    float *red = reinterpret_cast<float *>(dsm);   // [16][NB][2T]
    if (lg == 0) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < 8; ++e) red[(wid * NB + b) * 2 * T + mat * T + col8 + e] = tot[b][e];
    }
    __syncthreads();
    if (tid < T) {
        const int j = tile * T + tid;
        float best = 0.0f;
        for (int b = 0; b < nb; ++b) {
            float gu[2];
#pragma unroll
            for (int m2 = 0; m2 < 2; ++m2) {
                float s8[8];
#pragma unroll
                for (int q = 0; q < 8; ++q)
                    s8[q] = red[((2 * q) * NB + b) * 2 * T + m2 * T + tid] +
                            red[((2 * q + 1) * NB + b) * 2 * T + m2 * T + tid];
                gu[m2] = ((s8[0] + s8[1]) + (s8[2] + s8[3])) + ((s8[4] + s8[5]) + (s8[6] + s8[7]));
            }
            best = fmaxf(best, fabsf(silu(gu[0]) * gu[1]));
        }
        if (j < f) scores[j] = accumulate ? fmaxf(scores[j], best) : best;
    }
}

template <int NB, int DT, int QB, int T>
static hipError_t launch_proxy_t(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                 int group, int k_in, const void *blob, Ctrl *ctrl,
                                 uint8_t *in_mask, float *scores, int accumulate, hipStream_t s) {
    const BlobLayout L(d, f, QB, group);
    const size_t lds = proxy_lds_bytes(k_in, d / group, NB, T);
    if (lds > 65536) {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void *>(proxy_kernel<NB, DT, QB, T>),
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    proxy_kernel<NB, DT, QB, T><<<L.n_tiles, kBlock, lds, s>>>(
        static_cast<const uint16_t *>(x_all), B_all, row0, nb, d, f, group, k_in,
        static_cast<const uint8_t *>(blob), ctrl, in_mask, scores, accumulate);
    return hipGetLastError();
}

template <int DT, int QB, int T>
static hipError_t launch_proxy_nb(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                  int group, int k_in, const void *blob, Ctrl *ctrl,
                                  uint8_t *in_mask, float *scores, int accumulate, hipStream_t s) {
    switch (proxy_nb_t(nb)) {
        case 1: return launch_proxy_t<1, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
        case 2: return launch_proxy_t<2, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
        default: return launch_proxy_t<4, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
    }
}

template <int DT, int QB>
static hipError_t launch_proxy_tile(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                    int group, int k_in, const void *blob, Ctrl *ctrl,
                                    uint8_t *in_mask, float *scores, int accumulate,
                                    hipStream_t s) {
    if (proxy_tile(f) == 128)
        return launch_proxy_nb<DT, QB, 128>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
    return launch_proxy_nb<DT, QB, 64>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
}

int proxy_max_nb(int d) { return d <= 8192 ? kProxyMaxNB : 2; }

hipError_t launch_proxy(int dtype, int qbits, const void *x_all, int B_all, int row0, int nb,
                        int d, int f, int group, int k_in, const void *blob, Ctrl *ctrl,
                        uint8_t *in_mask, float *scores, int accumulate, hipStream_t s) {
    if (dtype == kBF16 && qbits == 4) return launch_proxy_tile<kBF16, 4>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
    if (dtype == kBF16) return launch_proxy_tile<kBF16, 8>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
    if (qbits == 4) return launch_proxy_tile<kF16, 4>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
    return launch_proxy_tile<kF16, 8>(x_all, B_all, row0, nb, d, f, group, k_in, blob, ctrl, in_mask, scores, accumulate, s);
}

}  // namespace prox
