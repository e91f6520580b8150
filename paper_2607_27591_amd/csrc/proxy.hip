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
// padded per quantisation group to an even count.  Each lane group then
// streams a contiguous range of row pairs.
//
// A lane reads 8 (INT4), 8 or 16 (INT8) or 16 (unquantised 16-bit proxy)
// bytes of both rows' contiguous segments, i.e. the same proxy columns of two
// input rows.  INT4 codes are dequantised in fp16 whatever the model dtype:
// byte k of both rows goes side by side (one v_perm), its low nibble OR-ed
// under the exponent of 1024.0 is the exact fp16 pair (1024 + n_a, 1024 + n_b),
// n = q + 8, and its high nibble in place, with the same OR, is
// (1024 + 16 n_a, 1024 + 16 n_b); one v_dot2_f32_f16 each accumulates
// x_a (...) + x_b (...) in fp32.  Both nibbles of a byte need no shift, which
// bf16 (7 mantissa bits) would.  The kept x go to the list in fp16: bf16 x are
// scaled by one power of two 2^s that puts the largest |x| in [2^14, 2^15), so
// every kept x is exact in fp16 down to 2^-28 of the largest, and the sums are
// scaled back by 2^-s.  The code bias ((1024 + 8) or (1024 + 128) times sum(x))
// is subtracted and the group's scale applied once per group, column and lane
// group; high-nibble columns are divided by 16 at the end.  Lane groups and waves are summed in a fixed order, so results are
// deterministic.  This kernel takes up to 4 batch rows per launch; five or
// more rows with an INT4 proxy go to proxy_mfma_kernel (the matrix cores).
#include "common.hpp"
#include "kernels.hpp"
#include "topk.hpp"

namespace prox {

// acc[c] += x_a (1024 + n_a[c]) + x_b (1024 + n_b[c]) (even c) or
// x_a (1024 + 16 n_a[c]) + x_b (1024 + 16 n_b[c]) (odd c) for the 8 INT4
// columns of one 32-bit word of each row, x fp16: byte k of both words side by
// side, then its low nibble (column 2k) or its high nibble in place (column
// 2k + 1) OR-ed under the exponent of 1024.0, each exact in fp16.
template <bool FUSED>
__device__ __forceinline__ void int4_pair_dot8_h(uint32_t a, uint32_t b, uint32_t xpair,
                                                 float *acc) {
    constexpr uint32_t M = Int4Magic<kF16>::pair;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t p = __builtin_amdgcn_perm(b, a, (uint32_t)k | ((uint32_t)(k + 4) << 16));
        acc[2 * k] = dot2<kF16>(xpair, and_or<FUSED>(p, 0x000F000Fu, M), acc[2 * k]);
        acc[2 * k + 1] = dot2<kF16>(xpair, and_or<FUSED>(p, 0x00F000F0u, M), acc[2 * k + 1]);
    }
}
// Code bias of column e of an fp16-dequantised INT4 word, and its scale.
constexpr float kInt4HBias[2] = {1024.0f + 8.0f, 1024.0f + 128.0f};
constexpr float kInt4HScale[2] = {1.0f, 1.0f / 16.0f};

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

// Dynamic LDS of the proxy kernel: the input selection's histogram, then the
// kept-row list (row ids and x values per batch row), then the cross-wave
// reduction.
__host__ __device__ inline int proxy_list_cap(int k_in, int ng) {
    return (k_in + ng + 1) / 2 * 2;   // kept rows + one pad per odd group, even
}
__host__ __device__ inline size_t proxy_list_bytes(int k_in, int ng, int nbt) {
    return align_up((size_t)proxy_list_cap(k_in, ng) * 2 * (1 + nbt), 16);
}
// One tile's scales, [ng][gate T | up T] fp16, follow the list.  With
// proxy_max_nb rows per launch list and scales fit in every case (k_in <= d:
// at most 115 KB at d = 8192 and 4 rows, 130 KB at d = 16384 and 1 row).
__host__ __device__ inline size_t proxy_scale_bytes(int ng, int T) { return (size_t)ng * 2 * T * 2; }
constexpr size_t kProxyDynLdsMax = 152 * 1024;   // the static tables take the rest
__host__ __device__ inline size_t proxy_lds_bytes(int k_in, int ng, int nbt, int T) {
    const size_t list = proxy_list_bytes(k_in, ng, nbt) + proxy_scale_bytes(ng, T);
    const size_t red = (size_t)kMaxBlockWaves * nbt * 2 * T * 4;
    const size_t m = list > red ? list : red;
    return m > kSelHistU16Bytes ? m : kSelHistU16Bytes;   // the selection's histogram first
}

// Columns each lane accumulates: 16 for one batch row of INT4 codes, else 8
// (register budget).
template <int NB>
struct ProxyCols {
    static constexpr int value = NB == 1 ? 16 : 8;
};
template <int NB, int QB>
constexpr int proxy_cols() { return QB == 4 ? ProxyCols<NB>::value : 8; }

template <int QB, int CPL>
struct ProxyLoad;   // bytes of one row a lane reads
template <> struct ProxyLoad<4, 16> { using type = uint2; };
template <> struct ProxyLoad<4, 8> { using type = uint32_t; };
template <> struct ProxyLoad<8, 16> { using type = uint4; };
template <> struct ProxyLoad<8, 8> { using type = uint2; };
template <> struct ProxyLoad<16, 8> { using type = uint4; };   // unquantised 16-bit proxy

template <int DT, int QB, int CPL, bool FUSED>
__device__ __forceinline__ void pair_accumulate(const typename ProxyLoad<QB, CPL>::type &a,
                                                const typename ProxyLoad<QB, CPL>::type &b,
                                                uint32_t xp, float *acc) {
    if constexpr (QB == 4 && CPL == 16) {
        int4_pair_dot8_h<FUSED>(a.x, b.x, xp, acc);
        int4_pair_dot8_h<FUSED>(a.y, b.y, xp, acc + 8);
    } else if constexpr (QB == 4) {
        int4_pair_dot8_h<FUSED>(a, b, xp, acc);
    } else if constexpr (QB == 8 && CPL == 16) {
        int8_pair_fma8<DT>(make_uint2(a.x, a.y), make_uint2(b.x, b.y), xp, acc);
        int8_pair_fma8<DT>(make_uint2(a.z, a.w), make_uint2(b.z, b.w), xp, acc + 8);
    } else if constexpr (QB == 8) {
        int8_pair_fma8<DT>(a, b, xp, acc);
    } else {
        // 16-bit weights: (w_a[c], w_b[c]) side by side, one dot2 with (x_a, x_b).
        const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            acc[2 * q] = dot2<DT>(xp, __builtin_amdgcn_perm(bw[q], aw[q], 0x05040100u), acc[2 * q]);
            acc[2 * q + 1] = dot2<DT>(xp, __builtin_amdgcn_perm(bw[q], aw[q], 0x07060302u), acc[2 * q + 1]);
        }
    }
}

template <int NB, int DT, int QB, int T, int C>
__global__ __launch_bounds__(kBlock) void proxy_kernel(
    const uint16_t *__restrict__ x_all, int B_all,  // every batch row (selection keys)
    int row0, int nb,                                 // rows [row0, row0 + nb) are projected
    int d, int f, int group, int k_in, const uint8_t *__restrict__ blob,
    uint8_t *__restrict__ in_mask, float *__restrict__ scores,
    int accumulate, Select sel_rule, int act) {   // k_in: the list capacity when sel_rule.tau_mode
    constexpr int CPL = proxy_cols<NB, QB>();
    constexpr int LPS = 2 * T / CPL;              // lanes per row segment (gate + up)
    constexpr int NGRP = kWave / LPS;             // lane groups per wave
    constexpr int NLG = kMaxBlockWaves * NGRP;    // lane groups per workgroup
    static_assert(C * kBlock <= kMaxDModel, "input rows per thread");
    constexpr int U = ((QB == 8 && NB == 4) || QB == 16) ? 4 : 8;   // row pairs in flight per lane group
    constexpr int SZ = CPL / 8;                   // uint4 of scales per lane and group
    constexpr bool kEarlyX = NB <= 2;             // projected x loaded with the keys
    constexpr bool kHoistX = NB == 1;             // x pairs read with the code loads
    constexpr float off = QB == 8 ? 128.0f : 0.0f;   // code bias (INT4: per column, kInt4HBias)
    constexpr bool kHx = QB == 4;                     // x in fp16 (INT4 codes dequantised in fp16)
    using W = typename ProxyLoad<QB, CPL>::type;
    const BlobLayout L(d, f, QB, group);
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();
    const int tile = stage1_tile<2 * T * QB / 8 < 128>(blockIdx.x, gridDim.x);
    const int ng = d / group;

    __shared__ SelScratch ss;
    __shared__ TopKOrder<C> ord;
    __shared__ int gsel0[kMaxDModel / 128 + 1];  // kept rows before each group
    __shared__ int gstart[kMaxDModel / 128 + 1]; // padded list position of each group
    extern __shared__ __align__(16) unsigned char dsm[];

    const int cap = proxy_list_cap(k_in, ng);
    uint16_t *rows_sh = reinterpret_cast<uint16_t *>(dsm);   // [cap]
    uint16_t *xs_sh = rows_sh + cap;                          // [NB][cap]

    // This tile's scales go to LDS behind the list: loaded here, held in
    // registers through the input selection, stored once its histogram is
    // dead.  A group change in the stream then waits on LDS only, never on
    // the global loads in flight.
    uint16_t *sc_sh = reinterpret_cast<uint16_t *>(dsm + proxy_list_bytes(k_in, ng, NB));
    const uint4 *tsc = reinterpret_cast<const uint4 *>(
        reinterpret_cast<const uint16_t *>(blob + L.scales_offset) + (size_t)tile * ng * 2 * T);
    const int nsc4 = ng * T / 4;                         // uint4 of this tile's scales
    constexpr int SPT = C * T / 512 > 1 ? C * T / 512 : 1;   // 1, 2 or 4 >= nsc4 / kBlock
    static_assert(SPT == 1 || SPT == 2 || SPT == 4, "scale vectors per thread");
    // Clamped indices keep every load in flight at once (a repeat stores the
    // same value); named registers, as an array here went to scratch.
    auto sc_idx = [&](int k) { return min(k * kBlock + tid, nsc4 - 1); };
    uint4 scr0 = tsc[sc_idx(0)], scr1, scr2, scr3;
    if constexpr (SPT > 1) scr1 = tsc[sc_idx(1)];
    if constexpr (SPT > 2) {
        scr2 = tsc[sc_idx(2)];
        scr3 = tsc[sc_idx(3)];
    }

    // ---- input top-k: item r of thread t is row r * kBlock + t ----
    // Key of row i: max over the batch of |x_i| as its 15-bit magnitude
    // pattern (monotone in |x| for fp16 and bf16, +0 and -0 equal).  Loads use
    // clamped indices and are masked afterwards, so all of them are in flight
    // at once.
    uint32_t key[C];
#pragma unroll
    for (int r = 0; r < C; ++r) key[r] = 0u;
    for (int b = 0; b < B_all; ++b) {
        const uint16_t *xb = x_all + (size_t)b * d;
        uint32_t raw[C];
#pragma unroll
        for (int r = 0; r < C; ++r) {
            raw[r] = xb[min(r * kBlock + tid, d - 1)];
        }
#pragma unroll
        for (int r = 0; r < C; ++r) {
            if (r * kBlock + tid < d) key[r] = max(key[r], raw[r] & 0x7FFFu);
        }
    }
    uint32_t xw[kEarlyX ? NB : 1][C / 2];   // x of the projected rows, two per word
    if constexpr (kEarlyX) {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const uint16_t *xb = x_all + (size_t)(row0 + min(b, nb - 1)) * d;
#pragma unroll
            for (int q = 0; q < C / 2; ++q) {
                xw[b][q] = (uint32_t)xb[min(2 * q * kBlock + tid, d - 1)] |
                           ((uint32_t)xb[min((2 * q + 1) * kBlock + tid, d - 1)] << 16);
            }
        }
    }
    // bf16 x for fp16-dequantised codes: the largest key sets the power of two
    // that takes the kept x into fp16 (per wave here, across waves after the
    // bookkeeping barrier; 15-bit magnitude patterns order like the values).
    constexpr bool kScaleX = kHx && DT == kBF16;
    __shared__ uint32_t wmax[kMaxBlockWaves];
    if constexpr (kScaleX) {
        uint32_t m = 0;
#pragma unroll
        for (int r = 0; r < C; ++r) m = max(m, key[r]);
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, o));
        if (lane == 0) wmax[wid] = m;
    }
    uint64_t sel = 0;
    if (sel_rule.tau_mode) {
        // Threshold rule: keep row i when max_b |x_{b,i}| >= tau_x, compared
        // as floats (exact for the 16-bit magnitudes).
#pragma unroll
        for (int r = 0; r < C; ++r) {
            const bool in = r * kBlock + tid < d && half_to_float<DT>((uint16_t)key[r]) >= sel_rule.tau;
            sel |= (uint64_t)in << r;
        }
        topk_order<kBlock, C>(sel, ord);
        if (tile == 0 && row0 == 0 && tid == 0 && sel_rule.count)
            *sel_rule.count = topk_selected_before<kBlock, C>(ord, C * kBlock);
    } else {
        topk_select_u15<kBlock, C>(key, d, k_in, reinterpret_cast<uint32_t *>(dsm), ss, ord);
    }

    // ---- group bookkeeping, one wave: kept rows before each group, padded
    // list starts, and for every (row, wave) entry of the order tables the
    // list position of its first kept input (into ord.off) ----
    // The 64 inputs of an entry share one quantisation group (group is a
    // multiple of 128), and a group boundary is an entry boundary, so the
    // kept rows before it are that entry's offset.  i / group is a 32-bit
    // reciprocal multiply: exact for i < 2^14 and group < 2^15 (the rounding
    // error i * group / 2^32 stays below 1 / group).
    const uint32_t gmagic = 0xFFFFFFFFu / (uint32_t)group + 1u;
    if (wid == 0) {
        const int total = topk_selected_before<kBlock, C>(ord, C * kBlock);
        auto before = [&](int gg) {
            const int i = gg * group;
            return i >= C * kBlock ? total : ord.off[(i / kBlock) * kMaxBlockWaves + (i % kBlock) / kWave];
        };
        int carry = 0;
        for (int g0 = 0; g0 <= ng; g0 += kWave) {
            const int g = g0 + lane;
            const int s0 = g <= ng ? before(g) : 0;
            const int cnt = g < ng ? before(g + 1) - s0 : 0;
            const int padded = (cnt + 1) / 2 * 2;
            const int incl = wave_inclusive_scan(padded);
            if (g <= ng) {
                gsel0[g] = s0;
                gstart[g] = carry + incl - padded;
            }
            carry += __builtin_amdgcn_readlane(incl, kWave - 1);
        }
        for (int e = lane; e < C * kMaxBlockWaves; e += kWave) {
            const uint32_t i0 = (uint32_t)((e / kMaxBlockWaves) * kBlock + (e % kMaxBlockWaves) * kWave);
            const int g = (int)__umulhi(i0, gmagic);
            ord.off[e] += gstart[g] - gsel0[g];
        }
    }
    __syncthreads();

    {
        uint4 *sc4 = reinterpret_cast<uint4 *>(sc_sh);
        sc4[sc_idx(0)] = scr0;
        if constexpr (SPT > 1) sc4[sc_idx(1)] = scr1;
        if constexpr (SPT > 2) {
            sc4[sc_idx(2)] = scr2;
            sc4[sc_idx(3)] = scr3;
        }
    }

    float xscale = 1.0f, xunscale = 1.0f;   // 2^s and 2^-s (bf16 x to fp16)
    if constexpr (kScaleX) {
        uint32_t m = 0;
#pragma unroll
        for (int w = 0; w < kMaxBlockWaves; ++w) m = max(m, wmax[w]);
        const int sx = min(100, max(-100, 141 - (int)(m >> 7)));   // 2^14 <= max |x| 2^s < 2^15
        xscale = __uint_as_float((uint32_t)(127 + sx) << 23);
        xunscale = __uint_as_float((uint32_t)(127 - sx) << 23);
    }

    // ---- kept rows to their padded list positions (x as 16-bit bits) ----
    // A kept input's position: its entry's first position plus its rank in
    // the entry (a lane count).
    const int swid = wave_id();
    int pos[C];   // list position of each of this thread's inputs, -1 if not kept
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const int i = r * kBlock + tid;
        const uint64_t bs = ord.sel[r][swid];
        const bool s = (bs >> lane) & 1;   // inputs past d are never kept
        pos[r] = s ? ord.off[r * kMaxBlockWaves + swid] + (int)lanes_below(bs) : -1;
        if (s) rows_sh[pos[r]] = (uint16_t)i;
    }
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        uint16_t xv[C];
        if constexpr (kEarlyX) {
#pragma unroll
            for (int r = 0; r < C; ++r) {
                xv[r] = (uint16_t)(xw[b][r / 2] >> (16 * (r & 1)));
            }
        } else {
            const uint16_t *xb = x_all + (size_t)(row0 + min(b, nb - 1)) * d;
#pragma unroll
            for (int r = 0; r < C; ++r) {
                xv[r] = xb[min(r * kBlock + tid, d - 1)];
            }
        }
#pragma unroll
        for (int r = 0; r < C; ++r) {
            if (pos[r] >= 0) {
                uint16_t v = b < nb ? xv[r] : (uint16_t)0;
                if constexpr (kScaleX) v = float_to_f16_rne(bf16_lo(v) * xscale);   // exact above 2^-28 of the largest
                xs_sh[b * cap + pos[r]] = v;
            }
        }
    }
    for (int g = tid; g < ng; g += kBlock) {
        const int cnt = gsel0[g + 1] - gsel0[g];
        if (cnt & 1) {   // zero-weight pad row keeps every pair inside one group
            const int p = gstart[g] + cnt;
            rows_sh[p] = (uint16_t)(g * group);
#pragma unroll
            for (int b = 0; b < NB; ++b) xs_sh[b * cap + p] = 0;
        }
    }
    __syncthreads();
    if (tile == 0 && in_mask) {   // after the last barrier: the stores overlap the stream
#pragma unroll
        for (int r = 0; r < C; ++r)
            if (r * kBlock + tid < d) in_mask[r * kBlock + tid] = pos[r] >= 0 ? 1 : 0;
    }

    // ---- stream the kept row pairs: lane group l owns a contiguous range ----
    // Per group the lane accumulates x_a (M + n_a) + x_b (M + n_b) and the x
    // sum; at a group change acc - (M + 8) * xsum is scaled into tot.
    const int npairs = gstart[ng] / 2;
    const int lgi = wid * NGRP + lane / LPS;
    const int pa = (int)((long long)lgi * npairs / NLG);
    const int pb = (int)((long long)(lgi + 1) * npairs / NLG);
    const uint32_t *rows32 = reinterpret_cast<const uint32_t *>(rows_sh);
    const uint32_t *xs32 = reinterpret_cast<const uint32_t *>(xs_sh);
    const int li = lane % LPS;
    const int mat = li / (LPS / 2);                 // 0: gate, 1: up
    const int colc = (li % (LPS / 2)) * CPL;        // first of this lane's columns
    const uint8_t *tbase = blob + L.codes_offset + (size_t)tile * L.row_bytes;
    const uint32_t rstride = (uint32_t)L.row_stride;   // < 2^24: 24-bit multiplies
    const uint32_t lane_off = (uint32_t)(mat * (T * QB / 8) + colc * QB / 8);

    float tot[NB][CPL];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < CPL; ++e) tot[b][e] = 0.0f;

    if (pa < pb) {
        int g = 0;
        while (gstart[g + 1] / 2 <= pa) ++g;
        int gend = gstart[g + 1] / 2;
        uint4 sc[SZ];
        auto load_sc = [&](int gg) {
            const uint4 *q = reinterpret_cast<const uint4 *>(sc_sh + (size_t)gg * 2 * T + mat * T + colc);
#pragma unroll
            for (int z = 0; z < SZ; ++z) sc[z] = q[z];
        };
        load_sc(g);
        float acc[NB][CPL], xs[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            xs[b] = 0.0f;
#pragma unroll
            for (int e = 0; e < CPL; ++e) acc[b][e] = 0.0f;
        }
        auto flush = [&]() {
#pragma unroll
            for (int z = 0; z < SZ; ++z) {
                const uint32_t sw[4] = {sc[z].x, sc[z].y, sc[z].z, sc[z].w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float sg = f16_bits_to_float((e & 1) ? (sw[e >> 1] >> 16) : (sw[e >> 1] & 0xFFFFu));
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const float offe = kHx ? kInt4HBias[e & 1] : off;
                        tot[b][z * 8 + e] = fmaf(sg, acc[b][z * 8 + e] - offe * xs[b], tot[b][z * 8 + e]);
                        acc[b][z * 8 + e] = 0.0f;
                    }
                }
            }
#pragma unroll
            for (int b = 0; b < NB; ++b) xs[b] = 0.0f;
        };
        for (int p0 = pa; p0 < pb; p0 += U) {
            // Unconditional loads (the tail repeats the last pair, with x = 0
            // below), so the compiler keeps all 2U loads in flight.
            W wa[U], wb[U];
            // x pairs read alongside (one batch row), so their LDS latency
            // overlaps the global loads instead of stalling each slot.
            uint32_t xpre[kHoistX ? U : 1];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int pc = min(p0 + u, pb - 1);
                const uint32_t rr = rows32[pc];
                wa[u] = *reinterpret_cast<const W *>(tbase + (__umul24(rr & 0xFFFFu, rstride) + lane_off));
                wb[u] = *reinterpret_cast<const W *>(tbase + (__umul24(rr >> 16, rstride) + lane_off));
                if constexpr (kHoistX) xpre[u] = xs32[pc];
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int p = p0 + u;
                {
                    if (p < pb && p >= gend) {
                        flush();
                        do { ++g; } while (gstart[g + 1] / 2 <= p);
                        load_sc(g);
                        gend = gstart[g + 1] / 2;
                    }
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        uint32_t xp;
                        if constexpr (kHoistX) xp = p < pb ? xpre[u] : 0u;
                        else xp = p < pb ? xs32[b * (cap / 2) + p] : 0u;
                        pair_accumulate<DT, QB, CPL, (NB <= 2)>(wa[u], wb[u], xp, acc[b]);
                        if constexpr (kHx) xs[b] = dot2<kF16>(xp, Int4Magic<kF16>::one, xs[b]);
                        else xs[b] = dot2<DT>(xp, Int4Magic<DT>::one, xs[b]);
                    }
                }
            }
        }
        flush();
    }
    if constexpr (kHx) {   // high-nibble columns / 16, and 2^-s: exact powers of two
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < CPL; ++e) tot[b][e] *= kInt4HScale[e & 1] * xunscale;
    }

    // ---- combine lane groups, then waves, in a fixed order ----
    static_assert(LPS == 8 || LPS == 16 || LPS == 32, "lane-group sizes");
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
        for (int e = 0; e < CPL; ++e) {
            float t = tot[b][e];
            if constexpr (LPS == 8) t += dpp_move<kDppRor8>(t);   // lane ^ 8
            if constexpr (LPS <= 16) t = add_swap16(t);
            tot[b][e] = add_swap32(t);
        }
    __syncthreads();   // the list is dead; reuse the LDS for the reduction
    float *red = reinterpret_cast<float *>(dsm);   // [16][NB][2T]
    if (lane < LPS) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < CPL; ++e) red[(wid * NB + b) * 2 * T + mat * T + colc + e] = tot[b][e];
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
            best = fmaxf(best, fabsf(gate_act(gu[0], act) * gu[1]));
        }
        if (j < f) scores[j] = accumulate ? fmaxf(scores[j], best) : best;
    }
}

template <int NB, int DT, int QB, int T, int C>
static hipError_t launch_proxy_t(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                 int group, int k_in, const void *blob,
                                 uint8_t *in_mask, float *scores, int accumulate, Select sel_rule, int act, hipStream_t s) {
    const BlobLayout L(d, f, QB, group);
    const size_t lds = proxy_lds_bytes(k_in, d / group, NB, T);
    if (lds > kProxyDynLdsMax) return hipErrorInvalidValue;   // excluded by proxy_max_nb
    if (lds > 65536) {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void *>(proxy_kernel<NB, DT, QB, T, C>),
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    proxy_kernel<NB, DT, QB, T, C><<<L.n_tiles, kBlock, lds, s>>>(
        static_cast<const uint16_t *>(x_all), B_all, row0, nb, d, f, group, k_in,
        static_cast<const uint8_t *>(blob), in_mask, scores, accumulate, sel_rule, act);
    return hipGetLastError();
}

// C = input rows per thread of the input top-k: 4 up to d = 4096, 8 up to
// 8192, else 16.
template <int NB, int DT, int QB, int T>
static hipError_t launch_proxy_c(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                 int group, int k_in, const void *blob,
                                 uint8_t *in_mask, float *scores, int accumulate, Select sel_rule, int act, hipStream_t s) {
    if (d <= 4 * kBlock)
        return launch_proxy_t<NB, DT, QB, T, 4>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
    if (d <= 8 * kBlock)
        return launch_proxy_t<NB, DT, QB, T, 8>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
    return launch_proxy_t<NB, DT, QB, T, 16>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
}

template <int DT, int QB, int T>
static hipError_t launch_proxy_nb(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                  int group, int k_in, const void *blob,
                                  uint8_t *in_mask, float *scores, int accumulate, Select sel_rule, int act, hipStream_t s) {
    switch (proxy_nb_t(nb)) {
        case 1: return launch_proxy_c<1, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
        case 2: return launch_proxy_c<2, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
        default: return launch_proxy_c<4, DT, QB, T>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
    }
}

template <int DT, int QB>
static hipError_t launch_proxy_tile(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                    int group, int k_in, const void *blob,
                                    uint8_t *in_mask, float *scores, int accumulate, Select sel_rule, int act,
                                    hipStream_t s) {
    if (proxy_tile(f) == 128)
        return launch_proxy_nb<DT, QB, 128>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
    return launch_proxy_nb<DT, QB, 64>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s);
}

int proxy_max_nb(int d) { return d <= 8192 ? kProxyMaxNB : 1; }

hipError_t launch_proxy(int dtype, int qbits, const void *x_all, int B_all, int row0, int nb,
                        int d, int f, int group, int k_in, const void *blob,
                        uint8_t *in_mask, float *scores, int accumulate, Select sel_rule, int act, hipStream_t s) {
#define PX(DT_, QB_) launch_proxy_tile<DT_, QB_>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel_rule, act, s)
    if (dtype == kBF16) return qbits == 4 ? PX(kBF16, 4) : qbits == 8 ? PX(kBF16, 8) : PX(kBF16, 16);
    return qbits == 4 ? PX(kF16, 4) : qbits == 8 ? PX(kF16, 8) : PX(kF16, 16);
#undef PX
}

}  // namespace prox
