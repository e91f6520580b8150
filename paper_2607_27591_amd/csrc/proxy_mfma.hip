// Stage 1 of the sparse decode step for several batch rows at once, on the
// matrix cores (Sec. 4.1 Stage 1 with the INT4 proxy of Sec. 3.2 / 4.3).  It
// computes what proxy_kernel computes (the same input selection, the same
// per-group scales and the same score) for up to 16 rows per launch, so the
// proxy codes of a kept input row are read once for all of them.
//
// The proxy GEMV of a column tile is a product of x (batch rows x kept input
// rows) with the dequantised codes (kept input rows x columns), done as
// 16 x 16 x 16 MFMAs (bf16 or fp16 operands, fp32 accumulation).  The kept-row
// list is padded per quantisation group to a multiple of 16, so one 16-row
// block never mixes groups.  A pad row repeats a kept row of its group (its
// codes come from lines that are read anyway) and has x = 0.
//
// Lane l of a wave feeds batch row l % 16 to the A operand and column set
// l % 16 to the B operand, for block rows 4 (l / 16) .. 4 (l / 16) + 3.  In a
// 64-column half of the tile and one matrix (gate or up, per wave) the lane
// owns columns 4n .. 4n + 3 (n = l % 16).  Per block it loads 2 bytes (4
// codes) from each of its 4 rows, pairs the rows, and ORs each nibble under
// the exponent of the magic constant M.  That gives the exact 16-bit pair
// (M + n_a, M + n_b), n = q + 8, and two such pairs are one B operand: 4 MFMAs
// per block.  Waves split the blocks of their half and matrix, so a wave may
// see only part of a group: a fifth MFMA per block, with B all ones, sums x
// over the blocks the wave has taken, in the accumulator layout, and at a
// group change the lane subtracts (M + 8) times that sum and applies the
// group's scale.  The waves' partial sums meet in LDS in wave order, so results are
// deterministic.
#include "common.hpp"
#include "kernels.hpp"
#include "topk.hpp"

namespace prox {

typedef unsigned short us2 __attribute__((ext_vector_type(2)));   // two rows' codes, one VGPR

constexpr int kMfmaBlock = 16;    // kept input rows per block (the MFMA's K)
constexpr int kMfmaU = 4;         // blocks in flight per wave


// Dynamic LDS: first the input selection's histogram; then rows [cap] u16,
// x [cap][NX] u16 (position-major), block groups [cap / 16] u16; after the stream the same space holds the cross-wave partial sums
// [16 waves][64 lanes][16] f32.
__host__ __device__ inline int mfma_list_cap(int k_in, int ng) {
    return (k_in + ng * (kMfmaBlock - 1) + kMfmaBlock - 1) / kMfmaBlock * kMfmaBlock;
}
__host__ __device__ inline size_t mfma_list_bytes(int cap, int nx) {
    return align_up((size_t)cap * 2, 16) + align_up((size_t)nx * cap * 2, 16) +
           align_up((size_t)(cap / kMfmaBlock) * 2, 16);
}
constexpr size_t kMfmaRedBytes = (size_t)kMaxBlockWaves * kWave * 16 * 4;   // 64 KiB
__host__ __device__ inline size_t mfma_lds_bytes(int k_in, int ng, int nx) {
    const size_t list = mfma_list_bytes(mfma_list_cap(k_in, ng), nx);
    const size_t m = list > kMfmaRedBytes ? list : kMfmaRedBytes;
    return m > kSelHistU16Bytes ? m : kSelHistU16Bytes;
}

template <int DT, int T, int C, int NX>
__global__ __launch_bounds__(kBlock) void proxy_mfma_kernel(
    const uint16_t *__restrict__ x_all, int B_all, int row0, int nb, int d, int f, int group,
    int k_in, const uint8_t *__restrict__ blob, uint8_t *__restrict__ in_mask,
    float *__restrict__ scores, int accumulate, Select sel_rule, int act,
    int32_t *__restrict__ klist, int list_mode) {   // kept-row list of a multi-launch call
    static_assert(T == 64 || T == 128, "tile widths of the blob layout");
    static_assert(NX == 8 || NX == 16, "x rows kept in LDS");
    constexpr int WH = T / 64;                       // 64-column halves per tile
    constexpr int WPG = kMaxBlockWaves / (WH * 2);   // waves per (half, matrix)
    constexpr uint32_t M = Int4Magic<DT>::pair;
    constexpr float off = Int4Magic<DT>::offset;
    const BlobLayout L(d, f, 4, group);
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();
    const int tile = stage1_tile<T == 64>(blockIdx.x, gridDim.x);   // INT4 codes
    const int ng = d / group;

    __shared__ SelScratch ss;
    __shared__ TopKOrder<C> ord;
    __shared__ int gsel0[kMaxDModel / 128 + 1];   // kept rows before each group
    __shared__ int gstart[kMaxDModel / 128 + 1];  // padded list position of each group
    extern __shared__ __align__(16) unsigned char dsm[];

    const int cap = mfma_list_cap(k_in, ng);
    uint16_t *rows_sh = reinterpret_cast<uint16_t *>(dsm);
    uint16_t *xs_sh = reinterpret_cast<uint16_t *>(dsm + align_up((size_t)cap * 2, 16));
    uint16_t *kbg_sh = reinterpret_cast<uint16_t *>(dsm + align_up((size_t)cap * 2, 16) +
                                                    align_up((size_t)NX * cap * 2, 16));

    // List start of each group: the kept counts padded to whole blocks, scanned.
    auto group_starts = [&]() {
        if (wid == 0) {
            int carry = 0;
            for (int g0 = 0; g0 <= ng; g0 += kWave) {
                const int g = g0 + lane;
                const int cnt = g < ng ? gsel0[g + 1] - gsel0[g] : 0;
                const int padded = (cnt + kMfmaBlock - 1) / kMfmaBlock * kMfmaBlock;
                const int incl = wave_inclusive_scan(padded);
                if (g <= ng) gstart[g] = carry + incl - padded;
                carry += __builtin_amdgcn_readlane(incl, kWave - 1);
            }
        }
        __syncthreads();
    };
    const uint32_t gmagic = 0xFFFFFFFFu / (uint32_t)group + 1u;   // i / group, exact here
    int pos[C];   // list position of each of this thread's inputs, -1 if not kept
#pragma unroll
    for (int r = 0; r < C; ++r) pos[r] = -1;
    if (list_mode == kListRead) {
        // Another launch of this call selected: its list (ascending kept rows,
        // count at klist[d]) gives the same groups and list positions.
        const int n = klist[d];
        for (int g = tid; g <= ng; g += kBlock) {   // kept rows below g * group
            const int v = g * group;
            int lo = 0, hi = n;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (klist[mid] < v) lo = mid + 1;
                else hi = mid;
            }
            gsel0[g] = lo;
        }
        __syncthreads();
        group_starts();
        for (int idx = tid; idx < n; idx += kBlock) {
            const int i = klist[idx];
            const int g = (int)__umulhi((uint32_t)i, gmagic);
            const int p = gstart[g] + idx - gsel0[g];
            rows_sh[p] = (uint16_t)i;
            for (int b = 0; b < nb; ++b) xs_sh[(size_t)p * NX + b] = x_all[(size_t)(row0 + b) * d + i];
        }
    } else {
        // ---- input selection (as proxy_kernel): key = max_b |x_{b,i}| bits ----
        // x is read XQ rows at a time, two rows' 16-bit values per register,
        // so a round's loads are in flight together (XQ * C = 64 values in 32
        // registers per thread: one round trip for 16 rows of d <= 4096; two
        // rows at a time for d > 8192, where registers are short).
        constexpr int XQ = C <= 8 ? 64 / C : 2;
        uint32_t key[C];
    #pragma unroll
        for (int r = 0; r < C; ++r) key[r] = 0u;
        // With 4 inputs per thread one round holds all 16 rows: a single
        // launch keeps them in registers for the list instead of reloading.
        constexpr bool kKeepX = C == 4;
        uint32_t raw[XQ / 2][C];
        for (int b0 = 0; b0 < B_all; b0 += XQ) {
    #pragma unroll
            for (int q = 0; q < XQ / 2; ++q) {
                const uint16_t *xa = x_all + (size_t)min(b0 + 2 * q, B_all - 1) * d;
                const uint16_t *xc = x_all + (size_t)min(b0 + 2 * q + 1, B_all - 1) * d;
    #pragma unroll
                for (int r = 0; r < C; ++r)
                    raw[q][r] = (uint32_t)xa[min(r * kBlock + tid, d - 1)] |
                                ((uint32_t)xc[min(r * kBlock + tid, d - 1)] << 16);
            }
    #pragma unroll
            for (int q = 0; q < XQ / 2; ++q)
    #pragma unroll
                for (int r = 0; r < C; ++r)
                    if (r * kBlock + tid < d)
                        key[r] = max(key[r], max(raw[q][r] & 0x7FFFu, (raw[q][r] >> 16) & 0x7FFFu));
        }
        uint64_t sel = 0;
        if (sel_rule.tau_mode) {
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

        // ---- groups: kept rows per group, list starts padded to whole blocks ----
        for (int g = tid; g <= ng; g += kBlock) gsel0[g] = topk_selected_before<kBlock, C>(ord, g * group);
        __syncthreads();
        group_starts();

        // ---- kept rows and their x values to the list ----
        // The 64 inputs of a (row, wave) share one quantisation group: a kept
        // input's position is wave-uniform table entries plus a lane count.
        const int swid = wave_id();
    #pragma unroll
        for (int r = 0; r < C; ++r) {
            const int i = r * kBlock + tid;
            const uint64_t bs = ord.sel[r][swid];
            const int g = (int)__umulhi((uint32_t)(r * kBlock + swid * kWave), gmagic);
            const bool s = (bs >> lane) & 1;   // inputs past d are never kept
            pos[r] = s ? gstart[g] - gsel0[g] + ord.off[r * kMaxBlockWaves + swid] +
                             (int)lanes_below(bs)
                       : -1;
            if (s) rows_sh[pos[r]] = (uint16_t)i;
        }
        // Only the nb real batch rows are stored: the stream feeds zeros for the
        // others.  XL rows at a time, only the kept inputs loaded, all of a
        // round in flight together.
        constexpr int XL = 32 / C;   // rows per round: 32 values per thread
        if (kKeepX && B_all <= XQ && row0 == 0 && nb == B_all) {
            // raw[q][r] already holds rows 2q and 2q + 1 side by side: NX rows
            // of a kept input are NX / 8 16-byte stores (rows past nb hold
            // copies, never read).
    #pragma unroll
            for (int r = 0; r < C; ++r)
                if (pos[r] >= 0) {
                    uint4 *dst = reinterpret_cast<uint4 *>(xs_sh + (size_t)pos[r] * NX);
    #pragma unroll
                    for (int h = 0; h < NX / 8; ++h)
                        dst[h] = make_uint4(raw[4 * h][r], raw[4 * h + 1][r], raw[4 * h + 2][r], raw[4 * h + 3][r]);
                }
        } else
        for (int b0 = 0; b0 < nb; b0 += XL) {
            uint16_t xv[XL][C];
    #pragma unroll
            for (int q = 0; q < XL; ++q) {
                const uint16_t *xb = x_all + (size_t)(row0 + min(b0 + q, nb - 1)) * d;
    #pragma unroll
                for (int r = 0; r < C; ++r) xv[q][r] = pos[r] >= 0 ? xb[min(r * kBlock + tid, d - 1)] : (uint16_t)0;
            }
            // The round's XL rows of a kept input are contiguous: one store
            // (rows past nb hold copies, never read; b0 + XL <= NX).
    #pragma unroll
            for (int r = 0; r < C; ++r)
                if (pos[r] >= 0) {
                    uint32_t w[XL / 2];
    #pragma unroll
                    for (int q = 0; q < XL / 2; ++q)
                        w[q] = (uint32_t)xv[2 * q][r] | ((uint32_t)xv[2 * q + 1][r] << 16);
                    uint16_t *dst = xs_sh + (size_t)pos[r] * NX + b0;
                    if constexpr (XL == 8)
                        *reinterpret_cast<uint4 *>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
                    else if constexpr (XL == 4)
                        *reinterpret_cast<uint2 *>(dst) = make_uint2(w[0], w[1]);
                    else
                        *reinterpret_cast<uint32_t *>(dst) = w[0];
                }
        }
        if (list_mode == kListWrite && tile == 0) {   // the list for the later launches
#pragma unroll
            for (int r = 0; r < C; ++r)
                if (pos[r] >= 0) klist[topk_pos<C>(ord, r)] = r * kBlock + tid;
            if (tid == 0) klist[d] = gsel0[ng];
        }
    }
    __syncthreads();   // the kept rows are in place: pads copy the group's last one
    // Pads, one thread per (group, pad slot): at most 15 per group.
    for (int it = tid; it < ng * kMfmaBlock; it += kBlock) {
        const int g = it / kMfmaBlock, j = it % kMfmaBlock;
        const int cnt = gsel0[g + 1] - gsel0[g];
        const int p0 = gstart[g], p = p0 + cnt + j;
        if (p < gstart[g + 1]) {   // a pad only when cnt > 0
            rows_sh[p] = rows_sh[p0 + cnt - 1];
            uint4 *dst = reinterpret_cast<uint4 *>(xs_sh + (size_t)p * NX);
#pragma unroll
            for (int h = 0; h < NX / 8; ++h) dst[h] = make_uint4(0u, 0u, 0u, 0u);
        }
    }
    // The group of every 16-row block: the last g with gstart[g] <= its start.
    const int nkb_all = gstart[ng] / kMfmaBlock;
    for (int kb = tid; kb < nkb_all; kb += kBlock) {
        int lo = 0, hi = ng - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (gstart[mid] <= kb * kMfmaBlock) lo = mid;
            else hi = mid - 1;
        }
        kbg_sh[kb] = (uint16_t)lo;
    }
    __syncthreads();
    if (tile == 0 && in_mask && list_mode != kListRead) {   // stores overlap the stream
#pragma unroll
        for (int r = 0; r < C; ++r)
            if (r * kBlock + tid < d) in_mask[r * kBlock + tid] = pos[r] >= 0 ? 1 : 0;
    }

    // ---- stream the blocks: this wave's half and share of the blocks ----
    const int nkb = gstart[ng] / kMfmaBlock;
    const int hm = wid / WPG, wi = wid % WPG;
    const int h = hm / 2, mat = hm % 2;             // column half, matrix (0 gate, 1 up)
    const int kb0 = (int)((long long)wi * nkb / WPG), kb1 = (int)((long long)(wi + 1) * nkb / WPG);
    const int ln = lane % 16, lg = lane / 16;
    const uint8_t *tbase = blob + L.codes_offset + (size_t)tile * L.row_bytes + mat * (T / 2) +
                           h * 32 + ln * 2;
    const uint16_t *sbase = reinterpret_cast<const uint16_t *>(blob + L.scales_offset) +
                            (size_t)tile * ng * 2 * T + (size_t)mat * T + h * 64 + ln * 4;
    const uint32_t rstride = (uint32_t)L.row_stride;

    v4f acc[4], tot[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        acc[c] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
        tot[c] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    }
    v4f xacc = v4f{0.0f, 0.0f, 0.0f, 0.0f};   // x sums of this wave's blocks, current group
    const uint2 ones = make_uint2(Int4Magic<DT>::one, Int4Magic<DT>::one);

    if (kb0 < kb1) {
        int gcur = kbg_sh[kb0];
        // this lane's 4 fp16 scales of the current group
        uint2 sc = *reinterpret_cast<const uint2 *>(sbase + (size_t)gcur * 2 * T);
        auto flush = [&]() {
            const uint32_t sw[2] = {sc.x, sc.y};
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float s = f16_bits_to_float((c & 1) ? (sw[c >> 1] >> 16) : (sw[c >> 1] & 0xFFFFu));
#pragma unroll
                for (int j = 0; j < 4; ++j) tot[c][j] = fmaf(s, acc[c][j] - off * xacc[j], tot[c][j]);
                acc[c] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
            }
            xacc = v4f{0.0f, 0.0f, 0.0f, 0.0f};
        };
        for (int kb = kb0; kb < kb1; kb += kMfmaU) {
            // All loads first (the tail repeats the last block, unused).
            us2 code[kMfmaU][2];   // [block]: rows (0, 1) and (2, 3)
            uint2 xa[kMfmaU];
            int gk[kMfmaU];
#pragma unroll
            for (int u = 0; u < kMfmaU; ++u) {
                const int k = min(kb + u, kb1 - 1);
                const uint2 rr = *reinterpret_cast<const uint2 *>(rows_sh + k * kMfmaBlock + lg * 4);
                const uint32_t r4[4] = {rr.x & 0xFFFFu, rr.x >> 16, rr.y & 0xFFFFu, rr.y >> 16};
                // x of batch row ln at the block's rows 4 lg .. 4 lg + 3
                // (position-major: NX rows per kept position).
                const uint16_t *xq = xs_sh + (size_t)(k * kMfmaBlock + lg * 4) * NX + min(ln, NX - 1);
                xa[u] = ln < nb ? make_uint2((uint32_t)xq[0] | ((uint32_t)xq[NX] << 16),
                                             (uint32_t)xq[2 * NX] | ((uint32_t)xq[3 * NX] << 16))
                                : make_uint2(0u, 0u);
                gk[u] = kbg_sh[k];
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    code[u][q].x = *reinterpret_cast<const uint16_t *>(tbase + r4[2 * q] * rstride);
                    code[u][q].y = *reinterpret_cast<const uint16_t *>(tbase + r4[2 * q + 1] * rstride);
                }
            }
#pragma unroll
            for (int u = 0; u < kMfmaU; ++u) {
                if (kb + u >= kb1) break;   // uniform
                if (gk[u] != gcur) {
                    flush();
                    gcur = gk[u];
                    sc = *reinterpret_cast<const uint2 *>(sbase + (size_t)gcur * 2 * T);
                }
                xacc = mfma16<DT>(xa[u], ones, xacc);   // x sums of rows 4 lg + j
                const uint32_t p01 = __builtin_bit_cast(uint32_t, code[u][0]);   // rows a, b
                const uint32_t p23 = __builtin_bit_cast(uint32_t, code[u][1]);   // rows c, d
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint2 bop = make_uint2(((p01 >> (4 * c)) & 0x000F000Fu) | M,
                                                 ((p23 >> (4 * c)) & 0x000F000Fu) | M);
                    acc[c] = mfma16<DT>(xa[u], bop, acc[c]);
                }
            }
        }
        flush();
    }

    // ---- partial sums of the waves meet in LDS, in wave order ----
    __syncthreads();   // the list is dead
    float *red = reinterpret_cast<float *>(dsm);   // [wave][lane][c * 4 + j]
#pragma unroll
    for (int c = 0; c < 4; ++c)
        *reinterpret_cast<float4 *>(red + ((size_t)(wid * kWave + lane) * 16 + c * 4)) =
            make_float4(tot[c][0], tot[c][1], tot[c][2], tot[c][3]);
    __syncthreads();
    // Every (row b, column col): the sums of the WPG waves of the gate and of
    // the up matrix in wave order, then |act(g~) u~|, then the max over the 16
    // rows inside each 16-lane row of the wave (lane % 16 = b, one column).
    const int b = tid % 16;
#pragma unroll
    for (int q = 0; q < T / 64; ++q) {
        const int col = tid / 16 + q * 64;
        const int hh = col / 64, cl = col % 64;
        const int src = ((b / 4) * 16 + cl / 4) * 16 + (cl % 4) * 4 + b % 4;   // lane, c, j
        const float *rg = red + (size_t)(hh * 2 + 0) * WPG * kWave * 16 + src;
        const float *ru = red + (size_t)(hh * 2 + 1) * WPG * kWave * 16 + src;
        float gs = 0.0f, us = 0.0f;
        for (int w2 = 0; w2 < WPG; ++w2) {
            gs += rg[(size_t)w2 * kWave * 16];
            us += ru[(size_t)w2 * kWave * 16];
        }
        float v = b < nb ? fabsf(gate_act(gs, act) * us) : 0.0f;
        v = fmaxf(v, dpp_move<kDppXor1>(v));
        v = fmaxf(v, dpp_move<kDppXor2>(v));
        v = fmaxf(v, dpp_move<kDppRor4>(v));
        v = fmaxf(v, dpp_move<kDppRor8>(v));
        const int j = tile * T + col;
        if (b == 0 && j < f) scores[j] = accumulate ? fmaxf(scores[j], v) : v;
    }
}

// ---------------------------------------------------------------------------
// Launcher
// ---------------------------------------------------------------------------

int proxy_mfma_rows(int d, int group, int k_in) {
    const int ng = d / group;
    const size_t limit = 136 * 1024;   // dynamic LDS beside the ~22 KiB of statics
    if (mfma_lds_bytes(k_in, ng, 16) <= limit) return 16;
    if (mfma_lds_bytes(k_in, ng, 8) <= limit) return 8;
    return 0;
}

template <int DT, int T, int C, int NX>
static hipError_t launch_mfma_t(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                int group, int k_in, const void *blob, uint8_t *in_mask,
                                float *scores, int accumulate, Select sel, int act,
                                int32_t *klist, int list_mode, hipStream_t s) {
    const BlobLayout L(d, f, 4, group);
    const size_t lds = mfma_lds_bytes(k_in, d / group, NX);
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void *>(proxy_mfma_kernel<DT, T, C, NX>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    proxy_mfma_kernel<DT, T, C, NX><<<L.n_tiles, kBlock, lds, s>>>(
        static_cast<const uint16_t *>(x_all), B_all, row0, nb, d, f, group, k_in,
        static_cast<const uint8_t *>(blob), in_mask, scores, accumulate, sel, act, klist, list_mode);
    return hipGetLastError();
}

template <int DT, int T>
static hipError_t launch_mfma_c(const void *x_all, int B_all, int row0, int nb, int d, int f,
                                int group, int k_in, const void *blob, uint8_t *in_mask,
                                float *scores, int accumulate, Select sel, int act,
                                int32_t *klist, int list_mode, hipStream_t s) {
    const int nx = proxy_mfma_rows(d, group, k_in);
#define MF(C_, NX_) launch_mfma_t<DT, T, C_, NX_>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel, act, klist, list_mode, s)
    if (d <= 4 * kBlock) return nx == 16 ? MF(4, 16) : MF(4, 8);
    if (d <= 8 * kBlock) return nx == 16 ? MF(8, 16) : MF(8, 8);
    return nx == 16 ? MF(16, 16) : MF(16, 8);
#undef MF
}

hipError_t launch_proxy_mfma(int dtype, const void *x_all, int B_all, int row0, int nb, int d,
                             int f, int group, int k_in, const void *blob, uint8_t *in_mask,
                             float *scores, int accumulate, Select sel, int act, int32_t *klist,
                             int list_mode, hipStream_t s) {
    if (nb < 1 || nb > proxy_mfma_rows(d, group, k_in)) return hipErrorInvalidValue;
    if (list_mode != kListNone && !klist) return hipErrorInvalidValue;
    if (proxy_tile(f) == 128)
        return dtype == kBF16 ? launch_mfma_c<kBF16, 128>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel, act, klist, list_mode, s)
                              : launch_mfma_c<kF16, 128>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel, act, klist, list_mode, s);
    return dtype == kBF16 ? launch_mfma_c<kBF16, 64>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel, act, klist, list_mode, s)
                          : launch_mfma_c<kF16, 64>(x_all, B_all, row0, nb, d, f, group, k_in, blob, in_mask, scores, accumulate, sel, act, klist, list_mode, s);
}

}  // namespace prox
