// Stage 2 of the sparse decode step (Sec. 4.1 Stage 2) and the dense FFN
// (Sec. 2.1), which runs the same kernel over every channel.
//
// stage2_kernel, one workgroup per equal slice of the kept channels:
//  prologue  (sparse only) every workgroup finds the channel threshold of the
//            top-k_ff proxy scores itself, and the ascending global position
//            of every kept channel, so it can take exactly its slice of the
//            kept list (balanced to +-1 channel) without another launch.  When
//            a batch takes several launches, the first writes the kept list
//            to the workspace and the later ones read their slice from it.
//  gate/up   the slice's channels are cut into (channel, part of d) units
//            spread over the 16 waves; each unit streams two contiguous rows
//            with 16-byte loads and dot2 instructions (fp32 accumulation);
//            s_j = act(g_j) u_j is kept in LDS in fp32.
//  down      every thread owns 8 output columns and accumulates
//            s_j W_down[j, c..c+8] over the slice; the workgroup writes one
//            partial y.
// With INT4 base weights (WQ = 4) the two streaming loops read codes and
// per-group scales instead of 16-bit rows and dequantise on the fly.
// stage2_mfma_kernel and stage2_down_kernel (below) take batches of more than
// 8 rows of 16-bit weights.
// reduce_kernel sums the partial y of all workgroups in workgroup order and
// rounds y once.  No floating-point atomics: results are deterministic.
#include "common.hpp"
#include "kernels.hpp"
#include "topk.hpp"

namespace prox {

constexpr int kMaxSlice = (kMaxDFF + kStage2MaxWGs - 1) / kStage2MaxWGs;   // channels per WG
constexpr int kMaxParts = 8;

// d is cut into Q parts for the gate/up units: each part >= 2048 columns of
// 16-bit weights (up to four 16-byte loads per lane and matrix); with INT4
// codes, a power of two of equal parts of at most 4096 columns, so a part is
// one round of two 16-byte loads per lane and matrix.
__host__ __device__ inline int gateup_parts(int d, int nbt, int wq) {
    if (nbt > 2) return 1;
    if (wq == 4) {
        int q = 1;
        while (q * 4096 < d && q < kMaxParts) q *= 2;
        return q;
    }
    const int q = d / 2048;
    return q < 1 ? 1 : (q > kMaxParts ? kMaxParts : q);
}

__host__ __device__ inline bool x_in_lds(int d, int nbt) { return (size_t)nbt * d <= 32768; }

// Thread groups sharing the down projection's channels (> 1 only when d/8 <
// the block size), summed through LDS.
__host__ __device__ inline int stage2_down_groups(int d, int nbt) {
    const int ncg = d / 8;
    return (ncg >= kBlock || nbt > 4) ? 1 : kBlock / ncg;
}

// Dynamic LDS ahead of s: x (when staged; with INT4 weights as permuted
// pairs plus two sums per 32 inputs) or the down reduction buffer.
__host__ __device__ inline size_t stage2_head_bytes(int d, int nbt, int wq) {
    const size_t xbytes = x_in_lds(d, nbt) ? (size_t)nbt * d * 2 + (wq == 4 ? (size_t)nbt * (d / 32) * 8 : 0)
                                           : 0;
    const size_t red = stage2_down_groups(d, nbt) > 1 ? (size_t)(d / 8) * nbt * 8 * 4 : 0;
    return xbytes > red ? xbytes : red;
}

// Score keys of one thread (item r = channel r * kBlock + base): the high
// halves in registers, the complete key re-read from the scores
// (L2-resident) when the high half ties.
struct Stage2Smem {
    int list[kMaxSlice];
    float gu[kMaxSlice * kMaxParts * 2 * 2];   // [t][q][b][2] for nbt <= 2
};

// The selection prologue of both Stage 2 kernels: this workgroup's slice of the
// kept channels (their ids to list[0..n), n returned, the slice's first
// kept-list position to p0_out) and its chunk of the mask.
// Every workgroup ranks the scores itself (top-k or the threshold rule), or,
// for the later launches of a multi-launch batch, reads the first launch's list.
// The caller synchronises before reading list.
template <int C>
__device__ __forceinline__ int stage2_slice(const float *__restrict__ scores, int f, int k_ff,
                                            uint8_t *__restrict__ mask,
                                            float *__restrict__ scores_copy, Select sel_rule,
                                            int32_t *__restrict__ klist, int klist_mode,
                                            uint32_t *hist, SelScratch &ss, TopKOrder<C> &ord,
                                            int *list, int &p0_out) {
    const int tid = threadIdx.x;
    const int nwg = gridDim.x, w = blockIdx.x;
    const bool sparse = scores != nullptr;
    // Channels of this workgroup: an even share of the n_ch kept channels
    // (with the threshold rule n_ch is only known after the selection).
    int n_ch = sparse ? k_ff : f;
    int p0 = (int)((long long)w * n_ch / nwg), p1 = (int)((long long)(w + 1) * n_ch / nwg);
    int n = p1 - p0;


    // ---- prologue: this workgroup's slice of the kept channels ----
    if (sparse && klist_mode == kListRead) {
        // A launch for the same call already selected: its list gives the
        // same slice as ranking again would.
        n_ch = klist[f];
        if (sel_rule.tau_mode) {
            const int nwg_k = min(nwg, stage2_wgs(n_ch));
            p0 = w < nwg_k ? (int)((long long)w * n_ch / nwg_k) : n_ch;
            p1 = w < nwg_k ? (int)((long long)(w + 1) * n_ch / nwg_k) : n_ch;
            n = p1 - p0;
        }
        for (int t = tid; t < n; t += kBlock) list[t] = klist[p0 + t];
        __syncthreads();
    } else if (sparse) {
        // Item r of thread t is channel r * kBlock + t (coalesced loads).
        // Scores are |s~| >= 0, so their IEEE bit patterns order like the
        // values; channels past f get key 0.
        uint32_t key[C];
#pragma unroll
        for (int r = 0; r < C; ++r) {
            key[r] = r * kBlock + tid < f ? __float_as_uint(scores[r * kBlock + tid]) : 0u;
        }
        uint64_t sel = 0;
        if (sel_rule.tau_mode) {
            // Threshold rule: keep channel j when score_j >= tau_s.
#pragma unroll
            for (int r = 0; r < C; ++r)
                sel |= (uint64_t)(r * kBlock + tid < f && __uint_as_float(key[r]) >= sel_rule.tau) << r;
            topk_order<kBlock, C>(sel, ord);
            n_ch = topk_selected_before<kBlock, C>(ord, C * kBlock);
            // Split over the workgroups a launch for this count would have
            // (the grid is sized for every channel; the rest get none), so
            // the partial sums are those of the top-k launch with k = n_ch.
            const int nwg_k = min(nwg, stage2_wgs(n_ch));
            p0 = w < nwg_k ? (int)((long long)w * n_ch / nwg_k) : n_ch;
            p1 = w < nwg_k ? (int)((long long)(w + 1) * n_ch / nwg_k) : n_ch;
            n = p1 - p0;
            if (w == 0 && tid == 0 && sel_rule.count) *sel_rule.count = n_ch;
        } else {
            topk_select_f32<kBlock, C>(key, f, k_ff, hist, ss, ord);
        }
        // This workgroup's slice of positions straight from the order tables.
        // The (row, wave) entry holding position p0 is found by one thread;
        // then wave v expands entries e0 + v, e0 + v + 16, ... lane by lane
        // (lane l: bit l of the entry's ballot, its position by a lane count)
        // until the entries pass p1.
        if (n > 0) {
            if (tid < C * kMaxBlockWaves) {
                const int pos = ord.off[tid];
                const int cnt = __popcll(ord.sel[tid / kMaxBlockWaves][tid % kMaxBlockWaves]);
                if (pos <= p0 && p0 < pos + cnt) ss.pick[0] = tid;   // exactly one entry
            }
            __syncthreads();
            const int wid = wave_id(), lane = lane_id();
            for (int e = ss.pick[0] + wid; e < C * kMaxBlockWaves; e += kMaxBlockWaves) {
                const int pos = ord.off[e];   // wave-uniform
                if (pos >= p1) break;
                const uint64_t m = ord.sel[e / kMaxBlockWaves][e % kMaxBlockWaves];
                const int q = pos + (int)lanes_below(m);
                if (((m >> lane) & 1) && q >= p0 && q < p1) {
                    const int j = min((e / kMaxBlockWaves) * kBlock + (e % kMaxBlockWaves) * kWave + lane,
                                      f - 1);   // rows in bounds
                    list[q - p0] = j;
                    if (klist_mode == kListWrite) klist[q] = j;
                }
            }
        }
        if (klist_mode == kListWrite && w == 0 && tid == 0) klist[f] = n_ch;
        (void)sel;
        __syncthreads();
    } else {
        for (int t = tid; t < n; t += kBlock) list[t] = p0 + t;
    }
    p0_out = p0;
    return n;
}

// This workgroup's chunk of the channel mask (and of the score copy) from
// the order tables of a launch that selected.  Called after the prologue's
// last barrier, so the stores overlap the weight stream instead of holding a
// barrier until they are acknowledged.
template <int C>
__device__ __forceinline__ void stage2_mask_chunk(const TopKOrder<C> &ord, const float *scores,
                                                  int f, uint8_t *mask, float *scores_copy,
                                                  int klist_mode) {
    if (!scores || klist_mode == kListRead) return;
    const int nwg = gridDim.x, w = blockIdx.x;
    const int mchunk = (f + nwg - 1) / nwg;   // mask entries written by this workgroup
    const int m_lo = w * mchunk, m_hi = min(m_lo + mchunk, f);
    for (int i = m_lo + (int)threadIdx.x; i < m_hi; i += kBlock) {
        mask[i] = topk_is_selected<kBlock, C>(ord, i) ? 1 : 0;
        if (scores_copy) scores_copy[i] = scores[i];
    }
}

// WQ: 16 for 16-bit weights, 4 for INT4 codes (wt.sg/su/sd: their scales).
template <int NB, int DT, int C, int WQ>
__global__ __launch_bounds__(kBlock) void stage2_kernel(
    const uint16_t *__restrict__ x, int nb, int d, int f, Stage2Weights wt,
    const float *__restrict__ scores,   // NULL: dense FFN over all f channels
    int k_ff, uint8_t *__restrict__ mask, float *__restrict__ scores_copy,
    float *__restrict__ ypart, int ypart_stride,   // partial y rows per workgroup
    Select sel_rule, int act,                       // act: gate activation
    int32_t *__restrict__ klist, int klist_mode) {  // kept-channel list, KeptList mode
    static_assert(WQ == 16 || WQ == 4, "16-bit or INT4 weights");
    const uint16_t *__restrict__ wg = static_cast<const uint16_t *>(wt.wg);
    const uint16_t *__restrict__ wu = static_cast<const uint16_t *>(wt.wu);
    const uint16_t *__restrict__ wd = static_cast<const uint16_t *>(wt.wd);
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();

    __shared__ SelScratch ss;
    __shared__ TopKOrder<C> ord;
    __shared__ Stage2Smem sm;
    // The channel selection's histogram, then x [NB][d] or the down reduction
    // | s [slice][NB].
    extern __shared__ __align__(16) float dyn[];

    // x (when it goes to LDS) is loaded before the selection, so its load
    // latency hides behind the ranking, and stored once the selection's
    // histogram is dead; with 64 score rows per thread the registers are
    // short, and x is loaded after it.  Thread t holds uint4 number
    // k * kBlock + t of the [NB][d / 8] vectors.
    const bool xl = x_in_lds(d, NB);   // always true with INT4 weights (host-checked)
    const int nvec = d / 8;
    constexpr int XPT = NB * kMaxDModel / 8 / kBlock < 4 ? NB * kMaxDModel / 8 / kBlock : 4;
    static_assert(XPT * kBlock * 8 >= 32768 || XPT * kBlock * 8 >= NB * kMaxDModel,
                  "x vectors per thread cover every x that fits in LDS");
    constexpr bool kEarlyX = C <= 32;
    uint4 xr[XPT];
    auto load_x = [&]() {
#pragma unroll
        for (int k = 0; k < XPT; ++k) {
            const int e = k * kBlock + tid, b = e / nvec;
            xr[k] = xl && e < NB * nvec && b < nb
                        ? reinterpret_cast<const uint4 *>(x + (size_t)b * d)[e % nvec]
                        : make_uint4(0, 0, 0, 0);
        }
    };
    if constexpr (kEarlyX) load_x();

    int p0;
    const int n = stage2_slice<C>(scores, f, k_ff, mask, scores_copy, sel_rule, klist,
                                  klist_mode, reinterpret_cast<uint32_t *>(dyn), ss, ord,
                                  sm.list, p0);
    (void)p0;
    if constexpr (!kEarlyX) load_x();

    uint16_t *xs = reinterpret_cast<uint16_t *>(dyn);
    float2 *xsum = reinterpret_cast<float2 *>(dyn + (size_t)NB * d / 2);   // INT4: [NB][d / 32]
    if constexpr (WQ == 4) {
        // x as pairs (x_{8m+k}, x_{8m+k+4}), k = 0..3, one uint4 per 8
        // inputs: nibble k of a code word and nibble k + 4 sit in the two
        // halves of the word at the same bit offsets, so one dot2 takes both.
        // Per 32 inputs, the sums of x over the even-k pairs (the low halves
        // of the input words) and the odd-k pairs (the high halves): 4 per
        // lane in order, then the four lanes of a 32-input run (consecutive
        // threads) as (s0 + s1) + (s2 + s3).
#pragma unroll
        for (int k = 0; k < XPT; ++k) {
            const int e = k * kBlock + tid;
            const uint4 v = xr[k];
            if (e < NB * nvec)
                reinterpret_cast<uint4 *>(xs)[e] = make_uint4(
                    __builtin_amdgcn_perm(v.z, v.x, 0x05040100u), __builtin_amdgcn_perm(v.z, v.x, 0x07060302u),
                    __builtin_amdgcn_perm(v.w, v.y, 0x05040100u), __builtin_amdgcn_perm(v.w, v.y, 0x07060302u));
            const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
            float se = 0.0f, so = 0.0f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                se += lo_to_float<DT>(vw[q]);
                so += hi_to_float<DT>(vw[q]);
            }
            se += dpp_move<kDppXor1>(se);
            so += dpp_move<kDppXor1>(so);
            se += dpp_move<kDppXor2>(se);
            so += dpp_move<kDppXor2>(so);
            if (e < NB * nvec && (tid & 3) == 0) xsum[e / 4] = make_float2(se, so);
        }
    } else if (xl) {
#pragma unroll
        for (int k = 0; k < XPT; ++k) {
            const int e = k * kBlock + tid;
            if (e < NB * nvec) reinterpret_cast<uint4 *>(xs)[e] = xr[k];
        }
    }
    __syncthreads();
    stage2_mask_chunk<C>(ord, scores, f, mask, scores_copy, klist_mode);

    // ---- gate/up: units (channel t, part q) over the 16 waves ----
    const int Q = gateup_parts(d, NB, WQ);
    float *s_sh = dyn + align_up(stage2_head_bytes(d, NB, WQ), 16) / 4;   // [slice][NB]
    if constexpr (WQ == 4) {
        // 16-byte code vectors (32 inputs, inside one group) per row.  Each
        // code word's nibbles go under the exponent of the magic constant M
        // in pairs (k, k + 4): the even-k pairs from the low nibble of a byte
        // (value M + n), the odd-k pairs from its high nibble, moved only to
        // the top of the 16-bit mantissa (M + 8n for bf16 after one shift,
        // M + 16n in place for fp16).  Per vector and batch row the dot2 sums
        // t_e, t_o then give sum x (n - 8) = (t_e - B_e X_e) + (t_o - B_o X_o) / s
        // with the even and odd x sums X_e, X_o, and the group scale
        // multiplies that into the row's total.
        constexpr uint32_t M = Int4Magic<DT>::pair;
        constexpr bool kBf = DT == kBF16;
        constexpr uint32_t kOddMask = kBf ? 0x00780078u : 0x00F000F0u;
        constexpr int kOddShift = kBf ? 1 : 0;
        constexpr float kBiasE = kBf ? 136.0f : 1032.0f;                   // M + 8
        constexpr float kBiasO = kBf ? 128.0f + 64.0f : 1024.0f + 128.0f;  // M + 8 s
        constexpr float kInvO = kBf ? 0.125f : 0.0625f;                     // 1 / s
        const int ng = d / wt.group;
        const int nv4 = d / 32;
        // Scale index of vector v: v / (group / 32) by a multiply (exact for
        // v < 2^16).
        const uint32_t smagic = 0xFFFFFFFFu / (uint32_t)(wt.group / 32) + 1u;
        const uint4 *xs4 = reinterpret_cast<const uint4 *>(xs);
        constexpr int U = 2;   // vectors per lane and matrix in one round
        // One round of a unit: the codes and group scales of U vectors of
        // both rows.
        struct Round {
            uint4 g[U], u[U];
            uint16_t sg[U], su[U];
        };
        // Q is a power of two here: unit = t Q + q by shifts.
        const int lq = __builtin_ctz((unsigned)Q);
        auto part = [&](int q, int &v_begin, int &v_end) {
            v_begin = (q * nv4) >> lq;
            v_end = ((q + 1) * nv4) >> lq;
        };
        // The loads are issued unconditionally (lanes past the part read its
        // last vector, whose data consume skips), so the compiler can wait
        // for exactly the loads of the round it consumes while the next
        // round's are in flight.
        auto issue = [&](int unit, int v0, Round &R) {
            const int t = unit >> lq, q = unit & (Q - 1);
            const int j = sm.list[t];
            const uint4 *rg = reinterpret_cast<const uint4 *>(static_cast<const uint8_t *>(wt.wg) + (size_t)j * (d / 2));
            const uint4 *ru = reinterpret_cast<const uint4 *>(static_cast<const uint8_t *>(wt.wu) + (size_t)j * (d / 2));
            const uint16_t *sgr = wt.sg + (size_t)j * ng, *sur = wt.su + (size_t)j * ng;
            int v_begin, v_end;
            part(q, v_begin, v_end);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int vv = min(v_begin + v0 + u * kWave, v_end - 1);
                R.g[u] = load_stream16(rg + vv);
                R.u[u] = load_stream16(ru + vv);
                const int si = (int)__umulhi((uint32_t)vv, smagic);
                R.sg[u] = sgr[si];
                R.su[u] = sur[si];
            }
        };
        // Branch-free as well: a lane past the part computes on the part's
        // last vector with scale 0.
        auto consume = [&](int unit, int v0, const Round &R, float (&ag)[NB], float (&au)[NB]) {
            int v_begin, v_end;
            part(unit & (Q - 1), v_begin, v_end);
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const bool in = v_begin + v0 + u * kWave < v_end;
                const int vv = min(v_begin + v0 + u * kWave, v_end - 1);
                {
                    const float scg = in ? f16_bits_to_float(R.sg[u]) : 0.0f;
                    const float scu = in ? f16_bits_to_float(R.su[u]) : 0.0f;
                    const uint32_t cgw[4] = {R.g[u].x, R.g[u].y, R.g[u].z, R.g[u].w};
                    const uint32_t cuw[4] = {R.u[u].x, R.u[u].y, R.u[u].z, R.u[u].w};
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        float tge = 0.0f, tgo = 0.0f, tue = 0.0f, tuo = 0.0f;
#pragma unroll
                        for (int w4 = 0; w4 < 4; ++w4) {
                            const uint4 P = xs4[(size_t)b * nvec + vv * 4 + w4];
                            const uint32_t g8 = cgw[w4] >> 8, u8 = cuw[w4] >> 8;
                            tge = dot2<DT>(P.x, and_or<true>(cgw[w4], 0x000F000Fu, M), tge);
                            tue = dot2<DT>(P.x, and_or<true>(cuw[w4], 0x000F000Fu, M), tue);
                            tgo = dot2<DT>(P.y, and_or<true>(cgw[w4] >> kOddShift, kOddMask, M), tgo);
                            tuo = dot2<DT>(P.y, and_or<true>(cuw[w4] >> kOddShift, kOddMask, M), tuo);
                            tge = dot2<DT>(P.z, and_or<true>(g8, 0x000F000Fu, M), tge);
                            tue = dot2<DT>(P.z, and_or<true>(u8, 0x000F000Fu, M), tue);
                            tgo = dot2<DT>(P.w, and_or<true>(g8 >> kOddShift, kOddMask, M), tgo);
                            tuo = dot2<DT>(P.w, and_or<true>(u8 >> kOddShift, kOddMask, M), tuo);
                        }
                        const float2 xv = xsum[b * nv4 + vv];
                        const float ge = tge - kBiasE * xv.x, go = tgo - kBiasO * xv.y;
                        const float ue = tue - kBiasE * xv.x, uo = tuo - kBiasO * xv.y;
                        ag[b] = fmaf(scg, fmaf(go, kInvO, ge), ag[b]);
                        au[b] = fmaf(scu, fmaf(uo, kInvO, ue), au[b]);
                    }
                }
            }
        };
        auto finish = [&](int unit, float (&ag)[NB], float (&au)[NB]) {
            const int t = unit >> lq, q = unit & (Q - 1);
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const float gs = wave_sum(ag[b]);
                const float us = wave_sum(au[b]);
                if (lane == 0) {
                    if (Q == 1) {
                        s_sh[t * NB + b] = gate_act(gs, act) * us;
                    } else {
                        sm.gu[((t * Q + q) * 2 + b) * 2 + 0] = gs;
                        sm.gu[((t * Q + q) * 2 + b) * 2 + 1] = us;
                    }
                }
            }
        };
        const int nunits = n * Q;
        if constexpr (NB == 1) {
            // A unit is one round (a part holds at most U * kWave vectors).
            // The wave's next unit is loaded before this one is computed, so
            // its load latency hides behind this unit's dequant and dot
            // products; two register sets take turns.
            auto run = [&](int unit, const Round &cur, Round &nxt) {
                // The last unit of the wave loads itself again (unused).
                issue(min(unit + kMaxBlockWaves, nunits - 1), lane, nxt);
                float ag[NB], au[NB];
#pragma unroll
                for (int b = 0; b < NB; ++b) ag[b] = au[b] = 0.0f;
                consume(unit, lane, cur, ag, au);
                finish(unit, ag, au);
            };
            Round ra, rb;
            // Nothing loaded before the loop is left in flight, so the waits
            // inside it only ever count the loop's own loads.
            __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            // The loop leaves at either half, so its back edge is taken only
            // after both register sets were consumed in turn (unit and count
            // wave-uniform, so the branches are scalar).
            int unit = __builtin_amdgcn_readfirstlane(wid);
            const int nu = __builtin_amdgcn_readfirstlane(nunits);
            if (unit < nu) {
                issue(unit, lane, ra);
                while (true) {
                    run(unit, ra, rb);
                    unit += kMaxBlockWaves;
                    if (unit >= nu) break;
                    run(unit, rb, ra);
                    unit += kMaxBlockWaves;
                    if (unit >= nu) break;
                }
            }
        } else {
            for (int unit = wid; unit < nunits; unit += kMaxBlockWaves) {
                int v_begin, v_end;
                part(unit & (Q - 1), v_begin, v_end);
                float ag[NB], au[NB];
#pragma unroll
                for (int b = 0; b < NB; ++b) ag[b] = au[b] = 0.0f;
                for (int v0 = lane; v_begin + v0 < v_end; v0 += kWave * U) {
                    Round R;
                    issue(unit, v0, R);
                    consume(unit, v0, R, ag, au);
                }
                finish(unit, ag, au);
            }
        }
    } else {
    const int qv = nvec / Q;                                   // 16-byte vectors per part
    constexpr int U = 4;
    for (int unit = wid; unit < n * Q; unit += kMaxBlockWaves) {
        const int t = unit / Q, q = unit % Q;
        const int j = sm.list[t];
        const uint4 *rg = reinterpret_cast<const uint4 *>(wg + (size_t)j * d);
        const uint4 *ru = reinterpret_cast<const uint4 *>(wu + (size_t)j * d);
        const int v_begin = q * qv, v_end = (q == Q - 1) ? nvec : v_begin + qv;
        float ag[NB], au[NB];
#pragma unroll
        for (int b = 0; b < NB; ++b) ag[b] = au[b] = 0.0f;
        for (int v0 = v_begin + lane; v0 < v_end; v0 += kWave * U) {
            uint4 gv[U], uv[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (v0 + u * kWave < v_end) {
                    gv[u] = load_stream16(rg + v0 + u * kWave);
                    uv[u] = load_stream16(ru + v0 + u * kWave);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int vv = v0 + u * kWave;
                if (vv < v_end) {
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        uint4 xv;
                        if (xl) xv = reinterpret_cast<const uint4 *>(xs)[b * nvec + vv];
                        else xv = b < nb ? reinterpret_cast<const uint4 *>(x + (size_t)b * d)[vv]
                                         : make_uint4(0, 0, 0, 0);
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
            if (lane == 0) {
                if (Q == 1) {
                    s_sh[t * NB + b] = gate_act(gs, act) * us;
                } else {
                    sm.gu[((t * Q + q) * 2 + b) * 2 + 0] = gs;
                    sm.gu[((t * Q + q) * 2 + b) * 2 + 1] = us;
                }
            }
        }
    }
    }
    __syncthreads();
    if (Q > 1) {
        for (int e = tid; e < n * NB; e += kBlock) {
            const int t = e / NB, b = e % NB;
            float gs = 0.0f, us = 0.0f;
            for (int q = 0; q < Q; ++q) {
                gs += sm.gu[((t * Q + q) * 2 + b) * 2 + 0];
                us += sm.gu[((t * Q + q) * 2 + b) * 2 + 1];
            }
            s_sh[t * NB + b] = gate_act(gs, act) * us;
        }
        __syncthreads();
    }

    // ---- down: partial y over this slice ----
    // d/8 groups of 8 columns; with fewer groups than threads (and NB <= 4)
    // the channels are split over G thread groups, summed through LDS in
    // group order.
    const int ncg = d / 8;
    constexpr int UD = 8;
    if constexpr (WQ == 16 && NB == 8) {
        // Eight batch rows up to d = 4096: 4 columns per thread, so that every
        // thread takes part (split channel sums would need more registers than
        // eight rows leave).  Each column is still summed over the slice in
        // order by one thread, as below.
        if (ncg < kBlock && d / 4 <= kBlock) {
            const int c4 = tid;
            if (c4 < d / 4) {
                float acc[NB][4];
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[b][e] = 0.0f;
                for (int t0 = 0; t0 < n; t0 += UD) {
                    uint2 wv[UD];
#pragma unroll
                    for (int u = 0; u < UD; ++u) {
                        const int t = t0 + u;
                        if (t < n) wv[u] = load_stream8(wd + (size_t)sm.list[t] * d + c4 * 4);
                    }
#pragma unroll
                    for (int u = 0; u < UD; ++u) {
                        const int t = t0 + u;
                        if (t < n) {
                            const float wf[4] = {lo_to_float<DT>(wv[u].x), hi_to_float<DT>(wv[u].x),
                                                 lo_to_float<DT>(wv[u].y), hi_to_float<DT>(wv[u].y)};
#pragma unroll
                            for (int b = 0; b < NB; ++b) {
                                const float sv = s_sh[t * NB + b];
#pragma unroll
                                for (int e = 0; e < 4; ++e) acc[b][e] = fmaf(sv, wf[e], acc[b][e]);
                            }
                        }
                    }
                }
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    if (b < nb)
                        *reinterpret_cast<float4 *>(ypart + ((size_t)blockIdx.x * ypart_stride + b) * d + c4 * 4) =
                            make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
                }
            }
            return;
        }
    }
    const int G = stage2_down_groups(d, NB);
    const int stride = G > 1 ? ncg : kBlock;
    const int gi = tid / stride, cgt = tid % stride;
    // Reuses the x area: [NB][8][ncg], so that the threads of a wave (adjacent
    // column groups) store to adjacent words.
    float *dred = dyn;
    for (int cg0 = 0; cg0 < ncg; cg0 += stride) {
        const int cg = cg0 + cgt;
        const bool active = cg < ncg && gi < G;
        float acc[NB][8];
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[b][e] = 0.0f;
        if constexpr (WQ == 4) {
            // 8 columns per thread: one 32-bit code word and the scale of
            // their group per channel row.  The word's nibbles go under the
            // exponent of 1024.0 in fp16 pairs (columns e, e + 4): even e
            // from the low nibble of a byte (1024 + n), odd e from its high
            // nibble in place (1024 + 16 n); mixed-precision FMAs take each
            // half straight into the fp32 sums.  With S = sum_j s_j sigma_j,
            // sum_j s_j sigma_j (n - 8) is acc - 1032 S (even e) or
            // (acc - 1152 S) / 16 (odd e).
            const int ng = d / wt.group;
            constexpr uint32_t M16 = Int4Magic<kF16>::pair;
            constexpr int UD4 = NB == 1 ? 8 : 4;   // rows per round: 4 bytes each
            const uint32_t smagic = 0xFFFFFFFFu / (uint32_t)(wt.group / 8) + 1u;
            const int si = (int)__umulhi((uint32_t)cg, smagic);   // cg * 8 / group
            float ssum[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) ssum[b] = 0.0f;
            // One round: UD4 rows of this thread group's channels, loaded
            // unconditionally (rows past n repeat the last one and get s = 0)
            // so the loop can keep the next round in flight while it
            // computes this one.
            struct DRound {
                uint32_t cw[UD4];
                uint16_t sb[UD4];
            };
            auto issue = [&](int t0, DRound &R) {
#pragma unroll
                for (int u = 0; u < UD4; ++u) {
                    const int j = sm.list[min(t0 + u * G, n - 1)];
                    R.cw[u] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(
                        static_cast<const uint8_t *>(wt.wd) + (size_t)j * (d / 2) + cg * 4));
                    R.sb[u] = wt.sd[(size_t)j * ng + si];
                }
            };
            auto consume = [&](int t0, const DRound &R) {
#pragma unroll
                for (int u = 0; u < UD4; ++u) {
                    const int t = t0 + u * G;
                    const float sc = t < n ? f16_bits_to_float(R.sb[u]) : 0.0f;
                    const int tc = min(t, n - 1);
                    const uint32_t w8 = R.cw[u] >> 8;
                    const uint32_t h[4] = {and_or<true>(R.cw[u], 0x000F000Fu, M16),
                                           and_or<true>(R.cw[u], 0x00F000F0u, M16),
                                           and_or<true>(w8, 0x000F000Fu, M16),
                                           and_or<true>(w8, 0x00F000F0u, M16)};
#pragma unroll
                    for (int b = 0; b < NB; ++b) {
                        const float sv = s_sh[tc * NB + b] * sc;
                        ssum[b] += sv;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            acc[b][e] = fmaf(sv, lo_to_float<kF16>(h[e]), acc[b][e]);
                            acc[b][e + 4] = fmaf(sv, hi_to_float<kF16>(h[e]), acc[b][e + 4]);
                        }
                    }
                }
            };
            // The loop leaves at either half, so its back edge follows the
            // use of both register sets.
            auto rounds = [&](int t0) {
                const int step = G * UD4;
                DRound ra, rb;
                issue(t0, ra);
                while (true) {
                    issue(min(t0 + step, n - 1), rb);
                    consume(t0, ra);
                    t0 += step;
                    if (t0 >= n) break;
                    issue(min(t0 + step, n - 1), ra);
                    consume(t0, rb);
                    t0 += step;
                    if (t0 >= n) break;
                }
            };
            if (active && n > 0) {
                // Thread groups of whole waves (the usual case) take scalar
                // round starts, and the loop's branches are uniform.
                if (stride % kWave == 0) rounds(__builtin_amdgcn_readfirstlane(gi));
                else rounds(gi);
            }
            // acc[b][e] is column 8 cg + e: columns e < 4 from the low halves
            // of the fp16 pairs, e + 4 from the high halves; odd columns came
            // from high nibbles.
#pragma unroll
            for (int b = 0; b < NB; ++b)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc[b][e] = (e & 1) ? (acc[b][e] - 1152.0f * ssum[b]) * 0.0625f
                                        : acc[b][e] - 1032.0f * ssum[b];
        } else if (active) {
            for (int t0 = gi; t0 < n; t0 += G * UD) {
                uint4 wv[UD];
#pragma unroll
                for (int u = 0; u < UD; ++u) {
                    const int t = t0 + u * G;
                    if (t < n) wv[u] = load_stream16(wd + (size_t)sm.list[t] * d + cg * 8);
                }
#pragma unroll
                for (int u = 0; u < UD; ++u) {
                    const int t = t0 + u * G;
                    if (t < n) {
                        const uint32_t w4[4] = {wv[u].x, wv[u].y, wv[u].z, wv[u].w};
                        float wf[8];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            wf[2 * q] = lo_to_float<DT>(w4[q]);
                            wf[2 * q + 1] = hi_to_float<DT>(w4[q]);
                        }
#pragma unroll
                        for (int b = 0; b < NB; ++b) {
                            const float sv = s_sh[t * NB + b];
#pragma unroll
                            for (int e = 0; e < 8; ++e) acc[b][e] = fmaf(sv, wf[e], acc[b][e]);
                        }
                    }
                }
            }
        }
        if (G > 1) {
            // G > 1 implies ncg < kBlock, so this body runs exactly once and
            // every thread reaches these barriers.
            __syncthreads();   // x (aliased by dred) is no longer read
            for (int g2 = 0; g2 < G; ++g2) {
                if (active && gi == g2) {
#pragma unroll
                    for (int b = 0; b < NB; ++b)
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            float *dst = &dred[(b * 8 + e) * ncg + cg];
                            *dst = g2 == 0 ? acc[b][e] : *dst + acc[b][e];
                        }
                }
                __syncthreads();
            }
            if (active && gi == 0) {
#pragma unroll
                for (int b = 0; b < NB; ++b)
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[b][e] = dred[(b * 8 + e) * ncg + cg];
            }
        }
        if (active && gi == 0) {
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                if (b < nb) {
                    float4 *dst = reinterpret_cast<float4 *>(ypart + ((size_t)blockIdx.x * ypart_stride + b) * d + cg * 8);
                    dst[0] = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
                    dst[1] = make_float4(acc[b][4], acc[b][5], acc[b][6], acc[b][7]);
                }
            }
        }
    }
}

// ---------------------------------------------------------------------------
// stage2_mfma_kernel + stage2_down_kernel: Stage 2 for up to 16 batch rows of
// 16-bit weights, so every kept row of the three matrices is read once for
// all of them.
//  prologue  the slice of kept channels, as in stage2_kernel.
//  gate/up   on the matrix cores: the slice is cut into tiles of 16 channels,
//            and wave w takes the w-th sixteenth of d for every tile, so the
//            waves stream equal bytes however few channels the slice holds.
//            Per 32 inputs a lane loads 16 contiguous bytes of one channel row
//            of each matrix (A) and of one batch row of x (B, from L2), and two
//            16 x 16 x 16 MFMAs per matrix add the products into the tile's
//            [16 channels][16 rows] fp32 sums.  The 16 waves' sums of a tile
//            are added through LDS in wave order; s = act(g) u goes to the
//            workspace at the channel's kept-list position.
//  down      a second launch: the kept list is cut into kStage2DownGroups
//            groups, and each workgroup takes one group and 1024 columns,
//            with the group's s in LDS; every thread owns 4 columns and all 16
//            rows (VALU), and four thread groups split the channels.  With 64
//            groups the partial y are a quarter of what one partial per Stage 2
//            workgroup would be: at 16 rows those are as large as the weights
//            the step reads.
// ---------------------------------------------------------------------------
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
constexpr int kS2mTiles = 2;   // channel tiles per pass through the gate/up loop
constexpr int kS2mRed = kS2mTiles * 2 * kMaxBlockWaves * kWave;   // float4 per pass

size_t stage2_mfma_lds_bytes() {
    return (size_t)kS2mRed * 16 > kSelHistF32Bytes ? (size_t)kS2mRed * 16 : kSelHistF32Bytes;
}

bool stage2_mfma_ok(int d, int wq) { return stage2_mfma_shape(d, wq); }

template <int DT, int C>
__global__ __launch_bounds__(kBlock) void stage2_mfma_kernel(
    const uint16_t *__restrict__ x, int nb, int d, int f, Stage2Weights wt,
    const float *__restrict__ scores, int k_ff, uint8_t *__restrict__ mask,
    float *__restrict__ scores_copy, float *__restrict__ sbuf, Select sel_rule, int act,
    int32_t *__restrict__ klist, int klist_mode) {
    constexpr int R = kStage2MfmaRows;
    const uint16_t *__restrict__ wg = static_cast<const uint16_t *>(wt.wg);
    const uint16_t *__restrict__ wu = static_cast<const uint16_t *>(wt.wu);
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();

    __shared__ SelScratch ss;
    __shared__ TopKOrder<C> ord;
    __shared__ int list[kMaxSlice];
    // The channel selection's histogram, then red [tiles][2][waves][lanes] float4.
    extern __shared__ __align__(16) float dyn[];
    float4 *red = reinterpret_cast<float4 *>(dyn);

    int p0;
    const int n = stage2_slice<C>(scores, f, k_ff, mask, scores_copy, sel_rule, klist,
                                  klist_mode, reinterpret_cast<uint32_t *>(dyn), ss, ord, list,
                                  p0);
    __syncthreads();
    stage2_mask_chunk<C>(ord, scores, f, mask, scores_copy, klist_mode);

    // ---- gate/up ----
    const int nsteps = d / 32;   // steps of 32 inputs
    const int k_lo = wid * nsteps / kMaxBlockWaves, k_hi = (wid + 1) * nsteps / kMaxBlockWaves;
    const int r = lane % 16, g4 = lane / 16;
    const bool xrow = r < nb;
    const uint16_t *xr = x + (size_t)(xrow ? r : 0) * d + 8 * g4;
    const int ntiles = (n + 15) / 16;
    constexpr int U = 2;   // steps in flight per lane
    for (int t0 = 0; t0 < ntiles; t0 += kS2mTiles) {
        const uint16_t *rg[kS2mTiles], *ru[kS2mTiles];
        bool live[kS2mTiles];
        v4f ag[kS2mTiles], au[kS2mTiles];
#pragma unroll
        for (int tt = 0; tt < kS2mTiles; ++tt) {
            const int t = (t0 + tt) * 16 + r;
            live[tt] = t < n;
            const int j = live[tt] ? list[t] : 0;
            rg[tt] = wg + (size_t)j * d + 8 * g4;
            ru[tt] = wu + (size_t)j * d + 8 * g4;
            ag[tt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
            au[tt] = ag[tt];
        }
        for (int k = k_lo; k < k_hi; k += U) {
            uint4 xv[U], gv[kS2mTiles][U], uv[kS2mTiles][U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int kk = k + u;
                const bool in = kk < k_hi;
                xv[u] = in && xrow ? *reinterpret_cast<const uint4 *>(xr + kk * 32) : make_uint4(0, 0, 0, 0);
#pragma unroll
                for (int tt = 0; tt < kS2mTiles; ++tt) {
                    const bool ld = in && live[tt];
                    gv[tt][u] = ld ? load_stream16(rg[tt] + kk * 32) : make_uint4(0, 0, 0, 0);
                    uv[tt][u] = ld ? load_stream16(ru[tt] + kk * 32) : make_uint4(0, 0, 0, 0);
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                // Inputs 8 g4 + 0..3 of the step in the first MFMA, 8 g4 + 4..7
                // in the second: A and B take the same inputs in the same slots.
                const uint2 xa = make_uint2(xv[u].x, xv[u].y), xb = make_uint2(xv[u].z, xv[u].w);
#pragma unroll
                for (int tt = 0; tt < kS2mTiles; ++tt) {
                    ag[tt] = mfma16<DT>(make_uint2(gv[tt][u].x, gv[tt][u].y), xa, ag[tt]);
                    ag[tt] = mfma16<DT>(make_uint2(gv[tt][u].z, gv[tt][u].w), xb, ag[tt]);
                    au[tt] = mfma16<DT>(make_uint2(uv[tt][u].x, uv[tt][u].y), xa, au[tt]);
                    au[tt] = mfma16<DT>(make_uint2(uv[tt][u].z, uv[tt][u].w), xb, au[tt]);
                }
            }
        }
        // Lane l holds channel 4 (l / 16) + e, batch row l % 16 of each tile.
#pragma unroll
        for (int tt = 0; tt < kS2mTiles; ++tt) {
            red[((tt * 2 + 0) * kMaxBlockWaves + wid) * kWave + lane] =
                make_float4(ag[tt][0], ag[tt][1], ag[tt][2], ag[tt][3]);
            red[((tt * 2 + 1) * kMaxBlockWaves + wid) * kWave + lane] =
                make_float4(au[tt][0], au[tt][1], au[tt][2], au[tt][3]);
        }
        __syncthreads();
        if (tid < kS2mTiles * kWave * 4) {
            const int tt = tid / (kWave * 4), ln = (tid / 4) % kWave, e = tid % 4;
            const float *rf = reinterpret_cast<const float *>(red);
            float gs = 0.0f, us = 0.0f;
            for (int w = 0; w < kMaxBlockWaves; ++w) {
                gs += rf[(((tt * 2 + 0) * kMaxBlockWaves + w) * kWave + ln) * 4 + e];
                us += rf[(((tt * 2 + 1) * kMaxBlockWaves + w) * kWave + ln) * 4 + e];
            }
            const int t = (t0 + tt) * 16 + 4 * (ln / 16) + e;
            if (t < n) sbuf[(size_t)(p0 + t) * R + ln % 16] = gate_act(gs, act) * us;
        }
        __syncthreads();
    }
}

constexpr int kDownCols = 256;              // 4-column groups per workgroup: 1024 columns
constexpr int kDownSplit = kBlock / kDownCols;   // thread groups splitting its channels

size_t stage2_down_lds_bytes(int n_max) {
    const size_t m = (size_t)(n_max + kStage2DownGroups - 1) / kStage2DownGroups;
    return (size_t)kStage2MfmaRows * kDownCols * 16 + m * (kStage2MfmaRows * 4 + 4);
}

template <int DT>
__global__ __launch_bounds__(kBlock) void stage2_down_kernel(
    int nb, int d, int f, const uint16_t *__restrict__ wd, const float *__restrict__ sbuf,
    const int32_t *__restrict__ klist, float *__restrict__ ypart, int ypart_stride) {
    constexpr int R = kStage2MfmaRows;
    extern __shared__ __align__(16) float dyn[];   // red [R][kDownCols] float4 | s [m][R] | ids [m]
    const int tid = threadIdx.x;
    const int n_ch = klist ? klist[f] : f;
    const int grp = blockIdx.y;
    const int q0 = (int)((long long)grp * n_ch / kStage2DownGroups);
    const int m = (int)((long long)(grp + 1) * n_ch / kStage2DownGroups) - q0;
    float4 *red = reinterpret_cast<float4 *>(dyn);
    float *s_l = dyn + (size_t)R * kDownCols * 4;
    int *ids = reinterpret_cast<int *>(s_l + (size_t)m * R);
    for (int e = tid; e < m * R; e += kBlock) s_l[e] = sbuf[(size_t)q0 * R + e];
    for (int t = tid; t < m; t += kBlock) ids[t] = klist ? klist[q0 + t] : q0 + t;
    __syncthreads();

    // Thread group sub takes channels sub, sub + kDownSplit, ... of the group.
    const int sub = tid / kDownCols, cgl = tid % kDownCols;
    const int cg = blockIdx.x * kDownCols + cgl;   // columns 4 cg .. 4 cg + 3
    const bool active = cg < d / 4;
    constexpr int UD = 12;   // rows in flight
    float acc[R][4];
#pragma unroll
    for (int b = 0; b < R; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[b][e] = 0.0f;
    if (active) {
        for (int t0 = sub; t0 < m; t0 += kDownSplit * UD) {
            uint2 wv[UD];
#pragma unroll
            for (int u = 0; u < UD; ++u) {
                const int t = t0 + u * kDownSplit;
                if (t < m) {
                    const u32x2 v = __builtin_nontemporal_load(
                        reinterpret_cast<const u32x2 *>(wd + (size_t)ids[t] * d + cg * 4));
                    wv[u] = make_uint2(v.x, v.y);
                }
            }
#pragma unroll
            for (int u = 0; u < UD; ++u) {
                const int t = t0 + u * kDownSplit;
                if (t < m) {
                    const float wf[4] = {lo_to_float<DT>(wv[u].x), hi_to_float<DT>(wv[u].x),
                                         lo_to_float<DT>(wv[u].y), hi_to_float<DT>(wv[u].y)};
#pragma unroll
                    for (int b = 0; b < R; ++b) {
                        const float sv = s_l[t * R + b];
#pragma unroll
                        for (int e = 0; e < 4; ++e) acc[b][e] = fmaf(sv, wf[e], acc[b][e]);
                    }
                }
            }
        }
    }
    // The thread groups' sums are added in group order through LDS; every
    // thread reaches every barrier.
    for (int g2 = 0; g2 < kDownSplit - 1; ++g2) {
        if (sub == g2) {
#pragma unroll
            for (int b = 0; b < R; ++b) {
                float4 v = make_float4(acc[b][0], acc[b][1], acc[b][2], acc[b][3]);
                if (g2 > 0) {
                    const float4 o = red[b * kDownCols + cgl];
                    v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
                }
                red[b * kDownCols + cgl] = v;
            }
        }
        __syncthreads();
    }
    if (sub == kDownSplit - 1 && active) {
#pragma unroll
        for (int b = 0; b < R; ++b) {
            if (b < nb) {
                const float4 o = red[b * kDownCols + cgl];
                float4 *dst = reinterpret_cast<float4 *>(
                    ypart + ((size_t)grp * ypart_stride + b) * d + cg * 4);
                *dst = make_float4(o.x + acc[b][0], o.y + acc[b][1], o.z + acc[b][2],
                                   o.w + acc[b][3]);
            }
        }
    }
}

// y[b][c] = sum over the Stage 2 workgroups of the partial y, rounded once.
// A 256-thread block covers kReduceCols columns; thread t takes column
// t % kReduceCols and every kReduceGroups-th workgroup from t / kReduceCols,
// with all its loads in flight at once, and the groups are added in a fixed
// order through LDS, so the result is deterministic.
constexpr int kReduceThreads = 256;
constexpr int kReduceCols = 32;
constexpr int kReduceGroups = kReduceThreads / kReduceCols;                 // 8
constexpr int kReducePerThread = (kStage2MaxWGs + kReduceGroups - 1) / kReduceGroups;   // 32
constexpr int kReduceSmall = kStage2DownGroups / kReduceGroups;   // 8: for <= 64 partials

// UPT: partials per thread (kReducePerThread, or kReduceSmall when nwg <= 64,
// which adds the same terms in the same order).

template <int DT, int UPT>
__global__ __launch_bounds__(kReduceThreads) void reduce_kernel(const float *__restrict__ ypart, int nwg,
                                                                int nbt, int d, uint16_t *__restrict__ y) {
    __shared__ float red[kReduceGroups][kReduceCols];
    const int b = blockIdx.y, col = threadIdx.x % kReduceCols, g = threadIdx.x / kReduceCols;
    const int c = blockIdx.x * kReduceCols + col;
    const int cc = min(c, d - 1);
    float v[UPT];
#pragma unroll
    for (int u = 0; u < UPT; ++u) {   // clamped loads, masked below
        const int w = min(g + u * kReduceGroups, nwg - 1);
        v[u] = ypart[((size_t)w * nbt + b) * d + cc];
    }
    float acc = 0.0f;
#pragma unroll
    for (int u = 0; u < UPT; ++u)
        if (g + u * kReduceGroups < nwg) acc += v[u];
    red[g][col] = acc;
    __syncthreads();
    if (g == 0 && c < d) {
        float s = 0.0f;
#pragma unroll
        for (int q = 0; q < kReduceGroups; ++q) s += red[q][col];
        y[(size_t)b * d + c] = float_to_half<DT>(s);
    }
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
    __syncthreads();   // every thread has read its x, y before out (which may alias x) is written
    for (int i = threadIdx.x; i < d; i += 1024) {
        const float r = half_to_float<DT>(xb[i]) + half_to_float<DT>(yb[i]);
        out[(size_t)b * d + i] = float_to_half<DT>(r * inv);
    }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

// sparse: the channel selection's histogram shares the front of the space.
size_t stage2_lds_bytes(int d, int nbt, int wq, bool sparse) {
    const size_t b = align_up(stage2_head_bytes(d, nbt, wq), 16) + (size_t)kMaxSlice * nbt * 4;
    return sparse && b < kSelHistF32Bytes ? kSelHistF32Bytes : b;
}

int stage2_rows(int d, int wq) {
    if (wq != 4) return kStage2MaxNB;
    int r = kStage2MaxNB;   // a power of two, so the launch's row template is r
    while (r > 1 && !x_in_lds(d, r)) r /= 2;
    return r;
}

template <typename K>
static hipError_t allow_lds(K kernel, size_t bytes) {
    // Dynamic LDS above 64 KiB must be allowed per kernel (gfx950 has 160 KiB).
    if (bytes <= 65536) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

template <int NB, int DT, int C, int WQ>
static hipError_t launch_stage2_t(const void *x, int nb, int d, int f, const Stage2Weights &wt,
                                  const float *scores, int k_ff, uint8_t *mask, float *scores_copy,
                                  float *ypart, int ystride, int nwg, Select sel_rule, int act,
                                  int32_t *klist, int klist_mode, hipStream_t st) {
    if (WQ == 4 && !x_in_lds(d, NB)) return hipErrorInvalidValue;
    const size_t lds = stage2_lds_bytes(d, NB, WQ, scores != nullptr);
    hipError_t e = allow_lds(stage2_kernel<NB, DT, C, WQ>, lds);
    if (e != hipSuccess) return e;
    stage2_kernel<NB, DT, C, WQ><<<nwg, kBlock, lds, st>>>(
        static_cast<const uint16_t *>(x), nb, d, f, wt, scores, k_ff, mask, scores_copy, ypart,
        ystride, sel_rule, act, klist, klist_mode);
    return hipGetLastError();
}

template <int NB, int DT, int WQ>
static hipError_t launch_stage2_c(const void *x, int nb, int d, int f, const Stage2Weights &wt,
                                  const float *scores, int k_ff, uint8_t *mask, float *scores_copy,
                                  float *ypart, int ystride, int nwg, Select sel_rule, int act,
                                  int32_t *klist, int klist_mode, hipStream_t st) {
    // C = score rows per thread of the channel top-k (the dense path has none).
#define S2C(C_) launch_stage2_t<NB, DT, C_, WQ>(x, nb, d, f, wt, scores, k_ff, mask, scores_copy, ypart, ystride, nwg, sel_rule, act, klist, klist_mode, st)
    // As few score rows per thread as d_ff needs (below 16 not for eight rows
    // of INT4 weights, whose registers are full).
    if constexpr (WQ == 16 || NB <= 4) {
        if (scores && f <= 4 * kBlock) return S2C(4);
        if (scores && f <= 8 * kBlock) return S2C(8);
        if (scores && f <= 12 * kBlock) return S2C(12);
    }
    if (!scores || f <= 16 * kBlock) return S2C(16);
    if (f <= 28 * kBlock) return S2C(28);
    if (f <= 32 * kBlock) return S2C(32);
    return S2C(64);
#undef S2C
}

hipError_t launch_stage2(int dtype, const void *x, int nb, int d, int f, const Stage2Weights &wt,
                         const float *scores, int k_ff, uint8_t *mask, float *scores_copy,
                         float *ypart, int ystride, int nwg, Select sel_rule, int act,
                         int32_t *klist, int klist_mode, hipStream_t st) {
    if (nb < 1 || nb > stage2_rows(d, wt.wq)) return hipErrorInvalidValue;
    if (klist_mode != kListNone && (!scores || !klist)) return hipErrorInvalidValue;
#define S2(NB_, DT_, WQ_) return launch_stage2_c<NB_, DT_, WQ_>(x, nb, d, f, wt, scores, k_ff, mask, scores_copy, ypart, ystride, nwg, sel_rule, act, klist, klist_mode, st)
#define S2NB(DT_, WQ_)                   \
    switch (stage2_nb_t(nb)) {           \
        case 1: S2(1, DT_, WQ_);         \
        case 2: S2(2, DT_, WQ_);         \
        case 4: S2(4, DT_, WQ_);         \
        default: S2(8, DT_, WQ_);        \
    }
    if (wt.wq == 4) {
        if (dtype == kBF16) { S2NB(kBF16, 4) }
        S2NB(kF16, 4)
    }
    if (dtype == kBF16) { S2NB(kBF16, 16) }
    S2NB(kF16, 16)
#undef S2NB
#undef S2
}

template <int DT, int C>
static hipError_t launch_stage2m_t(const void *x, int nb, int d, int f, const Stage2Weights &wt,
                                   const float *scores, int k_ff, uint8_t *mask,
                                   float *scores_copy, float *sbuf, int nwg, Select sel_rule,
                                   int act, int32_t *klist, int klist_mode, hipStream_t st) {
    const size_t lds = stage2_mfma_lds_bytes();
    hipError_t e = allow_lds(stage2_mfma_kernel<DT, C>, lds);
    if (e != hipSuccess) return e;
    stage2_mfma_kernel<DT, C><<<nwg, kBlock, lds, st>>>(
        static_cast<const uint16_t *>(x), nb, d, f, wt, scores, k_ff, mask, scores_copy, sbuf,
        sel_rule, act, klist, klist_mode);
    return hipGetLastError();
}

template <int DT>
static hipError_t launch_stage2m_c(const void *x, int nb, int d, int f, const Stage2Weights &wt,
                                   const float *scores, int k_ff, uint8_t *mask,
                                   float *scores_copy, float *sbuf, int nwg, Select sel_rule,
                                   int act, int32_t *klist, int klist_mode, hipStream_t st) {
#define S2M(C_) launch_stage2m_t<DT, C_>(x, nb, d, f, wt, scores, k_ff, mask, scores_copy, sbuf, nwg, sel_rule, act, klist, klist_mode, st)
    if (scores && f <= 4 * kBlock) return S2M(4);
    if (scores && f <= 8 * kBlock) return S2M(8);
    if (scores && f <= 12 * kBlock) return S2M(12);
    if (!scores || f <= 16 * kBlock) return S2M(16);
    if (f <= 28 * kBlock) return S2M(28);
    if (f <= 32 * kBlock) return S2M(32);
    return S2M(64);
#undef S2M
}

hipError_t launch_stage2_mfma(int dtype, const void *x, int nb, int d, int f,
                              const Stage2Weights &wt, const float *scores, int k_ff,
                              uint8_t *mask, float *scores_copy, float *sbuf, int nwg,
                              Select sel_rule, int act, int32_t *klist, int klist_mode,
                              hipStream_t st) {
    const int n_ch = scores && !sel_rule.tau_mode ? k_ff : f;   // the kept-list length
    if (nb < 1 || nb > kStage2MfmaRows || !stage2_mfma_ok(d, wt.wq) || nwg < 1 ||
        nwg > kStage2MaxWGs || (long long)n_ch > (long long)kMaxSlice * nwg || !sbuf)
        return hipErrorInvalidValue;
    // The down launch reads the kept list: a sparse call writes or reads it.
    if ((scores != nullptr) != (klist_mode != kListNone) || (scores && !klist))
        return hipErrorInvalidValue;
    if (dtype == kBF16)
        return launch_stage2m_c<kBF16>(x, nb, d, f, wt, scores, k_ff, mask, scores_copy, sbuf,
                                       nwg, sel_rule, act, klist, klist_mode, st);
    return launch_stage2m_c<kF16>(x, nb, d, f, wt, scores, k_ff, mask, scores_copy, sbuf, nwg,
                                  sel_rule, act, klist, klist_mode, st);
}

hipError_t launch_stage2_down(int dtype, int nb, int d, int f, const void *wd, const float *sbuf,
                              const int32_t *klist, int n_max, float *ypart, int ystride,
                              hipStream_t st) {
    if (nb < 1 || nb > kStage2MfmaRows || d % 4 != 0 || n_max < 0 || n_max > f || !sbuf ||
        (!klist && n_max != f))
        return hipErrorInvalidValue;
    const size_t lds = stage2_down_lds_bytes(n_max);
    const dim3 grid((d / 4 + kDownCols - 1) / kDownCols, kStage2DownGroups);
    const uint16_t *w = static_cast<const uint16_t *>(wd);
    if (dtype == kBF16) {
        hipError_t e = allow_lds(stage2_down_kernel<kBF16>, lds);
        if (e != hipSuccess) return e;
        stage2_down_kernel<kBF16><<<grid, kBlock, lds, st>>>(nb, d, f, w, sbuf, klist, ypart,
                                                                   ystride);
    } else {
        hipError_t e = allow_lds(stage2_down_kernel<kF16>, lds);
        if (e != hipSuccess) return e;
        stage2_down_kernel<kF16><<<grid, kBlock, lds, st>>>(nb, d, f, w, sbuf, klist, ypart,
                                                                  ystride);
    }
    return hipGetLastError();
}

hipError_t launch_reduce(int dtype, const float *ypart, int nwg, int nb, int d, void *y,
                         hipStream_t st) {
    dim3 grid((d + kReduceCols - 1) / kReduceCols, nb);
    const int nbt = ypart_rows(nb);
    if (nwg < 1 || nwg > kStage2MaxWGs) return hipErrorInvalidValue;
    uint16_t *yb = static_cast<uint16_t *>(y);
    if (nwg <= kReduceSmall * kReduceGroups) {
        if (dtype == kBF16)
            reduce_kernel<kBF16, kReduceSmall><<<grid, kReduceThreads, 0, st>>>(ypart, nwg, nbt, d, yb);
        else
            reduce_kernel<kF16, kReduceSmall><<<grid, kReduceThreads, 0, st>>>(ypart, nwg, nbt, d, yb);
    } else if (dtype == kBF16) {
        reduce_kernel<kBF16, kReducePerThread><<<grid, kReduceThreads, 0, st>>>(ypart, nwg, nbt, d, yb);
    } else {
        reduce_kernel<kF16, kReducePerThread><<<grid, kReduceThreads, 0, st>>>(ypart, nwg, nbt, d, yb);
    }
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
