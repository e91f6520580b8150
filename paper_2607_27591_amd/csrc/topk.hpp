// Block-wide exact top-k, used in the prologues of the Stage 1 and Stage 2
// kernels (App. A.6 per-token top-k rule, ties to the lower index).
//
// Items are owned strided: item r of thread t is index r * NT + t, so every
// key load is coalesced.  Keys are unsigned 32-bit and order like the values
// they stand for (magnitude patterns, non-negative IEEE floats).
//
// Fast path.  Every key is shifted left by a fixed amount so that its top 16
// significant bits (for non-negative floats: exponent and 8 mantissa bits)
// form its "window", kept in registers, two per VGPR.  Two MSB-first radix
// passes with 8-bit digits find the window value w* holding the k-th largest
// key.  When all items with window w* are needed the selection is
// {window >= w*}; otherwise, if at most one wave's worth of items share w*,
// one wave ranks them by (full key descending, index ascending).  Any other
// case (many equal windows) falls back to the general search below, which
// resolves the full key and ties by index over ballots of the whole block.
//
// Each pass: atomics into an LDS histogram replicated kHistCopies times
// (lane l counts into copy l % kHistCopies; score-like keys crowd a few
// digits, and the copies turn 64-way same-address atomics into 4-way ones),
// one barrier, all threads fold the copies (clearing them for the next pass),
// one barrier, and every wave scans the 256 digit counts itself, so no
// broadcast barrier is needed.
#pragma once

#include "common.hpp"

namespace prox {

constexpr int kHistCopies = 16;

struct alignas(16) TopKScratch {
    uint32_t hist[256 * kHistCopies];   // [digit][copy]; later selection words
    uint32_t cnt[256];                  // folded digit counts
    uint32_t pick[2];
    uint32_t wmax[kMaxBlockWaves];
    int scan[kMaxBlockWaves + 1];
    uint32_t cand_key[kWave];           // final-bucket candidates (fast path)
    int cand_idx[kWave];
    int cand_n;
};

// Per (item row r, wave w) ballots of the selected items and their exclusive
// prefix counts in index order.
template <int C>
struct TopKOrder {
    uint64_t sel[C][kMaxBlockWaves];
    int off[C * kMaxBlockWaves];
};

template <int NT>
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, TopKScratch &sh) {
    constexpr int NW = NT / kWave;
    v = wave_max_u32(v);
    if (lane_id() == 0) sh.wmax[threadIdx.x / kWave] = v;
    __syncthreads();
    uint32_t m = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) m = max(m, sh.wmax[w]);
    __syncthreads();
    return m;
}

// ---- general search (fallback) ----
// Keys through an accessor K:
//   K::hi(r)        the key of item r with its low 16 bits cleared, for a
//                   compile-time r (held in registers),
//   K::kHasLow      whether keys have low bits at all,
//   K::full_dyn(r)  the complete key for a run-time r (reads memory).
// Full keys are only read for items whose high half ties with the threshold
// prefix, visited by a bit loop.
//
// v = the k-th largest of the n keys (1 <= k <= n); need = how many of the
// keys equal to v belong to the top k (every key > v does).
template <int NT, int C, typename K>
__device__ __forceinline__ void topk_threshold(const K &keys, int n, int k, TopKScratch &sh, uint32_t &v_out,
                               int &need_out) {
    const int tid = threadIdx.x, lane = lane_id();
    uint32_t kmax = 0;
#pragma unroll
    for (int r = 0; r < C; ++r) {
            if (r * NT + tid < n) kmax = max(kmax, keys.hi(r));
    }
    kmax = block_max_u32<NT>(kmax, sh);
    // With every high half zero only the low half (if any) is searched.
    const int top_shift = kmax ? ((31 - __clz(kmax)) / 8) * 8 : (K::kHasLow ? 8 : 16);
    uint32_t prefix = 0, pmask = 0;
    int kk = k;
    const int copy = lane % kHistCopies;
    uint64_t cand = 0;   // items whose high half matches the prefix (low-half passes)
    const int last_shift = K::kHasLow ? 0 : 16;
#pragma unroll 1
    for (int shift = top_shift; shift >= last_shift; shift -= 8) {
        for (int b = tid; b < 256 * kHistCopies / 4; b += NT)
            reinterpret_cast<uint4 *>(sh.hist)[b] = make_uint4(0, 0, 0, 0);
        __syncthreads();
        if (shift >= 16) {
#pragma unroll
            for (int r = 0; r < C; ++r) {
                if (r * NT + tid >= n) continue;
                const uint32_t kh = keys.hi(r);
                if ((kh & pmask) == prefix)
                    atomicAdd(&sh.hist[((kh >> shift) & 255u) * kHistCopies + copy], 1u);
            }
        } else {
            if (shift == 8) {   // the high half is settled: collect its ties once
#pragma unroll
                for (int r = 0; r < C; ++r) {
                        if (r * NT + tid < n && keys.hi(r) == (prefix & 0xFFFF0000u)) cand |= 1ull << r;
                }
            }
            for (uint64_t m = cand; m; m &= m - 1) {
                const uint32_t key = keys.full_dyn(__builtin_ctzll(m));
                if ((key & pmask) == prefix)
                    atomicAdd(&sh.hist[((key >> shift) & 255u) * kHistCopies + copy], 1u);
            }
        }
        __syncthreads();
        if (tid < kWave) {
            // Lane l owns digits 255-4l ... 252-4l, i.e. descending key order.
            const int base = 255 - 4 * tid;
            int cnt[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint4 *h = reinterpret_cast<const uint4 *>(&sh.hist[(base - q) * kHistCopies]);
                int s = 0;
#pragma unroll
                for (int z = 0; z < kHistCopies / 4; ++z) {
                    const uint4 v4 = h[z];
                    s += (int)(v4.x + v4.y + v4.z + v4.w);
                }
                cnt[q] = s;
            }
            const int local = cnt[0] + cnt[1] + cnt[2] + cnt[3];
            const int incl = wave_inclusive_scan(local);
            const int excl = incl - local;
            if (excl < kk && kk <= incl) {
                int cum = excl, q = 0;
                for (q = 0; q < 3; ++q) {
                    if (cum + cnt[q] >= kk) break;
                    cum += cnt[q];
                }
                sh.pick[0] = (uint32_t)(base - q);
                sh.pick[1] = (uint32_t)cum;
            }
        }
        __syncthreads();
        const uint32_t digit = sh.pick[0];
        kk -= (int)sh.pick[1];
        prefix |= digit << shift;
        pmask |= 255u << shift;
        __syncthreads();
    }
    v_out = prefix;
    need_out = kk;
}

// Exclusive scan, in (r, w) order, of the C * 16 per-wave counts in off[]
// (written before the call by lane 0 of each wave).  One wave does it: lane l
// holds C / 4 consecutive entries.
template <int NT, int C>
__device__ __forceinline__ void topk_scan_table(int *off, TopKScratch &) {
    static_assert(C % 4 == 0 && C * kMaxBlockWaves == kWave * (C / 4), "C / 4 entries per lane");
    constexpr int E = C / 4;
    __syncthreads();
    if (threadIdx.x < kWave) {
        const int lane = lane_id();
        int v[E], run = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            v[e] = run;
            run += off[lane * E + e];
        }
        const int base = wave_inclusive_scan(run) - run;
#pragma unroll
        for (int e = 0; e < E; ++e) off[lane * E + e] = base + v[e];
    }
    __syncthreads();
}

// Selection bits of the top k given v and need from topk_threshold (bit r =
// item r); ord.off serves as scratch for ranking the keys equal to v.
template <int NT, int C, typename K>
__device__ __forceinline__ uint64_t topk_select_general(const K &keys, int n, uint32_t v, int need,
                                                        TopKScratch &sh, TopKOrder<C> &ord) {
    static_assert(C <= 64, "selection bits fit in 64");
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();
    uint64_t gt = 0, eq = 0;
    const uint32_t vh = v & 0xFFFF0000u;
#pragma unroll
    for (int r = 0; r < C; ++r) {
        if (r * NT + tid >= n) continue;
        const uint32_t kh = keys.hi(r);
        gt |= (uint64_t)(kh > vh) << r;
        eq |= (uint64_t)(kh == vh) << r;
    }
    if (K::kHasLow) {   // settle high-half ties on the full key
        for (uint64_t m = eq; m; m &= m - 1) {
            const int r = __builtin_ctzll(m);
            const uint32_t kf = keys.full_dyn(r);
            if (kf > v) gt |= 1ull << r;
            if (kf != v) eq &= ~(1ull << r);
        }
    }
    // Rank the keys equal to v in index order; the first `need` are kept.
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const uint64_t m = __ballot((eq >> r) & 1);
        if (lane == 0) ord.off[r * kMaxBlockWaves + wid] = __popcll(m);
    }
    topk_scan_table<NT, C>(ord.off, sh);
    uint64_t sel = gt;
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const uint64_t m = __ballot((eq >> r) & 1);
        if ((eq >> r) & 1) {
            const int rank = ord.off[r * kMaxBlockWaves + wid] + (int)lanes_below(m);
            if (rank < need) sel |= 1ull << r;
        }
    }
    __syncthreads();   // ord.off is rewritten by topk_order
    return sel;
}

// Ascending positions of the selected items: per (row, wave) ballots and their
// exclusive prefix counts in index order.
template <int NT, int C>
__device__ __forceinline__ void topk_order(uint64_t sel, int n, TopKScratch &sh, TopKOrder<C> &ord) {
    static_assert(C <= kWave, "one row per lane");
    const int wid = threadIdx.x / kWave, lane = lane_id();
    uint64_t mine = 0;   // lane r keeps row r's ballot (rows past n stay empty)
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const uint64_t m = __ballot((sel >> r) & 1);
        mine = lane == r ? m : mine;
    }
    if (lane < C) {
        ord.sel[lane][wid] = mine;
        ord.off[lane * kMaxBlockWaves + wid] = __popcll(mine);
    }
    topk_scan_table<NT, C>(ord.off, sh);
}

// ---- fast path ----
// One radix pass over the items for which item(r, digit) is true: returns the
// digit holding the kk-th largest (counting from the top), kk's rank inside
// that digit, and the digit's item count.  sh.hist must be zero on entry and
// is zero again on return.
template <int NT, int C, typename Item>
__device__ __forceinline__ void topk_pass(const Item &item, int n, TopKScratch &sh, int &kk,
                                          uint32_t &digit, int &bucket) {
    static_assert(NT == 256 * kHistCopies / 4, "one uint4 of copies per thread");
    const int tid = threadIdx.x, lane = lane_id();
    const int copy = lane % kHistCopies;
#pragma unroll
    for (int r = 0; r < C; ++r) {
        uint32_t dg;
        if (item(r, dg)) atomicAdd(&sh.hist[dg * kHistCopies + copy], 1u);
    }
    __syncthreads();
    {
        const int dgt = tid / 4;
        uint4 *h = reinterpret_cast<uint4 *>(&sh.hist[dgt * kHistCopies]) + (tid % 4);
        const uint4 c4 = *h;
        *h = make_uint4(0, 0, 0, 0);
        uint32_t t = c4.x + c4.y + c4.z + c4.w;
        t = quad_sum_u32(t);
        if ((tid % 4) == 0) sh.cnt[dgt] = t;
    }
    __syncthreads();
    // Lane l holds digits 255-4l ... 252-4l (descending key order).
    const uint4 c4 = *reinterpret_cast<const uint4 *>(&sh.cnt[252 - 4 * lane]);
    const int c0 = (int)c4.w, c1 = (int)c4.z, c2 = (int)c4.y, c3 = (int)c4.x;
    const int local = c0 + c1 + c2 + c3;
    const int incl = wave_inclusive_scan(local);
    const int excl = incl - local;
    const uint64_t hit = __ballot(excl < kk && kk <= incl);
    const int src = __builtin_ctzll(hit);   // exactly one lane: 1 <= kk <= total
    int q, cum = excl, cq;
    if (kk <= cum + c0) { q = 0; cq = c0; }
    else if (kk <= cum + c0 + c1) { q = 1; cum += c0; cq = c1; }
    else if (kk <= cum + c0 + c1 + c2) { q = 2; cum += c0 + c1; cq = c2; }
    else { q = 3; cum += c0 + c1 + c2; cq = c3; }
    digit = (uint32_t)__shfl(255 - 4 * lane - q, src, kWave);
    kk -= __shfl(cum, src, kWave);
    bucket = __shfl(cq, src, kWave);
}

// Window keys (top 16 bits of the shifted keys) for the general search.
template <int NT, int C2, bool HL, typename Reload>
struct WinKeys {
    static constexpr bool kHasLow = HL;
    const uint32_t (&h2)[C2];
    const Reload &reload;
    int shift;
    __device__ uint32_t hi(int r) const {
        const uint32_t w = h2[r >> 1];
        return (r & 1) ? (w & 0xFFFF0000u) : (w << 16);
    }
    __device__ uint32_t full_dyn(int r) const { return reload(r * NT + (int)threadIdx.x) << shift; }
};

// Top k of n keys (1 <= k <= n).  key[r] is item r's key (any value when its
// index is >= n); reload(i) returns key i again (only called when kHasLow:
// keys with bits below their 16-bit window).  Returns the selection bits and
// fills ord with the ascending positions of the selected items.
template <int NT, int C, bool kHasLow, typename Reload>
__device__ __forceinline__ uint64_t topk_block(const uint32_t (&key)[C], int n, int k, TopKScratch &sh,
                                               TopKOrder<C> &ord, const Reload &reload) {
    static_assert(C % 2 == 0 && C <= 64, "paired windows, 64 selection bits");
    const int tid = threadIdx.x, wid = tid / kWave, lane = lane_id();
    // Fixed windows: non-negative IEEE floats (kHasLow) have bit 31 clear, so
    // key << 1 puts the exponent and the top 8 mantissa bits in the high
    // half; keys of at most 16 bits are the window themselves.
    constexpr int shift = kHasLow ? 1 : 16;
    for (int b = tid; b < 256 * kHistCopies / 4; b += NT)
        reinterpret_cast<uint4 *>(sh.hist)[b] = make_uint4(0, 0, 0, 0);
    __syncthreads();
    uint32_t h2[C / 2];
    // Low key halves, two per word, kept for the tie step where registers
    // allow (up to 32 rows); otherwise they are reloaded.
    constexpr bool kLowRegs = kHasLow && C <= 32;
    uint32_t l2[kLowRegs ? C / 2 : 1];
#pragma unroll
    for (int q = 0; q < C / 2; ++q) {   // rows past n hold junk and are never read
        h2[q] = ((key[2 * q] << shift) >> 16) | ((key[2 * q + 1] << shift) & 0xFFFF0000u);
        if constexpr (kLowRegs) l2[q] = (key[2 * q] & 0xFFFFu) | (key[2 * q + 1] << 16);
    }
    auto win = [&](int r) -> uint32_t { return (r & 1) ? (h2[r >> 1] >> 16) : (h2[r >> 1] & 0xFFFFu); };
    auto valid = [&](int r) { return r * NT + tid < n; };

    int kk = k, bucket;
    uint32_t da, db;
    topk_pass<NT, C>([&](int r, uint32_t &dg) { dg = win(r) >> 8; return valid(r); }, n, sh, kk, da, bucket);
    uint64_t sel = 0;
    if (kk == bucket) {   // every item with this top digit is in
#pragma unroll
        for (int r = 0; r < C; ++r) {
            sel |= (uint64_t)(valid(r) && (win(r) >> 8) >= da) << r;
        }
    } else {
        if (tid == 0) sh.cand_n = 0;   // not touched again before the next barrier
        topk_pass<NT, C>([&](int r, uint32_t &dg) { dg = win(r) & 255u; return valid(r) && (win(r) >> 8) == da; },
                         n, sh, kk, db, bucket);
        const uint32_t w_star = (da << 8) | db;
#pragma unroll
        for (int r = 0; r < C; ++r) {
            sel |= (uint64_t)(valid(r) && win(r) > w_star) << r;
        }
        if (kk == bucket) {
#pragma unroll
            for (int r = 0; r < C; ++r) {
                sel |= (uint64_t)(valid(r) && win(r) == w_star) << r;
            }
        } else if (bucket <= kWave) {
            // Gather the bucket (slot order is arbitrary; ranking is explicit).
            // The histogram is idle now: its first NT 64-bit words become
            // per-thread selection words for the bucket items.
            uint64_t *selw = reinterpret_cast<uint64_t *>(sh.hist);
            static_assert(sizeof(sh.hist) >= NT * sizeof(uint64_t), "selection words fit");
            selw[tid] = 0;
#pragma unroll
            for (int r = 0; r < C; ++r) {
                if (valid(r) && win(r) == w_star) {
                    const int i = r * NT + tid;
                    const int slot = atomicAdd(&sh.cand_n, 1);
                    uint32_t ck = w_star << 16;
                    if constexpr (kLowRegs) {
                        const uint32_t lo = (r & 1) ? (l2[r >> 1] >> 16) : (l2[r >> 1] & 0xFFFFu);
                        ck |= (lo << shift) & 0xFFFFu;   // the shifted key's low half
                    } else if constexpr (kHasLow) {
                        ck = reload(i) << shift;
                    }
                    sh.cand_key[slot] = ck;
                    sh.cand_idx[slot] = i;
                }
            }
            __syncthreads();
            if (wid == 0) {
                // Lane l holds candidate l; the others are read with readlane.
                const bool act = lane < bucket;
                const uint32_t mk = act ? sh.cand_key[lane] : 0u;
                const int mi = act ? sh.cand_idx[lane] : 0;
                int rank = 0;
                for (int j = 0; j < bucket; ++j) {
                    const uint32_t kj = (uint32_t)__builtin_amdgcn_readlane((int)mk, j);
                    const int ij = __builtin_amdgcn_readlane(mi, j);
                    rank += (kj > mk || (kj == mk && ij < mi)) ? 1 : 0;
                }
                if (act && rank < kk)
                    atomicOr(reinterpret_cast<unsigned long long *>(&selw[mi % NT]), 1ull << (mi / NT));
            }
            __syncthreads();
            sel |= selw[tid];
        } else {
            // Many items share the window: general search on the shifted keys.
            const WinKeys<NT, C / 2, kHasLow, Reload> wk{h2, reload, shift};
            uint32_t v;
            int need;
            topk_threshold<NT, C>(wk, n, k, sh, v, need);
            sel = topk_select_general<NT, C>(wk, n, v, need, sh, ord);
        }
    }
    topk_order<NT, C>(sel, n, sh, ord);
    return sel;
}

// Ascending position (among the selected) of this thread's selected item r.
template <int C>
__device__ __forceinline__ int topk_pos(const TopKOrder<C> &ord, int r) {
    const int wid = threadIdx.x / kWave;
    return ord.off[r * kMaxBlockWaves + wid] + (int)lanes_below(ord.sel[r][wid]);
}

// Index of the selected item at ascending position p (0 <= p < number
// selected), any thread: binary search of the scanned table, then the
// position's set bit in that (row, wave) ballot.
template <int NT, int C>
__device__ __forceinline__ int topk_item_at(const TopKOrder<C> &ord, int p) {
    constexpr int E = C * kMaxBlockWaves;
    int lo = 0, hi = E - 1;   // largest e with off[e] <= p holds p
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (ord.off[mid] <= p) lo = mid; else hi = mid - 1;
    }
    const int r = lo / kMaxBlockWaves, w = lo % kMaxBlockWaves;
    uint64_t m = ord.sel[r][w];
    int n = p - ord.off[lo];   // the n-th set bit (from 0) of m
    int base = 0;
#pragma unroll
    for (int half = 32; half >= 1; half >>= 1) {
        const uint64_t lowmask = (half == 64) ? ~0ull : ((1ull << half) - 1);
        const int cnt = __popcll(m & lowmask);
        if (n >= cnt) { n -= cnt; m >>= half; base += half; }
        else m &= lowmask;
    }
    return r * NT + w * kWave + base;
}

// Whether item i (0 <= i < C * NT) is selected, any thread.
template <int NT, int C>
__device__ __forceinline__ bool topk_is_selected(const TopKOrder<C> &ord, int i) {
    const int r = i / NT, t = i % NT;
    return (ord.sel[r][t / kWave] >> (t % kWave)) & 1;
}

// Number of selected items with index < i (0 <= i <= C * NT), any thread.
template <int NT, int C>
__device__ __forceinline__ int topk_selected_before(const TopKOrder<C> &ord, int i) {
    if (i >= C * NT) {
        const uint64_t m = ord.sel[C - 1][kMaxBlockWaves - 1];
        return ord.off[C * kMaxBlockWaves - 1] + __popcll(m);
    }
    const int r = i / NT, t = i % NT, w = t / kWave, l = t % kWave;
    const uint64_t below = l ? (ord.sel[r][w] & ((1ull << l) - 1)) : 0ull;
    return ord.off[r * kMaxBlockWaves + w] + __popcll(below);
}

}  // namespace prox
