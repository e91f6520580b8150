// Block-wide exact top-k, used in the prologues of the Stage 1 and Stage 2
// kernels (App. A.6 per-token top-k rule, ties to the lower index).
//
// Items are owned strided: item r of thread t is index r * NT + t, so every
// key load is coalesced, and a wave's ballot over item r covers 64
// consecutive indices.  Keys are unsigned and order like the values they
// stand for: 15-bit magnitude patterns of 16-bit floats (input selection) or
// bit patterns of non-negative fp32 scores (channel selection).  Items past
// n hold key 0.
//
// The k-th largest key is found with histograms in LDS: one pass over all
// 2^15 values of a 16-bit magnitude (two 16-bit counters per word), or, for
// fp32 scores, three passes over 12 + 11 + 8 bits (11 + 11 + 9 up to 16 keys
// per thread), the later ones over the keys that match the digits found so
// far, ending as soon as the found bin is wholly in the top k.  Small blocks
// of 16-bit keys (at most 4096 items) take two passes of 12 + 3 bits instead,
// whose scans are cheaper than the items they add.  A pass is one round of
// LDS atomics and a block-wide scan of the bin counts from the top.  Ties at the k-th key are
// cut by index: of the keys equal to it, those up to the index of the needed
// one are in.  The selection then costs one or two compares per item: each
// wave keeps the ballots of its rows (TopKOrder), and one scan of their
// popcounts gives every selected item its ascending position.
//
// Per-item work is what these prologues cost: a 1024-thread block runs 16
// waves on 4 SIMDs, so every instruction per item is ~16 CU cycles per row.
#pragma once

#include "common.hpp"

namespace prox {

// Per (item row r, wave w) ballots of the selected items and their exclusive
// prefix counts in index order.
template <int C>
struct TopKOrder {
    uint64_t sel[C][kMaxBlockWaves];
    int off[C * kMaxBlockWaves];
};

// Scratch of the digit search (besides the histogram).
struct SelScratch {
    int wtot[kMaxBlockWaves];   // per-wave totals of the bin scan
    int pick[3];                // found digit, rank inside it, its count
};

// The 2^14-word histograms are padded by one word after every 16, so the 16
// words a thread scans start 17 words after its neighbour's: the scan's LDS
// reads are free of bank conflicts.  Word w sits at hist_pad(w).
__host__ __device__ constexpr uint32_t hist_pad(uint32_t w) { return w + (w >> 4); }
constexpr int kSelPadWords = 16384 + 1024;

// LDS words of the histograms: 2^15 packed 16-bit counters (input keys), or
// at most 2^12 + 2^11 + 2^8 counters (the three digits of a score key).
constexpr int kSelHistU16Words = kSelPadWords;
constexpr int kSelHistF32Words = 4096 + 2048 + 256;
constexpr size_t kSelHistU16Bytes = (size_t)kSelHistU16Words * 4;
constexpr size_t kSelHistF32Bytes = (size_t)kSelHistF32Words * 4;

// Wave index as a wave-uniform value (kept in an SGPR).
__device__ __forceinline__ int wave_id() {
    return __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
}

// v_writelane (lane `lane` of v replaced by the wave-uniform s) through its
// LLVM intrinsic, so the compiler also inserts the wait states it needs
// after the instruction that wrote s.
extern "C" __device__ int prox_llvm_writelane(int s, int lane, int v) __asm("llvm.amdgcn.writelane.i32");

__device__ __forceinline__ uint32_t write_lane(uint32_t v, uint32_t s, int lane) {
    return (uint32_t)prox_llvm_writelane((int)s, lane, (int)v);
}

// Every wave's row ballots to a [C][16] table (ord.sel, or another): lane r
// of two registers takes row r's ballot (lanes r < C), then one store per
// wave.
template <int C, typename B>
__device__ __forceinline__ void store_ballots(uint64_t *table, int wid, B &&ballot_of_row) {
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int r = 0; r < C; ++r) {
        const uint64_t b = ballot_of_row(r);
        lo = write_lane(lo, (uint32_t)b, r);
        hi = write_lane(hi, (uint32_t)(b >> 32), r);
    }
    const int lane = lane_id();
    if (lane < C) table[lane * kMaxBlockWaves + wid] = ((uint64_t)hi << 32) | lo;
}
template <int C, typename B>
__device__ __forceinline__ void store_ballots(TopKOrder<C> &ord, int wid, B &&ballot_of_row) {
    store_ballots<C>(&ord.sel[0][0], wid, ballot_of_row);
}

// Exclusive scan of the per-(row, wave) counts, taken as the popcounts of the
// ballots in ord.sel (written before the call), into ord.off.  One wave does
// it: lane l holds C / 4 consecutive entries.
template <int NT, int C>
__device__ __forceinline__ void topk_scan_ballots(TopKOrder<C> &ord) {
    static_assert(C % 4 == 0 && C * kMaxBlockWaves == kWave * (C / 4), "C / 4 entries per lane");
    constexpr int E = C / 4;
    __syncthreads();
    if (threadIdx.x < kWave) {
        const int lane = lane_id();
        const uint64_t *sel = &ord.sel[0][0];
        int v[E], run = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            v[e] = run;
            run += __popcll(sel[lane * E + e]);
        }
        const int base = wave_inclusive_scan(run) - run;
#pragma unroll
        for (int e = 0; e < E; ++e) ord.off[lane * E + e] = base + v[e];
    }
    __syncthreads();
}

// Ascending positions of the selected items (bit r of sel = item r): per
// (row, wave) ballots and their exclusive prefix counts in index order.
template <int NT, int C>
__device__ __forceinline__ void topk_order(uint64_t sel, TopKOrder<C> &ord) {
    store_ballots<C>(ord, wave_id(), [&](int r) { return __ballot((sel >> r) & 1); });
    topk_scan_ballots<NT, C>(ord);
}

// The bin holding the kk-th largest counted item (1 <= kk <= total count).
// The NBINS counters are in ascending digit order; PACKED holds two 16-bit
// counters per word, bin 2i in the low half of word i.  Thread t owns the BPT
// bins just below NBINS - t * BPT, so the threads in order walk the digits
// downwards and one block-wide scan of their sums finds the bin.  Returns, in
// every thread, the digit, kk's rank inside that bin and the bin's count.
template <int NBINS, bool PACKED>
__device__ __forceinline__ void find_digit(const uint32_t *h, int kk, SelScratch &ss,
                                           uint32_t &digit, int &kk_in, int &bucket) {
    constexpr int BPT = NBINS >= kBlock ? NBINS / kBlock : 1;   // bins per thread
    constexpr int PER = PACKED ? 2 : 1;                         // bins per word
    constexpr int WPT = BPT / PER;                              // words per thread
    static_assert(NBINS % kBlock == 0 || NBINS <= kBlock, "bins split evenly");
    static_assert(BPT % PER == 0 && (WPT == 1 || WPT == 2 || WPT % 4 == 0), "whole words");
    const int tid = threadIdx.x, lane = lane_id(), wid = wave_id();
    const bool own = tid * BPT < NBINS;
    const int lo_bin = NBINS - (tid + 1) * BPT;   // lowest bin of this thread
    uint32_t w[WPT];
    if (own) {
        const uint32_t *src = h + lo_bin / PER;
        if constexpr (WPT == 16) {
            // A 2^14-word histogram, padded (hist_pad): 17 words per thread.
            const uint32_t *p = h + hist_pad((uint32_t)(lo_bin / PER));
#pragma unroll
            for (int j = 0; j < WPT; ++j) w[j] = p[j];
        } else if constexpr (WPT % 4 == 0) {
#pragma unroll
            for (int j = 0; j < WPT / 4; ++j) {
                const uint4 v = reinterpret_cast<const uint4 *>(src)[j];
                w[4 * j] = v.x; w[4 * j + 1] = v.y; w[4 * j + 2] = v.z; w[4 * j + 3] = v.w;
            }
        } else if constexpr (WPT == 2) {
            const uint2 v = *reinterpret_cast<const uint2 *>(src);
            w[0] = v.x; w[1] = v.y;
        } else {
            w[0] = src[0];
        }
    } else {
#pragma unroll
        for (int j = 0; j < WPT; ++j) w[j] = 0;
    }
    // Packed words are summed whole (each half stays below 2^16), then the
    // two halves added.
    int local;
    if constexpr (PACKED) {
        uint32_t t = 0;
#pragma unroll
        for (int j = 0; j < WPT; ++j) t += w[j];
        local = (int)((t & 0xFFFFu) + (t >> 16));
    } else {
        local = 0;
#pragma unroll
        for (int j = 0; j < WPT; ++j) local += (int)w[j];
    }
    const int incl = wave_inclusive_scan(local);
    if (lane == kWave - 1) ss.wtot[wid] = incl;
    __syncthreads();
    // Counts of the waves before this one: lanes 0..15 scan the 16 totals.
    int base = 0;
    if (wid > 0) {
        int t = lane < kMaxBlockWaves ? ss.wtot[lane] : 0;
        t += __builtin_amdgcn_update_dpp(0, t, 0x111, 0xF, 0xF, false);   // row_shr:1
        t += __builtin_amdgcn_update_dpp(0, t, 0x112, 0xF, 0xF, false);   // row_shr:2
        t += __builtin_amdgcn_update_dpp(0, t, 0x114, 0xF, 0xF, false);   // row_shr:4
        t += __builtin_amdgcn_update_dpp(0, t, 0x118, 0xF, 0xF, false);   // row_shr:8
        base = __builtin_amdgcn_readlane(t, wid - 1);
    }
    const int excl = base + incl - local;
    if (own && excl < kk && kk <= excl + local) {   // exactly one thread
        // Words from the top down: the first whose running count reaches kk.
        int cum = excl, jw = 0;
        uint32_t ww = 0;
        bool found = false;
#pragma unroll
        for (int j = WPT - 1; j >= 0; --j) {
            const int c = PACKED ? (int)((w[j] & 0xFFFFu) + (w[j] >> 16)) : (int)w[j];
            if (!found && cum + c >= kk) {
                found = true;
                jw = j;
                ww = w[j];
            } else if (!found) {
                cum += c;
            }
        }
        int bin, cnt;
        if constexpr (PACKED) {
            const int hi = (int)(ww >> 16);
            if (cum + hi >= kk) {
                bin = lo_bin + 2 * jw + 1;
                cnt = hi;
            } else {
                cum += hi;
                bin = lo_bin + 2 * jw;
                cnt = (int)(ww & 0xFFFFu);
            }
        } else {
            bin = lo_bin + jw;
            cnt = (int)ww;
        }
        ss.pick[0] = bin;
        ss.pick[1] = kk - cum;
        ss.pick[2] = cnt;
    }
    __syncthreads();
    digit = (uint32_t)ss.pick[0];
    kk_in = ss.pick[1];
    bucket = ss.pick[2];
}

// Order tables of the rule "key >= v" (no tie to cut): the ballot of every
// (row, wave) and, after one scan of their popcounts, the exclusive prefix
// counts of the selected items in index order.  One compare per item; items
// past n hold key 0, so only v = 0 needs an index limit, a per-lane compare
// inside the ballot (VALU) rather than a wave mask built on the scalar unit,
// which the 16 waves of a CU share.
template <int NT, int C>
__device__ __forceinline__ void topk_table(const uint32_t (&key)[C], int n, uint32_t v,
                                           TopKOrder<C> &ord) {
    const int wid = wave_id();
    const int tid = threadIdx.x;
    store_ballots<C>(ord, wid, [&](int r) {
        return v == 0 ? __ballot(r * NT + tid < n) : __ballot(key[r] >= v);
    });
    topk_scan_ballots<NT, C>(ord);
}

// Order tables of the top-k rule with a tie cut: every key above v is in, and
// of the keys equal to v the first `need` in index order (0 < need < their
// count).  The ballots of "above" and "equal" are scanned together (one
// wave: exclusive prefixes G and Q per entry), the entry offsets are
// G + min(need, Q), and each wave then ballots its final rows with the
// equal-key rank Q + (equal lanes below) < need.  scratch: LDS words dead
// after the last digit search, at least 3 C kMaxBlockWaves.
template <int NT, int C>
__device__ __forceinline__ void topk_table_cut(const uint32_t (&key)[C], int n, uint32_t v,
                                               int need, uint32_t *scratch, TopKOrder<C> &ord) {
    static_assert(C % 4 == 0 && C * kMaxBlockWaves == kWave * (C / 4), "C / 4 entries per lane");
    constexpr int E = C / 4;
    const int wid = wave_id(), tid = threadIdx.x;
    uint64_t *eqs = reinterpret_cast<uint64_t *>(scratch);    // [C][16] equal-key ballots
    int *qpre = reinterpret_cast<int *>(eqs + C * kMaxBlockWaves);   // [C * 16] their prefixes
    // Items past n hold key 0: they are never above v, and equal to it only
    // when v = 0.
    auto equal = [&](int r) { return key[r] == v && (v != 0 || r * NT + tid < n); };
    store_ballots<C>(ord, wid, [&](int r) { return __ballot(key[r] > v); });
    store_ballots<C>(eqs, wid, [&](int r) { return __ballot(equal(r)); });
    __syncthreads();
    if (tid < kWave) {
        const int lane = lane_id();
        const uint64_t *gt = &ord.sel[0][0];
        int g[E], q[E], rg = 0, rq = 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            g[e] = rg;
            q[e] = rq;
            rg += __popcll(gt[lane * E + e]);
            rq += __popcll(eqs[lane * E + e]);
        }
        const int bg = wave_inclusive_scan(rg) - rg, bq = wave_inclusive_scan(rq) - rq;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            ord.off[lane * E + e] = bg + g[e] + min(need, bq + q[e]);
            qpre[lane * E + e] = bq + q[e];
        }
    }
    __syncthreads();
    store_ballots<C>(ord, wid, [&](int r) {
        const bool eq = equal(r);
        const int rank = qpre[r * kMaxBlockWaves + wid] + (int)lanes_below(__ballot(eq));
        return __ballot(key[r] > v || (eq && rank < need));
    });
    __syncthreads();
}

// One narrow digit pass: counts bits [shift, shift + log2 NBINS) of the keys
// whose higher bits equal `prefix` (bits from `shift + log2 NBINS` up), into
// h (NBINS words, zero), then finds the bin holding the kk-th largest.
template <int NT, int C, int NBINS>
__device__ __forceinline__ void narrow_pass(const uint32_t (&key)[C], int n, int shift,
                                            uint32_t prefix, uint32_t *h, SelScratch &ss,
                                            int &kk, int &bucket, uint32_t &digit) {
    const int tid = threadIdx.x;
    constexpr uint32_t kMaskBins = NBINS - 1;
    const int top = shift + __builtin_ctz(NBINS);   // bits at or above top: the prefix
#pragma unroll
    for (int r = 0; r < C; ++r) {
        // Keys past n are 0: masked whenever the prefix admits 0.
        const bool match = (top >= 32 || (key[r] >> top) == prefix) && (prefix != 0 || r * NT + tid < n);
        if (match) atomicAdd(&h[(key[r] >> shift) & kMaskBins], 1u);
    }
    __syncthreads();
    find_digit<NBINS, false>(h, kk, ss, digit, kk, bucket);
}

// Top k (1 <= k <= n) of 15-bit keys (magnitude patterns of 16-bit floats):
// one histogram pass over all 2^15 values finds the k-th largest key v; ties
// at v are cut by index.  hist: kSelHistU16Words words of LDS.  Fills ord.
template <int NT, int C>
__device__ __forceinline__ void topk_select_u15(const uint32_t (&key)[C], int n, int k,
                                                uint32_t *hist, SelScratch &ss,
                                                TopKOrder<C> &ord) {
    static_assert(C * NT < 65536, "a 16-bit counter holds every key");
    const int tid = threadIdx.x;
    if constexpr (C * NT <= 4096) {
        // Few keys: bits 14..3, then 2..0, over 4096- and 8-bin histograms.
        // The first pass takes mantissa bits as well as the exponent: keys
        // crowd into a few exponents, and same-word LDS atomics serialise.
        uint32_t *h1 = hist, *h2 = hist + 4096;
        for (int i = tid; i < (4096 + 8) / 4; i += NT)
            reinterpret_cast<uint4 *>(hist)[i] = make_uint4(0, 0, 0, 0);
        __syncthreads();
        int kk = k, bucket;
        uint32_t d1, d2;
        narrow_pass<NT, C, 4096>(key, n, 3, 0, h1, ss, kk, bucket, d1);
        uint32_t v = d1 << 3;
        if (kk < bucket) {
            narrow_pass<NT, C, 8>(key, n, 0, d1, h2, ss, kk, bucket, d2);
            v = (d1 << 3) | d2;
            if (kk < bucket) {
                topk_table_cut<NT, C>(key, n, v, kk, hist, ord);
                return;
            }
        }
        topk_table<NT, C>(key, n, v, ord);
        return;
    }
    for (int i = tid; i < kSelHistU16Words / 4; i += NT)
        reinterpret_cast<uint4 *>(hist)[i] = make_uint4(0, 0, 0, 0);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < C; ++r) atomicAdd(&hist[hist_pad(key[r] >> 1)], 1u << ((key[r] & 1u) << 4));
    if (tid == 0 && n < C * NT) atomicSub(&hist[0], (uint32_t)(C * NT - n));   // the items past n
    __syncthreads();
    uint32_t v;
    int need, bucket;
    find_digit<32768, true>(hist, k, ss, v, need, bucket);
    if (need < bucket) topk_table_cut<NT, C>(key, n, v, need, hist, ord);
    else topk_table<NT, C>(key, n, v, ord);
}

// Top k (1 <= k <= n) of non-negative fp32 keys (bit 31 clear) in three
// radix passes over small histograms: bits 30..20, 19..9 and 8..0 (2048, 2048
// and 512 bins) up to 16 keys per thread, else bits 30..19, 18..8 and 7..0
// (4096, 2048 and 256 bins); the later passes count only the keys matching
// the digits found so far, and stop once the found bin is wholly in the top
// k.  Ties at the k-th key are cut by index.  hist: kSelHistF32Words words of
// LDS.  Fills ord.
template <int NT, int C>
__device__ __forceinline__ void topk_select_f32(const uint32_t (&key)[C], int n, int k,
                                                uint32_t *hist, SelScratch &ss,
                                                TopKOrder<C> &ord) {
    const int tid = threadIdx.x;
    constexpr int L1 = C * NT <= 16384 ? 11 : 12, L2 = 11, L3 = 31 - L1 - L2;
    constexpr int S1 = 31 - L1, S2 = S1 - L2;
    static_assert((1 << L1) + (1 << L2) + (1 << L3) <= kSelHistF32Words, "histograms fit");
    uint32_t *g1 = hist, *g2 = hist + (1 << L1), *g3 = g2 + (1 << L2);
    for (int i = tid; i < ((1 << L1) + (1 << L2) + (1 << L3)) / 4; i += NT)
        reinterpret_cast<uint4 *>(hist)[i] = make_uint4(0, 0, 0, 0);
    __syncthreads();
    int kk = k, bucket;
    uint32_t d1, d2, d3;
    narrow_pass<NT, C, (1 << L1)>(key, n, S1, 0, g1, ss, kk, bucket, d1);
    uint32_t v = d1 << S1;
    if (kk < bucket) {
        narrow_pass<NT, C, (1 << L2)>(key, n, S2, d1, g2, ss, kk, bucket, d2);
        v = (d1 << S1) | (d2 << S2);
        if (kk < bucket) {
            narrow_pass<NT, C, (1 << L3)>(key, n, 0, (d1 << L2) | d2, g3, ss, kk, bucket, d3);
            v |= d3;
            if (kk < bucket) {
                topk_table_cut<NT, C>(key, n, v, kk, hist, ord);
                return;
            }
        }
    }
    topk_table<NT, C>(key, n, v, ord);
}

// Ascending position (among the selected) of this thread's selected item r.
template <int C>
__device__ __forceinline__ int topk_pos(const TopKOrder<C> &ord, int r) {
    const int wid = threadIdx.x / kWave;
    return ord.off[r * kMaxBlockWaves + wid] + (int)lanes_below(ord.sel[r][wid]);
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
