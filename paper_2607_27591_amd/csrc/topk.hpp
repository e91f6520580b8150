// Block-wide exact top-k, used in the prologues of the Stage 1 and Stage 2
// kernels (App. A.6 per-token top-k rule, ties to the lower index).
//
// Thread t owns the contiguous items [t*c, t*c + c) of the n keys
// (c = ceil(n / NT) <= C), so one block-wide prefix scan turns per-thread
// counts into ascending global positions.  Keys are unsigned 32-bit; a key
// accessor K provides them:
//   K::hi(r)  the key of item r with its low 16 bits cleared (cheap, held in
//             registers),
//   K::full(r) the complete key (may read memory).
// The full key is requested only for items whose high half equals the
// threshold's, so callers can keep just 16 bits per key in registers.
//
// The k-th largest key is found by an MSB-first radix search with 8-bit
// digits, starting at the byte that holds the most significant bit of the
// largest key.  Score and |x| keys are dominated by their exponent, so most
// lanes of a wave fall in a handful of digits: the LDS histogram is
// replicated kHistCopies times (lane l counts into copy l % kHistCopies, the
// copies of one digit in adjacent banks), turning 64-way same-address atomics
// into 4-way ones.
#pragma once

#include "common.hpp"

namespace prox {

constexpr int kHistCopies = 16;

struct TopKScratch {
    uint32_t hist[256 * kHistCopies];   // [digit][copy]
    uint32_t pick[2];
    uint32_t wmax[kMaxBlockWaves];
    int scan[kMaxBlockWaves + 1];
};

template <int NT>
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, TopKScratch &sh) {
    constexpr int NW = NT / kWave;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, o, kWave));
    if (lane_id() == 0) sh.wmax[threadIdx.x / kWave] = v;
    __syncthreads();
    uint32_t m = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) m = max(m, sh.wmax[w]);
    __syncthreads();
    return m;
}

// Key accessor over full 32-bit keys held in registers.
template <int C>
struct RegKeys {
    const uint32_t (&k)[C];
    __device__ uint32_t hi(int r) const { return k[r] & 0xFFFF0000u; }
    __device__ uint32_t full(int r) const { return k[r]; }
};

// v = the k-th largest of the n keys (1 <= k <= n); need = how many of the
// keys equal to v belong to the top k (every key > v does).
template <int NT, int C, typename K>
__device__ void topk_threshold(const K &keys, int c, int n, int k, TopKScratch &sh,
                               uint32_t &v_out, int &need_out) {
    const int tid = threadIdx.x, lane = lane_id();
    uint32_t kmax = 0;
#pragma unroll
    for (int r = 0; r < C; ++r)
        if (r < c && tid * c + r < n) kmax = max(kmax, keys.hi(r));
    kmax = block_max_u32<NT>(kmax, sh);
    // With all high halves zero the search runs on the low half (full keys).
    const int top_shift = kmax ? ((31 - __clz(kmax)) / 8) * 8 : 8;
    uint32_t prefix = 0, pmask = 0;
    int kk = k;
    const int copy = lane % kHistCopies;
#pragma unroll 1
    for (int shift = top_shift; shift >= 0; shift -= 8) {
        for (int b = tid; b < 256 * kHistCopies / 4; b += NT)
            reinterpret_cast<uint4 *>(sh.hist)[b] = make_uint4(0, 0, 0, 0);
        __syncthreads();
        const uint32_t hmask = pmask & 0xFFFF0000u, hpref = prefix & 0xFFFF0000u;
#pragma unroll
        for (int r = 0; r < C; ++r) {
            if (r >= c || tid * c + r >= n) continue;
            const uint32_t kh = keys.hi(r);
            if ((kh & hmask) != hpref) continue;
            const uint32_t key = shift >= 16 ? kh : keys.full(r);
            if ((key & pmask) == prefix)
                atomicAdd(&sh.hist[((key >> shift) & 255u) * kHistCopies + copy], 1u);
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

// Compare item r with the threshold v: +1 if key > v, 0 if equal, -1 if less.
template <typename K>
__device__ __forceinline__ int topk_cmp(const K &keys, int r, uint32_t v) {
    const uint32_t kh = keys.hi(r), vh = v & 0xFFFF0000u;
    if (kh != vh) return kh > vh ? 1 : -1;
    const uint32_t kf = keys.full(r);
    return kf > v ? 1 : (kf == v ? 0 : -1);
}

// Given the threshold (v, need), returns the ascending global position of
// this thread's first selected key and sets `eq_rank0` to the number of keys
// equal to v in earlier threads.  Item r is selected iff key > v, or key == v
// and its rank among the keys equal to v is < need.
template <int NT, int C, typename K>
__device__ int topk_positions(const K &keys, int c, int n, uint32_t v, int need, TopKScratch &sh,
                              int &eq_rank0) {
    const int tid = threadIdx.x;
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int r = 0; r < C; ++r) {
        if (r < c && tid * c + r < n) {
            const int cmp = topk_cmp(keys, r, v);
            n_gt += cmp > 0;
            n_eq += cmp == 0;
        }
    }
    int total;
    eq_rank0 = block_exclusive_scan<NT>(n_eq, sh.scan, total);
    const int my_eq = max(0, min(need - eq_rank0, n_eq));
    return block_exclusive_scan<NT>(n_gt + my_eq, sh.scan, total);
}

}  // namespace prox
