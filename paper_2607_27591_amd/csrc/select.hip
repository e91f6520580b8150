// Exact top-k selections of the sparse decode step, one workgroup each:
//  - input channels ranked by a_i = max_b |x_{b,i}| (Sec. 4.1 input mask,
//    per-token top-k rule of App. A.6);
//  - intermediate channels ranked by the proxy score (Sec. 4.1 channel mask).
// Ties go to the lower index.  The k-th largest key is found by an MSB-first
// radix search over keys held in registers; the tie cut and the ordered
// outputs then come from one block-wide prefix scan over contiguous chunks.
#include "common.hpp"
#include "kernels.hpp"

namespace prox {

constexpr int kSelThreads = 1024;

// |x| as its 15-bit magnitude pattern: monotone in |x| for fp16 and bf16,
// and +0 / -0 compare equal.
__device__ __forceinline__ uint32_t input_key(const uint16_t *__restrict__ x, int B, int d, int i) {
    uint32_t k = 0;
    for (int b = 0; b < B; ++b) k = max(k, (uint32_t)(x[(size_t)b * d + i] & 0x7FFFu));
    return k;
}

__global__ __launch_bounds__(kSelThreads) void select_inputs_kernel(
    const uint16_t *__restrict__ x, int B, int d, int k, Ctrl *__restrict__ ctrl,
    uint8_t *__restrict__ in_mask) {
    __shared__ uint32_t hist[258];
    __shared__ int scan_sh[kSelThreads / kWave + 1];
    const int tid = threadIdx.x;
    // Arrival counters of the later kernels of this call start at zero.
    for (int i = tid; i < 512; i += kSelThreads) ctrl->proxy_count[i] = 0;
    for (int i = tid; i < 256; i += kSelThreads) ctrl->down_count[i] = 0;

    constexpr int ITEMS = kMaxDModel / kSelThreads;
    uint32_t keys[ITEMS];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
        const int i = tid + r * kSelThreads;
        keys[r] = i < d ? input_key(x, B, d, i) : 0u;
    }
    uint32_t v;
    int need;
    block_kth_largest<kSelThreads, ITEMS, 16>(keys, d, k, hist, v, need);

    const int chunk = (d + kSelThreads - 1) / kSelThreads;
    const int lo = min(d, tid * chunk), hi = min(d, lo + chunk);
    int n_eq = 0;
    for (int i = lo; i < hi; ++i) n_eq += input_key(x, B, d, i) == v;
    int total;
    int rank = block_exclusive_scan<kSelThreads>(n_eq, scan_sh, total);
    for (int i = lo; i < hi; ++i) {
        const uint32_t key = input_key(x, B, d, i);
        bool sel = key > v;
        if (key == v) {
            sel = rank < need;
            if (rank == need - 1) ctrl->in_cut = (uint32_t)i;
            ++rank;
        }
        if (in_mask) in_mask[i] = sel ? 1 : 0;
    }
    if (tid == 0) ctrl->in_v = v;
}

template <int ITEMS>
__global__ __launch_bounds__(kSelThreads) void select_channels_kernel(
    const float *__restrict__ scores, int f, int k, Ctrl *__restrict__ ctrl,
    uint8_t *__restrict__ mask, int *__restrict__ ff_idx, float *__restrict__ scores_copy) {
    __shared__ uint32_t hist[258];
    __shared__ int scan_sh[kSelThreads / kWave + 1];
    const int tid = threadIdx.x;
    // Scores are |s~| >= 0, so their IEEE bit patterns order like the values.
    uint32_t keys[ITEMS];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
        const int i = tid + r * kSelThreads;
        keys[r] = i < f ? __float_as_uint(scores[i]) : 0u;
        if (scores_copy && i < f) scores_copy[i] = scores[i];
    }
    uint32_t v;
    int need;
    block_kth_largest<kSelThreads, ITEMS, 32>(keys, f, k, hist, v, need);

    const int chunk = (f + kSelThreads - 1) / kSelThreads;
    const int lo = min(f, tid * chunk), hi = min(f, lo + chunk);
    int n_gt = 0, n_eq = 0;
    for (int i = lo; i < hi; ++i) {
        const uint32_t key = __float_as_uint(scores[i]);
        n_gt += key > v;
        n_eq += key == v;
    }
    int total;
    int rank = block_exclusive_scan<kSelThreads>(n_eq, scan_sh, total);
    const int my_eq = max(0, min(need - rank, n_eq));
    int pos = block_exclusive_scan<kSelThreads>(n_gt + my_eq, scan_sh, total);
    for (int i = lo; i < hi; ++i) {
        const uint32_t key = __float_as_uint(scores[i]);
        bool sel = key > v;
        if (key == v) {
            sel = rank < need;
            if (rank == need - 1) ctrl->ff_cut = (uint32_t)i;
            ++rank;
        }
        mask[i] = sel ? 1 : 0;
        if (sel) ff_idx[pos++] = i;
    }
    if (tid == 0) ctrl->ff_v = v;
}

hipError_t launch_select_inputs(const void *x, int B, int d, int k, Ctrl *ctrl, uint8_t *in_mask,
                                hipStream_t s) {
    select_inputs_kernel<<<1, kSelThreads, 0, s>>>(static_cast<const uint16_t *>(x), B, d, k, ctrl,
                                                   in_mask);
    return hipGetLastError();
}

hipError_t launch_select_channels(const float *scores, int f, int k, Ctrl *ctrl, uint8_t *mask,
                                  int *ff_idx, float *scores_copy, hipStream_t s) {
    if (f <= 16 * kSelThreads)
        select_channels_kernel<16><<<1, kSelThreads, 0, s>>>(scores, f, k, ctrl, mask, ff_idx, scores_copy);
    else if (f <= 32 * kSelThreads)
        select_channels_kernel<32><<<1, kSelThreads, 0, s>>>(scores, f, k, ctrl, mask, ff_idx, scores_copy);
    else
        select_channels_kernel<64><<<1, kSelThreads, 0, s>>>(scores, f, k, ctrl, mask, ff_idx, scores_copy);
    return hipGetLastError();
}

}  // namespace prox
