// Host-side launchers of the libprox kernels.  Each enqueues on `stream` and
// returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout.hpp"

namespace prox {

// Column tile of Stage-1 workgroup b of n.  Workgroups are dealt to the 8 XCDs
// in turn (XCD b % 8), each with its own L2.  When a row segment of a tile is
// under 128 bytes (PAIRED: INT4 codes of a 64-column tile), one 128-byte line
// holds the same kept row of tiles 2p and 2p + 1, so the pair goes to
// workgroups b and b + 8 of one XCD and its L2 fetches the line once.  The
// last n % 16 workgroups keep tile b.  A bijection of [0, n).
template <bool PAIRED>
__device__ __forceinline__ int stage1_tile(int b, int n) {
    if constexpr (!PAIRED) {
        return b;
    } else {
        if (b >= (n & ~15)) return b;
        const int x = b & 7, q = b >> 3;
        return 2 * ((q >> 1) * 8 + x) + (q & 1);
    }
}

hipError_t launch_pack(int dtype, int qbits, const void *wg, const void *wu, int d, int f,
                       int group, void *blob, hipStream_t stream);
hipError_t launch_unpack(int qbits, const void *blob, int d, int f, int group, int8_t *cg,
                         uint16_t *sg, int8_t *cu, uint16_t *su, hipStream_t stream);

// Stage 1 for batch rows [row0, row0 + nb) of x_all (nb <= proxy_max_nb(d));
// the input selection ranks all B_all rows (top k_in, or the threshold rule
// of sel, for which k_in is the list capacity).  accumulate != 0 keeps
// max(previous, new) scores.
int proxy_max_nb(int d);
hipError_t launch_proxy(int dtype, int qbits, const void *x_all, int B_all, int row0, int nb,
                        int d, int f, int group, int k_in, const void *blob,
                        uint8_t *in_mask, float *scores, int accumulate, Select sel, int act,
                        hipStream_t stream);

// Stage 1 on the matrix cores for INT4 proxies: batch rows [row0, row0 + nb)
// with nb <= proxy_mfma_rows(d, group, k_in) (16, 8, or 0 when the kept-row
// list does not fit in LDS); otherwise as launch_proxy.
int proxy_mfma_rows(int d, int group, int k_in);
// klist, list_mode: as Stage 2's kept list (KeptList), for the input rows:
// the first launch of a call with several also writes the kept rows in
// ascending order to klist[0..n) and n to klist[d]; the later ones rebuild
// their list from it instead of selecting again.
hipError_t launch_proxy_mfma(int dtype, const void *x_all, int B_all, int row0, int nb, int d,
                             int f, int group, int k_in, const void *blob, uint8_t *in_mask,
                             float *scores, int accumulate, Select sel, int act, int32_t *klist,
                             int list_mode, hipStream_t stream);
// Batch rows from which Stage 1 uses the matrix cores: 3 up to d_model 4096,
// 5 above (where its 2-byte code loads keep too few bytes in flight).
inline int proxy_mfma_min_rows(int d) { return d <= 4096 ? 3 : 5; }

// The three matrices of Stage 2: channel-major 16-bit rows (wq == 16), or
// INT4 codes with fp16 scales per (channel, group along d), laid out as
// W4Layout describes (wq == 4).
struct Stage2Weights {
    const void *wg, *wu, *wd;
    const uint16_t *sg, *su, *sd;   // INT4 scales, else unused
    int wq, group;
};
// Batch rows one Stage 2 launch takes: kStage2MaxNB, fewer with INT4 weights
// when d is wide (their launch keeps all nb rows of x in LDS).
int stage2_rows(int d, int wq);
// act (both stages): the gate activation, 0 SiLU or 1 GELU.
// Stage 2 for batch rows x[0..nb) (nb <= stage2_rows(d, w.wq)).  scores ==
// NULL runs the dense FFN over all f channels; otherwise the top k_ff scores,
// or the threshold rule of sel, pick the channels.  Partial y rows go to
// ypart[(w * ystride + b) * d + c] for workgroup w < nwg.
// A batch split over several Stage 2 launches selects once: the first launch
// (kListWrite) also writes the kept channels in ascending order to klist[0..n)
// and their count n to klist[f]; the later ones (kListRead) take their slice
// from it.  kListNone: a single launch, klist unused.
enum KeptList { kListNone = 0, kListWrite = 1, kListRead = 2 };
hipError_t launch_stage2(int dtype, const void *x, int nb, int d, int f, const Stage2Weights &w,
                         const float *scores, int k_ff, uint8_t *mask, float *scores_copy,
                         float *ypart, int ystride, int nwg, Select sel, int act,
                         int32_t *klist, int klist_mode, hipStream_t stream);
// Stage 2 for up to kStage2MfmaRows batch rows (16-bit weights, d >= 4096:
// stage2_mfma_ok) in two launches.  launch_stage2_mfma selects like
// launch_stage2 (same kept-list modes; the sparse path must write or read
// klist, since the down launch takes the kept channels from it), runs gate/up
// on the matrix cores and writes s of kept-list position p and batch row b to
// sbuf[p * kStage2MfmaRows + b].  launch_stage2_down then splits the kept
// list (klist, or every channel when klist is NULL) into kStage2DownGroups
// groups and writes the partial y of group g to ypart[(g * ystride + b) * d +
// c]; n_max bounds the kept count (k_ff, or f).
bool stage2_mfma_ok(int d, int wq);
hipError_t launch_stage2_mfma(int dtype, const void *x, int nb, int d, int f,
                              const Stage2Weights &w, const float *scores, int k_ff,
                              uint8_t *mask, float *scores_copy, float *sbuf, int nwg, Select sel,
                              int act, int32_t *klist, int klist_mode, hipStream_t stream);
hipError_t launch_stage2_down(int dtype, int nb, int d, int f, const void *wd, const float *sbuf,
                              const int32_t *klist, int n_max, float *ypart, int ystride,
                              hipStream_t stream);
// INT4 base weights: quantise W_gate, W_up, W_down (channel-major [f][d]) into
// a W4Layout blob, and the inverse view of matrix m (0 gate, 1 up, 2 down).
hipError_t launch_pack_w4(int dtype, const void *wg, const void *wu, const void *wd, int d, int f,
                          int group, void *blob, hipStream_t stream);
hipError_t launch_unpack_w4(const void *blob, int d, int f, int group, int m, int8_t *codes,
                            uint16_t *scales, hipStream_t stream);
hipError_t launch_reduce(int dtype, const float *ypart, int nwg, int nb, int d, void *y,
                         hipStream_t stream);
hipError_t launch_add_rmsnorm(int dtype, const void *x, const void *y, int batch, int d, float eps,
                              void *out, hipStream_t stream);

}  // namespace prox
