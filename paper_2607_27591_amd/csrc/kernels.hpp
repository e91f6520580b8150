// Host-side launchers of the libprox kernels (one per .hip file).  Each
// enqueues on `s` and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "layout.hpp"

namespace prox {

hipError_t launch_pack(int dtype, int qbits, const void *wg, const void *wu, int d, int f,
                       int group, void *blob, hipStream_t stream);
hipError_t launch_unpack(int qbits, const void *blob, int d, int f, int group, int8_t *cg,
                         uint16_t *sg, int8_t *cu, uint16_t *su, hipStream_t stream);

hipError_t launch_select_inputs(const void *x, int B, int d, int k, Ctrl *ctrl, uint8_t *in_mask,
                                hipStream_t stream);
hipError_t launch_select_channels(const float *scores, int f, int k, Ctrl *ctrl, uint8_t *mask,
                                  int *ff_idx, float *scores_copy, hipStream_t stream);

hipError_t launch_proxy(int dtype, int qbits, const void *x, int nb, const void *x_all, int B_all,
                        int d, int f, int group, const void *blob, Ctrl *ctrl, float *part,
                        float *scores, int accumulate, hipStream_t stream);

hipError_t launch_gateup(int dtype, const void *x, int nb, int d, const void *wg, const void *wu,
                         const int *ff_idx, int n_ch, float *s_out, int s_stride,
                         Ctrl *ctrl_reset, hipStream_t stream);
hipError_t launch_down(int dtype, const void *wd, int d, const int *ff_idx, int n_ch,
                       const float *s, int s_stride, int nb, float *ypart, Ctrl *ctrl, void *y,
                       hipStream_t stream);
hipError_t launch_add_rmsnorm(int dtype, const void *x, const void *y, int batch, int d, float eps,
                              void *out, hipStream_t stream);

// Geometry helpers shared with the host API (sizes, LDS limits).
void down_geometry(int d, int n_ch, int &tiles, int &splits, int &ch_per_split);
size_t down_lds_bytes(int nbt, int ch_per_split);
int gateup_grid(int n_ch);

}  // namespace prox
