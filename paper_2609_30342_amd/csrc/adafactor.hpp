// adafactor.hpp -- host-side launchers of the Adafactor-m kernels
// (adafactor.hip).  The step runs over the same tile tables as R-iKFAD.
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "layout.hpp"

namespace rk {

// Optional timing events as for the R-iKFAD launchers (launch.hpp).

// Pass 1: row / column partial sums of G^2 + eps1 (matrices); the
// unfactored second moment and the tile sums of U^2 (vectors); tile sums
// of X^2 when x2 is set.  tilepart: 2 floats per tile (U^2, X^2).
hipError_t launch_adafm_stats(const TensorDesc *tensors, const void *const *grads,
                              const Tile *tiles, const TileGroup *groups, int ngroups, float *ws,
                              float *tilepart, const AdaCoeffs &k, bool x2, hipStream_t stream,
                              hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Pass 2: tile sums of U^2 for the matrix tiles (after the factor update).
hipError_t launch_adafm_rms(const TensorDesc *tensors, const void *const *grads,
                            const Tile *tiles, const TileGroup *groups, int ngroups,
                            const float *ws, float *tilepart, hipStream_t stream,
                            hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Per tensor: fold the tile sums, then scale = step size / clipping divisor.
hipError_t launch_adafm_scale(const TensorRange *ranges, int64_t ntensors, const float *tilepart,
                              float *scales, const AdaCoeffs &k, hipStream_t stream,
                              hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Pass 3: M <- beta1 M + (1 - beta1) scale U, X <- X - M.
hipError_t launch_adafm_update(const TensorDesc *tensors, const void *const *grads,
                               const Tile *tiles, const TileGroup *groups, int ngroups,
                               const float *ws, const float *scales, const AdaCoeffs &k,
                               hipStream_t stream, hipEvent_t start = nullptr,
                               hipEvent_t stop = nullptr);

}  // namespace rk
