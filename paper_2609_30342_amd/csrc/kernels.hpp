// kernels.hpp -- host-side launchers of the gfx950 kernels (kernels.hip).
#pragma once
#include <hip/hip_runtime_api.h>
#include <stdint.h>

#include "layout.hpp"

namespace rk {

// Each launcher takes optional timing events: `start` is attached to its
// first dispatch and `stop` to its last (see launch.hpp).

// Streaming pass over all tiles (matrix and vector) of a context: one
// launch per tile group.
// A vector tile whose updated friction is not finite sets *flag.
hipError_t launch_stream(const TensorDesc *tensors, const void *const *grads, const Tile *tiles,
                         const TileGroup *groups, int ngroups, float *ws, const Coeffs &k,
                         int pending, int *flag, hipStream_t stream,
                         hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Finalisation of R, C and the partial sums of R (init_only: sums only),
// in workgroups of 2^fin_log2 threads (the plan's choice).
hipError_t launch_finalize(const FinItem *items, int64_t nitems, int fin_log2, float *ws,
                           const Coeffs &k, int *flag, int init_only, hipStream_t stream,
                           hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Second half-kick + D over the matrix tiles of every tile group.
hipError_t launch_apply(const TensorDesc *tensors, const Tile *tiles, const TileGroup *groups,
                        int ngroups, const float *ws, const Coeffs &k, hipStream_t stream,
                        hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// Full-tensor element-wise iKFAD.
hipError_t launch_ikfad(const TensorDesc *tensors, const void *const *grads, const Tile *tiles,
                        int64_t ntiles, const Coeffs &k, int *flag, hipStream_t stream,
                        hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

hipError_t launch_probe_stream(const float *a, const float *b, const float *c, float *d,
                               float *e, int64_t nfloat, hipStream_t stream);
// Message for rikfad_last_error on the calling thread (api.cpp).
void set_last_error(const char *msg);

hipError_t launch_probe_mix(void *x, const void *g, float *p, int64_t nelem, int dtype,
                            int shape, hipStream_t stream);
hipError_t launch_probe_read(const void *a, int64_t nbytes, float *out, hipStream_t stream);
hipError_t launch_probe_write(void *dst, int64_t nbytes, uint32_t value, hipStream_t stream);
hipError_t launch_probe_copy(const void *s, void *d, int64_t nbytes, hipStream_t stream);

}  // namespace rk
