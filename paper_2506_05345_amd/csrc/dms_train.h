// Internal declarations of the training-time attention (continuous decisions).
#pragma once

#include <hip/hip_runtime.h>

#include "../../include/dms.h"

namespace dms {

constexpr int kTrainHeadDim = 128;   // head dimension of the training kernels

size_t train_workspace_bytes(const dms_train_config& c);
hipError_t launch_train_fwd(const dms_train_config& c, const void* q, const void* k, const void* v,
                            const float* alpha, float* out, float* lse, void* ws, hipStream_t st);
hipError_t launch_train_bwd(const dms_train_config& c, const void* q, const void* k, const void* v,
                            const float* alpha, const float* out, const float* lse,
                            const void* dout, float* dq, float* dk, float* dv, float* dalpha,
                            void* ws, hipStream_t st);
hipError_t launch_gumbel_fwd(int n, const float* x, const float* u, float tau, float* alpha,
                             hipStream_t st);
hipError_t launch_gumbel_bwd(int n, const float* alpha, const float* da, float tau, float* dx,
                             hipStream_t st);

}  // namespace dms
