// Kernel launchers (defined in the .hip files). Arguments are already validated.
#pragma once
#include <hip/hip_runtime.h>

#include "layer.h"

namespace aqmb {

hipError_t launch_retile(const Layer& L, const void* codes_plane_major, hipStream_t st);
hipError_t launch_dequant(const Layer& L, int k, void* W, aqmb_dtype w_dtype, hipStream_t st);
hipError_t launch_gemv(const Layer& L, int k, const void* x, aqmb_dtype x_dtype, int batch, void* y,
                       aqmb_dtype y_dtype, hipStream_t st);
size_t gemv_workspace_floats(const aqmb_desc& d, int G, int S);
hipError_t launch_gemm(const Layer& L, int k, const void* X, int n_tokens, void* Y, aqmb_dtype y_dtype,
                       hipStream_t st);

}  // namespace aqmb
