// slim_launch.h - launchers shared between the libslim translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "slim_host.h"

// tm = A Q^T: A [M, Kd] fp16 activations (the row-scaled copy), Q [r, Kd] fp16 row-major; fp16
// result at ws + p.off_t in 32 x 16 tiles (adapter_gemm.hip).
int slim_launch_adapter_gemm(const uint16_t* A, int64_t M, int64_t Kd, const uint16_t* Q, int64_t r, const SlimPlan& p,
                             char* ws, hipStream_t s);
