// slim_launch.h - launchers shared between the libslim translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "slim_host.h"

// tm = A Q^T: A [M, Kd] activations, Q [r, Kd] fp16 row-major; fp16 result [M, r] at ws + p.off_t.
int slim_launch_adapter_gemm(const uint16_t* A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* Q, int64_t r,
                             const SlimPlan& p, char* ws, hipStream_t s);
