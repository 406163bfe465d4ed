// slim_launch.h - launchers shared between the libslim translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "slim_host.h"

// tm = A Q^T: A [M, Kd] activations (fp16, or bf16 when a_bf16, in which case the kernel also
// writes their fp16 copy to a16), Q [r, Kd] fp16 row-major; fp16 result at ws + p.off_t in 32 x 16
// tiles (adapter_gemm.hip).
int slim_launch_adapter_gemm(const uint16_t* A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* Q, int64_t r,
                             const SlimPlan& p, char* ws, uint16_t* a16, hipStream_t s);
