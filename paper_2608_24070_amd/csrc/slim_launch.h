// slim_launch.h - launchers shared between the libslim translation units.
#pragma once

#include <hip/hip_runtime.h>

#include "slim_host.h"

// T = A B (nt == false: B is [Kd, r]) or T = A B^T (nt == true: B is [r, Kd]); fp16 result at ws + p.off_t.
int slim_launch_adapter_gemm(bool nt, const uint16_t* A, int a_bf16, int64_t M, int64_t Kd, const uint16_t* B,
                             int64_t r, const SlimPlan& p, char* ws, hipStream_t s);
