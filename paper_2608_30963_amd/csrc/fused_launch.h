// fused_launch.h -- launchers of the fused kernel, one per operand precision.
// Each is defined in its own translation unit (fused_launch.hip built with
// KVX_LAUNCH_PREC = 0, 1, 2), so the kernel's instantiations compile in
// parallel.
#pragma once

#include "kernel_mfma.h"

namespace kvx {

void launch_fused_bf16x2(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a);
void launch_fused_bf16(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a);
void launch_fused_f16(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a);

}  // namespace kvx
