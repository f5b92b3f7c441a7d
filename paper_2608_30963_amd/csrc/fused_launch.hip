// fused_launch.hip -- the fused kernel's variants for one operand precision
// (KVX_LAUNCH_PREC: 0 = BF16X2, 1 = BF16, 2 = F16) and their dispatch.
#include "fused_launch.h"

#ifndef KVX_LAUNCH_PREC
#error "define KVX_LAUNCH_PREC (0, 1 or 2)"
#endif

namespace kvx {
namespace {

template <int PREC, bool STREAM, bool PAGED, int ORDER>
void launch_pspi(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  if constexpr (ORDER == 2) {
    // the resident order serves span maps only
    fused_kernel<false, false, PREC, STREAM, PAGED, 2><<<dim3(grid), dim3(kThreads), 0, st>>>(a);
  } else {
    if (identity && ds128)
      fused_kernel<true, true, PREC, STREAM, PAGED, ORDER><<<dim3(grid), dim3(kThreads), 0, st>>>(a);
    else if (identity)
      fused_kernel<true, false, PREC, STREAM, PAGED, ORDER><<<dim3(grid), dim3(kThreads), 0, st>>>(a);
    else
      fused_kernel<false, false, PREC, STREAM, PAGED, ORDER><<<dim3(grid), dim3(kThreads), 0, st>>>(a);
  }
}

// tile order (contiguous ranges, interleaved, or resident) as a template
// argument; the host picks the resident order only for span maps with
// several N tiles, and runs it with streaming source loads
template <int PREC, bool STREAM, bool PAGED>
void launch_psp(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  if (a.interleave == 1) {
    launch_pspi<PREC, STREAM, PAGED, 1>(identity, ds128, grid, st, a);
    return;
  }
  if constexpr (STREAM) {
    if (a.interleave == 2) {
      launch_pspi<PREC, STREAM, PAGED, 2>(identity, ds128, grid, st, a);
      return;
    }
  }
  launch_pspi<PREC, STREAM, PAGED, 0>(identity, ds128, grid, st, a);
}

template <int PREC, bool STREAM>
void launch_ps(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  if (a.pg.table)
    launch_psp<PREC, STREAM, true>(identity, ds128, grid, st, a);
  else
    launch_psp<PREC, STREAM, false>(identity, ds128, grid, st, a);
}

// Streaming source loads when no tile re-reads a source row: a single N tile
// covers the output, or the resident order transforms a row tile once for
// all its N tiles; cached loads otherwise.
template <int PREC>
void launch_p(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  if (a.n_tiles == 1 || a.interleave == 2)
    launch_ps<PREC, true>(identity, ds128, grid, st, a);
  else
    launch_ps<PREC, false>(identity, ds128, grid, st, a);
}

}  // namespace

#if KVX_LAUNCH_PREC == 0
void launch_fused_bf16x2(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  launch_p<kBF16X2>(identity, ds128, grid, st, a);
}
#elif KVX_LAUNCH_PREC == 1
void launch_fused_bf16(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  launch_p<kBF16>(identity, ds128, grid, st, a);
}
#else
void launch_fused_f16(bool identity, bool ds128, int grid, hipStream_t st, const FusedArgs& a) {
  launch_p<kF16>(identity, ds128, grid, st, a);
}
#endif

}  // namespace kvx
