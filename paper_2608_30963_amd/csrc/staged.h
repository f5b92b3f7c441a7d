// staged.h -- the translation operator (Section 4) as three separate
// launches instead of one fused kernel:
//   stage_pool     source RoPE removal on K and pooling over each target
//                  row's alignment entries, in fp32, written as bf16 planes
//                  hi (+ lo = the rounding residual) of the pooled inputs Z,
//                  rows x din (the fused kernel's K-slot order) stored in
//                  matrix-core A-fragment order;
//   stage_project  U = Z W^T per (target layer, K|V) on the matrix cores,
//                  fp32 accumulation, against the plan's packed weights;
//   stage_store    bias, target RoPE on K, bf16 rounding, store into the
//                  target cache (contiguous or paged).
// Each stage reads and writes HBM once, so its time measures what the memory
// system delivers for that part of the operator; the fused kernel does the
// same work without the intermediate round trips.
#pragma once

#include "common.h"

namespace kvx {

constexpr int kStageRows = 128;  // rows per row tile

struct StagedArgs {
  const bf16_t* src[2];
  Strides ss;
  bf16_t* tgt[2];
  Strides ts;
  Paging pg;
  const bf16x8* wp[2];  // packed fragments [Lt][dout/32][din/16][64 lanes][8]
  const float* bias[2];  // [Lt][dout]
  const int32_t* layer_map;
  const double* fs;  // source theta_i / 2pi (zeros without RoPE)
  const double* ft;  // target theta_i / 2pi
  const int32_t* row_ptr;  // nullptr: identity alignment
  const int32_t* col_idx;
  const float* weight;
  bf16_t* z;  // [nl][2 (K|V)][2 (hi|lo)][rows_p / 32][din / 16][64 lanes][8]
  float* u;   // [nl][2 (K|V)][rows_p / 32][dout / 32][16 registers][64 lanes]
  int32_t mix, hs, ds, ht, dt, din, dout;
  int32_t l0, nl;         // target layers of this launch: l0 .. l0 + nl - 1
  int32_t tiles, rows_p;  // row tiles of the launch's contexts, rows_p = tiles * 128
  int32_t planes[2];      // per K|V: 2 (hi and lo planes) or 1 (hi only)
  BatchArgs ba;
};

void launch_stage_pool(const StagedArgs& a, hipStream_t st);
void launch_stage_project(const StagedArgs& a, hipStream_t st);
void launch_stage_store(const StagedArgs& a, hipStream_t st);

}  // namespace kvx
