// common.h -- device helpers shared by the kvx kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvx.h"

namespace kvx {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef uint16_t bf16_t;  // storage: bfloat16 bit pattern

// Status for a HIP call's result: KVX_OK on success, else KVX_ENOMEM or
// KVX_EHIP with the code recorded for kvx_last_hip_error() of the calling
// thread.  Host only; defined with the plan functions.
kvx_status hip_status(hipError_t e);

// Contexts handled by one launch; larger batches are split by the host.
constexpr int kMaxBatch = 64;

// Per-launch description of the contexts (passed by value as a kernel argument).
struct BatchArgs {
  int32_t n;                       // contexts in this launch
  int32_t tile_start[kMaxBatch + 1];  // prefix sum of row tiles per context
  int32_t t_tgt[kMaxBatch];        // T_t of each context
  int32_t row_base[kMaxBatch];     // first CSR row of each context
};

struct Strides {
  int64_t l, b, h, t;  // elements; head_dim is unit-stride
};

// Optional paged target layout (a block table in the manner of paged KV
// caches): target token t of context b is stored in physical block
// table[b * max_blocks + t / block_size] at slot t % block_size; the target
// strides' batch entry is then the block stride and their token entry the
// slot stride.  table == nullptr: the contiguous layout.
struct Paging {
  const int32_t* table;  // device, this launch's contexts
  int32_t block_size;
  int32_t max_blocks;
};

// Element offset of target row (context b, token t), layer and head excluded,
// given the row's physical block (ignored without paging).
__device__ __forceinline__ int64_t target_row(const Paging& pg, const Strides& ts, int b, int t,
                                              int32_t block) {
  return pg.table ? static_cast<int64_t>(block) * ts.b +
                        static_cast<int64_t>(t % pg.block_size) * ts.t
                  : static_cast<int64_t>(b) * ts.b + static_cast<int64_t>(t) * ts.t;
}

// Exact widening of a bfloat16 bit pattern.
__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// float -> bfloat16, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

template <typename T> __device__ __forceinline__ float load_f32(const T* p);
template <> __device__ __forceinline__ float load_f32<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float load_f32<bf16_t>(const bf16_t* p) {
  return bf16_to_f32(*p);
}

template <typename T> __device__ __forceinline__ T store_cvt(float f);
template <> __device__ __forceinline__ float store_cvt<float>(float f) { return f; }
template <> __device__ __forceinline__ bf16_t store_cvt<bf16_t>(float f) {
  return f32_to_bf16(f);
}

// cos and sin of the RoPE angle pos * theta, given f = theta / (2*pi) in fp64.
// The angle is formed and reduced to [-1/2, 1/2] revolutions in fp64, so its
// error does not grow with the position; the hardware sine/cosine (argument
// in revolutions) then evaluates the reduced angle (measured on gfx950 over
// [-1/2, 1/2]: max abs error 1.2e-7 against fp64).
__device__ __forceinline__ void rope_cs(double f, int32_t pos, float& c, float& s) {
  double r = static_cast<double>(pos) * f;
  r -= rint(r);
  float x = static_cast<float>(r);
  s = __builtin_amdgcn_sinf(x);
  c = __builtin_amdgcn_cosf(x);
}

// Workgroup id -> position in XCD-major order: workgroups are dealt
// round-robin to the 8 XCDs, so this makes each XCD own one contiguous range.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  const int q = total / 8, r = total % 8;
  const int x = id % 8, slot = id / 8;
  return x * q + min(x, r) + slot;
}

// Which context a linear row-tile index belongs to (batch is small).
__device__ __forceinline__ int find_context(const BatchArgs& ba, int tile) {
  int b = 0;
  while (b + 1 < ba.n && ba.tile_start[b + 1] <= tile) ++b;
  return b;
}

}  // namespace kvx
