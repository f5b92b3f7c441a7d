// kernel_tiled.h -- general translation kernel, fp32 arithmetic (any even
// head_dim, any layer mixing, identity or CSR alignment).  Serves fp32 plans
// and shapes the matrix-core kernel does not tile.
//
// One workgroup owns (target layer l, K|V, context b, a tile of target rows):
//   1. prologue: for every row of the tile, gather the source rows of its
//      alignment entries, undo the source RoPE at each source position, pool
//      with the entry weights (fp32) into LDS -- the pooled, de-rotated row z_t;
//   2. projection: each thread takes output pairs (i, i + Dt/2) of one target
//      head and forms u = W z_t + b by fp32 dot products over the LDS row;
//   3. epilogue: target RoPE on K at the target position, store.
#pragma once

#include "common.h"

namespace kvx {

template <typename T>
struct TiledArgs {
  const T* src[2];          // source K, V
  Strides ss;
  T* tgt[2];                // target K, V
  Strides ts;
  const T* w[2];            // [Lt][dout][din], nn.Linear order (plan copy)
  const float* bias[2];     // [Lt][dout] (zeros when the translator has none)
  const int32_t* layer_map; // [Lt][mix]
  int32_t mix, hs, ds, ht, dt, din, dout;
  const double* fs;         // [ds/2] source theta_i / 2pi (zeros: RoPE off)
  const double* ft;         // [dt/2] target
  const int32_t* row_ptr;   // CSR alignment (unused when identity != 0)
  const int32_t* col_idx;
  const float* weight;
  int32_t identity;
  int32_t rows;             // target rows per tile
  Paging pg;                // optional paged target layout
  BatchArgs ba;
};

template <typename T>
__global__ void __launch_bounds__(256) tiled_kernel(TiledArgs<T> a) {
  extern __shared__ float z[];  // [rows][din]
  const int tile = blockIdx.x;
  const int l = blockIdx.y;
  const int kv = blockIdx.z;
  const int b = find_context(a.ba, tile);
  const int t0 = (tile - a.ba.tile_start[b]) * a.rows;
  const int tt = a.ba.t_tgt[b];
  const int nrows = min(a.rows, tt - t0);
  if (nrows <= 0) return;
  const T* src = a.src[kv];
  const int hd = a.ds / 2;

  // 1. pooled, de-rotated source rows -> LDS
  const int n_items = nrows * a.mix * a.hs * hd;
  for (int it = threadIdx.x; it < n_items; it += blockDim.x) {
    int i = it % hd;
    int rest = it / hd;
    int h = rest % a.hs;
    rest /= a.hs;
    int j = rest % a.mix;
    int r = rest / a.mix;
    int t = t0 + r;
    int ls = a.layer_map[l * a.mix + j];
    const T* base = src + ls * a.ss.l + b * a.ss.b + h * a.ss.h + i;
    int e0 = 0, e1 = 1;
    if (!a.identity) {
      e0 = a.row_ptr[a.ba.row_base[b] + t];
      e1 = a.row_ptr[a.ba.row_base[b] + t + 1];
    }
    float z0 = 0.f, z1 = 0.f;
    for (int e = e0; e < e1; ++e) {
      int k = a.identity ? t : a.col_idx[e];
      float w = a.identity ? 1.f : a.weight[e];
      const T* p = base + k * a.ss.t;
      float x0 = load_f32(p), x1 = load_f32(p + hd);
      if (kv == 0) {  // undo the source rotation at source position k
        float c, s;
        rope_cs(a.fs[i], k, c, s);
        float y0 = x0 * c + x1 * s;
        float y1 = x1 * c - x0 * s;
        x0 = y0;
        x1 = y1;
      }
      z0 += w * x0;
      z1 += w * x1;
    }
    float* zr = z + r * a.din + (j * a.hs + h) * a.ds;
    zr[i] = z0;
    zr[i + hd] = z1;
  }
  __syncthreads();

  // 2-3. projection, bias, target rotation, store
  const int ht2 = a.dt / 2;
  const T* wl = a.w[kv] + static_cast<int64_t>(l) * a.dout * a.din;
  const float* bl = a.bias[kv] + static_cast<int64_t>(l) * a.dout;
  T* dst = a.tgt[kv] + l * a.ts.l;
  const int n_out = nrows * a.ht * ht2;
  for (int it = threadIdx.x; it < n_out; it += blockDim.x) {
    int i = it % ht2;
    int rest = it / ht2;
    int h = rest % a.ht;
    int r = rest / a.ht;
    int o0 = h * a.dt + i, o1 = o0 + ht2;
    const float* zr = z + r * a.din;
    const T* w0 = wl + static_cast<int64_t>(o0) * a.din;
    const T* w1 = wl + static_cast<int64_t>(o1) * a.din;
    float u0 = 0.f, u1 = 0.f;
    for (int k = 0; k < a.din; ++k) {
      u0 += zr[k] * load_f32(w0 + k);
      u1 += zr[k] * load_f32(w1 + k);
    }
    u0 += bl[o0];
    u1 += bl[o1];
    int t = t0 + r;
    if (kv == 0) {
      float c, s;
      rope_cs(a.ft[i], t, c, s);
      float y0 = u0 * c - u1 * s;
      float y1 = u1 * c + u0 * s;
      u0 = y0;
      u1 = y1;
    }
    const int32_t blk = a.pg.table ? a.pg.table[b * a.pg.max_blocks + t / a.pg.block_size] : 0;
    T* p = dst + h * a.ts.h + target_row(a.pg, a.ts, b, t, blk);
    p[i] = store_cvt<T>(u0);
    p[i + ht2] = store_cvt<T>(u1);
  }
}

}  // namespace kvx
