// staged.hip -- the three launches of the unfused translation (staged.h).
#include "staged.h"

namespace kvx {
namespace {

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 sbf16x2;

__device__ __forceinline__ void unpack_bf16x8(const uint4 r, float (&x)[8]) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Round 8 floats to bf16 (hardware round-to-nearest-even) and pack.
__device__ __forceinline__ uint4 round_bf16x8(const float (&z)[8]) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const sbf16x2 p = {static_cast<__bf16>(z[2 * i]), static_cast<__bf16>(z[2 * i + 1])};
    o[i] = __builtin_bit_cast(uint32_t, p);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// Write z as its bf16 rounding (hi plane) and, with two planes, the bf16
// rounding of the residual z - hi (lo plane).
__device__ __forceinline__ void store_planes(bf16_t* hi, bf16_t* lo, bool two, const float (&z)[8]) {
  const uint4 h = round_bf16x8(z);
  *reinterpret_cast<uint4*>(hi) = h;
  if (two) {
    float hv[8], r[8];
    unpack_bf16x8(h, hv);
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = z[i] - hv[i];
    *reinterpret_cast<uint4*>(lo) = round_bf16x8(r);
  }
}

// Stage 1.  grid: (row tiles, din / 128 chunks, layers x K|V); 256 threads.
// Chunk c holds the RoPE pairs 64c .. 64c+63 of the flattened (mixed layer,
// source head, frequency) list: first members in slots 0..63, second members
// in 64..127.  Thread: one 8-pair group g of the chunk for rows tid/8 + 32u.
__global__ void __launch_bounds__(256) stage_pool(StagedArgs a) {
  const int tile = blockIdx.x, c = blockIdx.y, sys = blockIdx.z;
  const int ll = sys / 2, kv = sys % 2, l = a.l0 + ll;
  const int b = find_context(a.ba, tile);
  const int tt = a.ba.t_tgt[b];
  const int t0 = (tile - a.ba.tile_start[b]) * kStageRows;
  const int g = threadIdx.x % 8;
  const int half = a.ds / 2;
  const int pair0 = 64 * c + 8 * g;  // 8 pairs of one head (half % 8 == 0)
  const int hp = pair0 / half, i0 = pair0 % half;
  const int j = hp / a.hs, h = hp % a.hs;
  const int ls = a.layer_map[l * a.mix + j];
  const bf16_t* base = a.src[kv] + ls * a.ss.l + b * a.ss.b + h * a.ss.h + i0;
  double f[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) f[q] = kv == 0 ? a.fs[i0 + q] : 0.0;
  const int64_t plane = static_cast<int64_t>(a.rows_p) * a.din;
  bf16_t* zb = a.z + static_cast<int64_t>(ll * 2 + kv) * 2 * plane;
  const bool two = a.planes[kv] == 2;
#pragma unroll 1
  for (int u = 0; u < 4; ++u) {
    const int i = threadIdx.x / 8 + 32 * u;
    const int t = t0 + i;
    float z1[8], z2[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) z1[q] = z2[q] = 0.f;
    if (t < tt) {
      int e0 = 0, e1 = 1;
      if (a.row_ptr) {
        const int rr = a.ba.row_base[b] + t;
        e0 = a.row_ptr[rr];
        e1 = a.row_ptr[rr + 1];
      }
      for (int e = e0; e < e1; ++e) {
        const int k = a.row_ptr ? a.col_idx[e] : t;
        const float w = a.row_ptr ? a.weight[e] : 1.f;
        const bf16_t* p = base + static_cast<int64_t>(k) * a.ss.t;
        float x1[8], x2[8];
        unpack_bf16x8(*reinterpret_cast<const uint4*>(p), x1);
        unpack_bf16x8(*reinterpret_cast<const uint4*>(p + half), x2);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          float y1 = x1[q], y2 = x2[q];
          if (kv == 0) {
            float cs, sn;
            rope_cs(f[q], k, cs, sn);  // rotate by -k positions
            y1 = x1[q] * cs + x2[q] * sn;
            y2 = x2[q] * cs - x1[q] * sn;
          }
          z1[q] = fmaf(w, y1, z1[q]);
          z2[q] = fmaf(w, y2, z2[q]);
        }
      }
    }
    const int64_t row = static_cast<int64_t>(tile * kStageRows + i) * a.din + c * 128;
    store_planes(zb + row + 8 * g, zb + plane + row + 8 * g, two, z1);
    store_planes(zb + row + 64 + 8 * g, zb + plane + row + 64 + 8 * g, two, z2);
  }
}

// Stage 2.  grid: (row tiles, 128-output tiles, layers x K|V); 4 waves, each
// 64 rows x 64 outputs (2 x 2 tiles of v_mfma_f32_32x32x16_bf16).  Operand
// fragments come straight from memory: Z rows (16 bytes per lane) and the
// plan's packed weight fragments (1 KiB each); the next k-step's fragments
// are loaded during the current one's MFMAs.
__global__ void __launch_bounds__(256) stage_project(StagedArgs a) {
  const int tile = blockIdx.x, nt = blockIdx.y, sys = blockIdx.z;
  const int ll = sys / 2, kv = sys % 2, l = a.l0 + ll;
  const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
  const int wi = w / 2, wj = w % 2;
  const int nb_n = a.dout / 32, ks_n = a.din / 16;
  const int nb0 = nt * 4 + wj * 2;  // first 32-output block of this wave
  const int nbv = min(2, nb_n - nb0);
  if (nbv <= 0) return;  // no barrier in this kernel
  const int64_t plane = static_cast<int64_t>(a.rows_p) * a.din;
  const bf16_t* zb = a.z + static_cast<int64_t>(ll * 2 + kv) * 2 * plane;
  const bf16x8* wl = a.wp[kv] + static_cast<int64_t>(l) * nb_n * ks_n * 64;
  const int r0 = tile * kStageRows + wi * 64;
  const bool two = a.planes[kv] == 2;
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jb = 0; jb < 2; ++jb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][jb][v] = 0.f;
  // A fragment: lane l holds Z[row 32i + l%32][slot 16ks + 8(l/32) .. +7]
  const bf16_t* zrow[2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
    zrow[i] = zb + static_cast<int64_t>(r0 + 32 * i + lane % 32) * a.din + 8 * (lane / 32);
  const bf16x8* wb[2];
#pragma unroll
  for (int jb = 0; jb < 2; ++jb)
    wb[jb] = wl + static_cast<int64_t>(min(nb0 + jb, nb_n - 1)) * ks_n * 64 + lane;
  struct Frag {
    bf16x8 A[2][2], B[2];
  };
  auto load = [&](Frag& f, int ks) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      f.A[i][0] = *reinterpret_cast<const bf16x8*>(zrow[i] + ks * 16);
      f.A[i][1] = two ? *reinterpret_cast<const bf16x8*>(zrow[i] + plane + ks * 16) : f.A[i][0];
    }
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) f.B[jb] = wb[jb][ks * 64];
  };
  auto mma = [&](const Frag& f) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int jb = 0; jb < 2; ++jb)
        if (jb < nbv) {
          acc[i][jb] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.A[i][0], f.B[jb], acc[i][jb], 0, 0, 0);
          if (two)
            acc[i][jb] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.A[i][1], f.B[jb], acc[i][jb], 0, 0, 0);
        }
  };
  Frag f0, f1;
  load(f0, 0);
  int ks = 0;
  for (; ks + 2 <= ks_n; ks += 2) {
    load(f1, ks + 1);
    mma(f0);
    if (ks + 2 < ks_n) load(f0, ks + 2);
    mma(f1);
  }
  if (ks < ks_n) mma(f0);
  // D register v of lane l: row 8(v/4) + 4(l/32) + v%4, column l%32
  float* ub = a.u + static_cast<int64_t>(ll * 2 + kv) * a.rows_p * a.dout;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jb = 0; jb < 2; ++jb)
      if (jb < nbv)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int row = r0 + 32 * i + 8 * (v / 4) + 4 * (lane / 32) + v % 4;
          ub[static_cast<int64_t>(row) * a.dout + (nb0 + jb) * 32 + lane % 32] = acc[i][jb][v];
        }
}

// Stage 3.  grid: (32-row slices, groups of 8 threads' pair groups, layers x
// K|V); thread: one row and one group of 8 RoPE pairs (i0 .. i0+7 and their
// partners + Dt/2) of one target head.
__global__ void __launch_bounds__(256) stage_store(StagedArgs a) {
  const int slice = blockIdx.x, sys = blockIdx.z;
  const int ll = sys / 2, kv = sys % 2, l = a.l0 + ll;
  const int gph = a.dt / 16;  // 8-pair groups per head
  const int q = blockIdx.y * 8 + threadIdx.x % 8;
  if (q >= a.ht * gph) return;
  const int tile = slice / 4;
  const int i = (slice % 4) * 32 + threadIdx.x / 8;
  const int b = find_context(a.ba, tile);
  const int t = (tile - a.ba.tile_start[b]) * kStageRows + i;
  if (t >= a.ba.t_tgt[b]) return;
  const int h = q / gph, i0 = (q % gph) * 8;
  const int half = a.dt / 2;
  const int o1 = h * a.dt + i0, o2 = o1 + half;
  const float* ur =
      a.u + (static_cast<int64_t>(ll * 2 + kv) * a.rows_p + tile * kStageRows + i) * a.dout;
  const float* bb = a.bias[kv] + static_cast<int64_t>(l) * a.dout;
  float u1[8], u2[8];
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    const float4 p1 = *reinterpret_cast<const float4*>(ur + o1 + 4 * v);
    const float4 p2 = *reinterpret_cast<const float4*>(ur + o2 + 4 * v);
    const float4 c1 = *reinterpret_cast<const float4*>(bb + o1 + 4 * v);
    const float4 c2 = *reinterpret_cast<const float4*>(bb + o2 + 4 * v);
    u1[4 * v + 0] = p1.x + c1.x; u1[4 * v + 1] = p1.y + c1.y;
    u1[4 * v + 2] = p1.z + c1.z; u1[4 * v + 3] = p1.w + c1.w;
    u2[4 * v + 0] = p2.x + c2.x; u2[4 * v + 1] = p2.y + c2.y;
    u2[4 * v + 2] = p2.z + c2.z; u2[4 * v + 3] = p2.w + c2.w;
  }
  if (kv == 0) {
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float cs, sn;
      rope_cs(a.ft[i0 + k], t, cs, sn);  // rotate by +t positions
      const float y1 = u1[k] * cs - u2[k] * sn;
      const float y2 = u2[k] * cs + u1[k] * sn;
      u1[k] = y1;
      u2[k] = y2;
    }
  }
  int32_t blk = 0;
  if (a.pg.table) blk = a.pg.table[b * a.pg.max_blocks + t / a.pg.block_size];
  bf16_t* dst = a.tgt[kv] + l * a.ts.l + h * a.ts.h + target_row(a.pg, a.ts, b, t, blk) + i0;
  *reinterpret_cast<uint4*>(dst) = round_bf16x8(u1);
  *reinterpret_cast<uint4*>(dst + half) = round_bf16x8(u2);
}

}  // namespace

void launch_stage_pool(const StagedArgs& a, hipStream_t st) {
  stage_pool<<<dim3(a.tiles, a.din / 128, a.nl * 2), dim3(256), 0, st>>>(a);
}

void launch_stage_project(const StagedArgs& a, hipStream_t st) {
  stage_project<<<dim3(a.tiles, (a.dout + 127) / 128, a.nl * 2), dim3(256), 0, st>>>(a);
}

void launch_stage_store(const StagedArgs& a, hipStream_t st) {
  const int groups = a.ht * (a.dt / 16);
  stage_store<<<dim3(a.tiles * 4, (groups + 7) / 8, a.nl * 2), dim3(256), 0, st>>>(a);
}

}  // namespace kvx
