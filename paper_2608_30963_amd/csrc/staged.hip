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

// Z is kept in the order stage_project's matrix-core loads read it: for
// each block of 32 rows and each 16-slot K step, the 64 lanes' A fragments
// (lane l: row l % 32, slots 8 (l / 32) .. +7) as one contiguous KiB, so a
// wave's fragment load is one coalesced 1 KiB read.  Element offset of the 8
// slots s .. s+7 (s % 8 == 0) of row r within one plane:
__device__ __forceinline__ int64_t zfrag(int64_t r, int s, int ks_n) {
  return (((r / 32) * ks_n + s / 16) * 64 + r % 32 + 32 * ((s / 8) % 2)) * 8;
}

// U (fp32, rows x dout) is kept in the order the MFMA accumulators hold it:
// for each block of 32 rows and 32 outputs, register v (0..15) of the 64
// lanes as 64 contiguous floats, lane l holding output l % 32 of row
// 8 (v / 4) + 4 (l / 32) + v % 4.  The 32 outputs of a row stay contiguous.
// Element offset of row r, output o:
__device__ __forceinline__ int64_t ufrag(int64_t r, int o, int nb_n) {
  const int rr = static_cast<int>(r % 32);
  const int v = 4 * (rr / 8) + rr % 4, lane = o % 32 + 32 * ((rr / 4) % 2);
  return (((r / 32) * nb_n + o / 32) * 16 + v) * 64 + lane;
}

// Stage 1.  grid: (row tiles, din / 128 chunks, layers x K|V); 256 threads.
// Chunk c holds the RoPE pairs 64c .. 64c+63 of the flattened (mixed layer,
// source head, frequency) list: first members in slots 0..63, second members
// in 64..127.  Thread: one 8-pair group g of the chunk for rows tid/8 + 32u.
// A wave's 64 stores cover 8 rows of 8 fragment slices each: 8 runs of
// 128 contiguous bytes.
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
  // fragment offset of slots c*128 + 8g of the thread's first row; the
  // second members (slots + 64) sit 4 K steps further
  const int64_t zu0 = zfrag(static_cast<int64_t>(tile) * kStageRows + threadIdx.x / 8,
                            c * 128 + 8 * g, a.din / 16);
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
    // rows i of this thread are i % 32 of row blocks 4 tile + u
    bf16_t* zu = zb + zu0 + static_cast<int64_t>(u) * a.din * 32;
    store_planes(zu, zu + plane, two, z1);
    store_planes(zu + 4 * 512, zu + 4 * 512 + plane, two, z2);
  }
}

// Stage 2.  One work item: 128 rows x 256 outputs of one (target layer,
// K|V) system, on 4 waves of 64 rows x 128 outputs (2 x 4 tiles of
// v_mfma_f32_32x32x16_bf16).  Z (in fragment order) and the plan's packed
// weights are copied slab by slab (two K steps: per plane 4 row blocks, and
// 8 output blocks, of 1 KiB fragments) from HBM straight into LDS with
// 16-byte-per-lane loads, which land lane-linear: the waves then read their
// fragments from LDS without bank conflicts, each fragment fetched from
// memory once per workgroup instead of once per wave.  Two stages: the copy
// of slab s + 1 is issued while slab s is contracted.  The 1-D grid is laid
// out for the 8 XCDs: workgroup n runs on XCD n % 8, so n is mapped to work
// item (n % 8) * per_xcd + n / 8 and each XCD walks one contiguous run of
// items (system-major, then row tile, then output tile): the items sharing a
// row tile, and the row tiles sharing a system's weights, run together on
// one L2.
constexpr int kProjRows = 128, kProjCols = 256;
constexpr int kProjChunks = 32;  // 1 KiB fragments per slab stage: A [2 planes][4][2], B [8][2]

typedef __attribute__((address_space(3))) char lds_char;

// Workgroup barrier for LDS hand-offs that leaves vector-memory operations in
// flight; the memory clobber keeps the compiler's LDS accesses on their side.
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// The slabs of one work item; TWO: the operand has a lo plane.  Output blocks
// past dout (nbv < 4) are computed against the last block's weights and not
// stored.
template <bool TWO>
__device__ __forceinline__ void project_slabs(const bf16_t* zb, int64_t plane, const bf16x8* wl,
                                              int rb0, int nb0w, int nb_n, int ks_n, int wi,
                                              int wj, bf16x8* lds, f32x16 (&acc)[2][4]) {
  constexpr int P = TWO ? 2 : 1;
  const int lane = threadIdx.x % 64;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x / 64);
  const int nb0 = nb0w - 4 * wj;  // first output block of the work item
  lds_char* const l3 = (lds_char*)(lds);
  // chunk c (wave w copies c = w + 4 m): A chunks (pl, row block, K step) at
  // (pl * 4 + rbl) * 2 + ksl, B chunks (output block, K step) at 16 + nbl * 2 + ksl
  auto copy_slab = [&](int s, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < (8 * P + 16) / 4; ++m) {
      const int c = w + 4 * m;
      const bool isb = c >= 8 * P;
      const int cc = isb ? c - 8 * P : c;
      const int slot = isb ? 16 + cc : cc;
      const void* g;
      if (isb) {
        const int nb = min(nb0 + cc / 2, nb_n - 1);
        g = wl + (static_cast<int64_t>(nb) * ks_n + 2 * s + cc % 2) * 64 + lane;
      } else {
        const int pl = cc / 8, rbl = (cc % 8) / 2;
        g = zb + pl * plane + ((static_cast<int64_t>(rb0 + rbl) * ks_n + 2 * s + cc % 2) * 64 + lane) * 8;
      }
      __builtin_amdgcn_global_load_lds(g, l3 + (st * kProjChunks + slot) * 1024, 16, 0, 0);
    }
  };
  const int nslab = ks_n / 2;
  copy_slab(0, 0);
  __builtin_amdgcn_s_waitcnt(0);
  lds_sync();
  for (int s = 0; s < nslab; ++s) {
    const bf16x8* f = lds + (s % 2) * kProjChunks * 64;
#pragma unroll
    for (int ksl = 0; ksl < 2; ++ksl) {
      bf16x8 fa[2][P], fb[4];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int pl = 0; pl < P; ++pl) fa[i][pl] = f[((pl * 4 + 2 * wi + i) * 2 + ksl) * 64 + lane];
#pragma unroll
      for (int jb = 0; jb < 4; ++jb) fb[jb] = f[(16 + (4 * wj + jb) * 2 + ksl) * 64 + lane];
      if (ksl == 0 && s + 1 < nslab) copy_slab(s + 1, (s + 1) % 2);
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
          acc[i][jb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i][0], fb[jb], acc[i][jb], 0, 0, 0);
          if constexpr (TWO)
            acc[i][jb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i][1], fb[jb], acc[i][jb], 0, 0, 0);
        }
    }
    // slab s + 1 has landed and every wave is done with this stage (the
    // MFMAs stay before the wait)
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(0);
    lds_sync();
  }
}

__global__ void __launch_bounds__(256, 2) stage_project(StagedArgs a, int per_xcd) {
  __shared__ __attribute__((aligned(16))) bf16x8 lds[2 * kProjChunks * 64];  // 64 KiB
  const int item = static_cast<int>(blockIdx.x % 8) * per_xcd + static_cast<int>(blockIdx.x / 8);
  const int n_ct = (a.dout + kProjCols - 1) / kProjCols;
  if (item >= a.nl * 2 * a.tiles * n_ct) return;  // whole workgroup: before any barrier
  const int ct = item % n_ct, tile = item / n_ct % a.tiles, sys = item / n_ct / a.tiles;
  const int ll = sys / 2, kv = sys % 2, l = a.l0 + ll;
  const int lane = threadIdx.x % 64, w = threadIdx.x / 64;
  const int wi = w / 2, wj = w % 2;
  const int nb_n = a.dout / 32, ks_n = a.din / 16;
  const int nb0 = ct * (kProjCols / 32) + wj * 4;  // first 32-output block of this wave
  const int nbv = min(4, nb_n - nb0);
  const int64_t plane = static_cast<int64_t>(a.rows_p) * a.din;
  const bf16_t* zb = a.z + static_cast<int64_t>(ll * 2 + kv) * 2 * plane;
  const bf16x8* wl = a.wp[kv] + static_cast<int64_t>(l) * nb_n * ks_n * 64;
  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][jb][v] = 0.f;
  // every wave takes part in the copies and barriers, also one whose
  // output blocks are all past dout (it stores nothing)
  if (a.planes[kv] == 2)
    project_slabs<true>(zb, plane, wl, tile * 4, nb0, nb_n, ks_n, wi, wj, lds, acc);
  else
    project_slabs<false>(zb, plane, wl, tile * 4, nb0, nb_n, ks_n, wi, wj, lds, acc);
  // U in D-fragment order: register v of every lane is 256 contiguous bytes
  const int r0 = tile * kProjRows + wi * 64;
  float* ub = a.u + static_cast<int64_t>(ll * 2 + kv) * a.rows_p * a.dout;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int jb = 0; jb < 4; ++jb)
      if (jb < nbv) {
        float* d = ub + ((static_cast<int64_t>(r0 / 32 + i) * nb_n + nb0 + jb) * 16) * 64 + lane;
#pragma unroll
        for (int v = 0; v < 16; ++v) d[v * 64] = acc[i][jb][v];
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
  const float* ub = a.u + static_cast<int64_t>(ll * 2 + kv) * a.rows_p * a.dout;
  const int64_t r = static_cast<int64_t>(tile) * kStageRows + i;
  const int nb_n = a.dout / 32;
  const float* bb = a.bias[kv] + static_cast<int64_t>(l) * a.dout;
  float u1[8], u2[8];
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    const float4 p1 = *reinterpret_cast<const float4*>(ub + ufrag(r, o1 + 4 * v, nb_n));
    const float4 p2 = *reinterpret_cast<const float4*>(ub + ufrag(r, o2 + 4 * v, nb_n));
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
  const int items = a.nl * 2 * a.tiles * ((a.dout + kProjCols - 1) / kProjCols);
  const int per_xcd = (items + 7) / 8;
  stage_project<<<dim3(per_xcd * 8), dim3(256), 0, st>>>(a, per_xcd);
}

void launch_stage_store(const StagedArgs& a, hipStream_t st) {
  const int groups = a.ht * (a.dt / 16);
  stage_store<<<dim3(a.tiles * 4, (groups + 7) / 8, a.nl * 2), dim3(256), 0, st>>>(a);
}

}  // namespace kvx
