// kernel_mfma.h -- fused bf16 translation kernel on the gfx950 matrix cores.
//
// One workgroup owns (target layer l, K|V, a tile of MT = 128 target rows of
// one context, an N tile of 256 output features) and runs 8 waves in two
// roles over a sequence of K-chunks:
//
//   producers (waves 0-3)  gather 16-byte pieces of the source rows named by
//       the alignment entries of each target row, undo the source RoPE at
//       each source position (fp64-reduced angle), pool with the entry
//       weights in fp32, and write the chunk into one of two LDS buffers as
//       bf16 -- as hi = bf16(z), lo = bf16(z - hi) when the operand is a
//       computed value and the plan asks for the split.  Raw source data of
//       the next chunk is prefetched into registers while the current one is
//       transformed.
//   consumers (waves 4-7)  contract the chunk on v_mfma_f32_32x32x16_bf16:
//       weight fragments (pre-packed at plan time, one contiguous 1 KiB load
//       each) straight from global memory, token fragments from LDS; the
//       accumulators hold U^T = W Z^T (rows = output features, columns =
//       tokens).  The epilogue adds the bias, applies the target RoPE to K,
//       rounds to bf16 and stores 16-byte pieces of target rows directly.
//
// K-chunks: the source features of a target layer are organised as RoPE
// pairs (d, d + Ds/2) of every (mixed layer j, head h); chunk c holds the
// pairs 64c .. 64c+63 of the flattened (j, h, d) list, first members in LDS
// slots 0..63 and second members in slots 64..127.  For Ds = 128 a chunk is
// exactly one source head in natural order.  Weights are packed at plan time
// in the same slot order.
//
// N tiling: output features are grouped in "pair blocks" of 64 -- 32
// consecutive features c0..c0+31 of a target head and their RoPE partners
// c0+Dt/2.. -- and consumer wave w of N tile nt owns pair block 4*nt + w.
// In the accumulator layout a lane then holds u_i and u_{i+Dt/2} of the same
// token in the same register slot of two accumulators.  Requires Dt % 64 == 0.
//
// Register layout of v_mfma_f32_32x32x16_bf16 (checked on the device):
//   A: lane l holds A[l%32][8*(l/32) + j], j < 8
//   B: lane l holds B[8*(l/32) + j][l%32]
//   D: register v of lane l holds D[8*(v/4) + 4*(l/32) + v%4][l%32]
#pragma once

#include "common.h"

namespace kvx {

constexpr int kMT = 128;         // target rows per tile
constexpr int kNT = 256;         // output features per tile (4 pair blocks)
constexpr int kThreads = 512;    // 4 producer + 4 consumer waves
constexpr int kProducers = 256;  // producer threads
constexpr int kLDA = 128 + 8;    // LDS row stride (bf16) of one A plane
constexpr int kPlane = kMT * kLDA;  // bf16 elements per plane
constexpr int kUnits = kMT * 8 / kProducers;  // (row, 8-pair group) units per producer

struct FusedArgs {
  const bf16_t* src[2];
  Strides ss;
  bf16_t* tgt[2];
  Strides ts;
  const bf16x8* wp[2];      // packed fragments [Lt][dout/32][din/16][64 lanes]
  const float* bias[2];     // [Lt][dout]
  const int32_t* layer_map; // [Lt][mix]
  int32_t mix, hs, ds, ht, dt, din, dout;
  const double* fs;         // [ds/2] source theta_i / 2pi
  const double* ft;         // [dt/2] target theta_i / 2pi
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const float* weight;
  int32_t split_k;          // split the (de-rotated) K operand
  int32_t split_v;          // split the (pooled) V operand
  int32_t n_tiles;          // N tiles per (layer, K|V)
  int32_t row_tiles;        // row tiles of this launch (all contexts)
  BatchArgs ba;
};

constexpr int fused_lds_bytes() { return 2 * 2 * kPlane * 2; }

// Linear block id -> logical tile, so each XCD (blocks are dealt round-robin
// to the 8 XCDs) sweeps one contiguous range of logical tiles and the weights
// of a (layer, K|V) stay in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  const int q = total / 8, r = total % 8;
  const int x = id % 8, slot = id / 8;
  return x * q + min(x, r) + slot;
}

__device__ __forceinline__ void unpack8(const uint4 v, float* x) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Round 8 floats to bf16 (hardware RNE) and pack; optionally the residuals.
__device__ __forceinline__ uint4 pack8(const float* z) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
    bf16x2 p = {static_cast<__bf16>(z[2 * i]), static_cast<__bf16>(z[2 * i + 1])};
    o[i] = __builtin_bit_cast(uint32_t, p);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

__device__ __forceinline__ void residual8(const float* z, const uint4 hi, float* r) {
  float h[8];
  unpack8(hi, h);
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = z[i] - h[i];
}

// Address of the first member of 8-pair group `grp` (pairs 8*grp .. 8*grp+7
// of the flattened (j, h, d) list) for source token k, and its first freq.
struct PairGroup {
  const bf16_t* p;  // first members; second members at p + ds/2
  int i0;           // frequency index of the first pair
};

__device__ __forceinline__ PairGroup pair_group(const FusedArgs& a, const bf16_t* src, int l,
                                                int b, int grp) {
  const int half = a.ds / 2;
  const int pair = grp * 8;
  const int head_pairs = pair / half;  // (j, h) flattened
  const int i0 = pair % half;
  const int j = head_pairs / a.hs;
  const int h = head_pairs % a.hs;
  const int ls = a.layer_map[l * a.mix + j];
  PairGroup g;
  g.p = src + ls * a.ss.l + b * a.ss.b + h * a.ss.h + i0;
  g.i0 = i0;
  return g;
}

template <bool IDENT>
__global__ void __launch_bounds__(kThreads) fused_kernel(FusedArgs a) {
  __shared__ __attribute__((aligned(16))) bf16_t lds[fused_lds_bytes() / 2];

  // ---- tile decode (XCD-aware) ----
  const int logical = xcd_remap(blockIdx.x, gridDim.x);
  const int rt = logical % a.row_tiles;
  int rest = logical / a.row_tiles;
  const int nt = rest % a.n_tiles;
  rest /= a.n_tiles;
  const int kv = rest % 2;
  const int l = rest / 2;
  const int b = find_context(a.ba, rt);
  const int t0 = (rt - a.ba.tile_start[b]) * kMT;
  const int tt = a.ba.t_tgt[b];
  const int row_base = a.ba.row_base[b];
  const bool is_k = (kv == 0);
  const bool split = is_k ? a.split_k : a.split_v;
  const int nchunks = a.din / 128;
  const int tid = threadIdx.x;

  if (tid < kProducers) {
    // =========================== producers ===========================
    const int g = tid % 8;  // 8-pair group within the chunk
    const bf16_t* src = a.src[kv];
    int t_of[kUnits], e0_of[kUnits], e1_of[kUnits], k0_of[kUnits];
    float w0_of[kUnits];
#pragma unroll
    for (int u = 0; u < kUnits; ++u) {
      const int r = tid / 8 + 32 * u;
      const int t = t0 + r;
      t_of[u] = t;
      if (IDENT) {
        e0_of[u] = 0;
        e1_of[u] = t < tt ? 1 : 0;
        k0_of[u] = t;
        w0_of[u] = 1.f;
      } else {
        int e0 = 0, e1 = 0;
        if (t < tt) {
          e0 = a.row_ptr[row_base + t];
          e1 = a.row_ptr[row_base + t + 1];
        }
        e0_of[u] = e0;
        e1_of[u] = e1;
        k0_of[u] = e1 > e0 ? a.col_idx[e0] : 0;
        w0_of[u] = e1 > e0 ? a.weight[e0] : 0.f;
      }
    }

    // raw first-entry data of one chunk, prefetched a chunk ahead
    uint4 raw0[kUnits], raw1[kUnits];
    auto fetch = [&](int c) {
      const PairGroup pg = pair_group(a, src, l, b, c * 8 + g);
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        if (e1_of[u] > e0_of[u]) {
          const bf16_t* p = pg.p + k0_of[u] * a.ss.t;
          raw0[u] = *reinterpret_cast<const uint4*>(p);
          raw1[u] = *reinterpret_cast<const uint4*>(p + a.ds / 2);
        } else {
          raw0[u] = make_uint4(0, 0, 0, 0);
          raw1[u] = make_uint4(0, 0, 0, 0);
        }
      }
    };

    auto transform = [&](int c, bf16_t* hi, bf16_t* lo) {
      const PairGroup pg = pair_group(a, src, l, b, c * 8 + g);
      double f[8];
      if (is_k) {
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = a.fs[pg.i0 + i];
      }
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        const int r = tid / 8 + 32 * u;
        float z0[8], z1[8];
        {
          float x0[8], x1[8];
          unpack8(raw0[u], x0);
          unpack8(raw1[u], x1);
          const int k = k0_of[u];
          const float w = w0_of[u];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            float y0 = x0[i], y1 = x1[i];
            if (is_k) {
              float cs, sn;
              rope_cs(f[i], k, cs, sn);
              y0 = x0[i] * cs + x1[i] * sn;
              y1 = x1[i] * cs - x0[i] * sn;
            }
            z0[i] = w * y0;
            z1[i] = w * y1;
          }
        }
        if (!IDENT) {
          for (int e = e0_of[u] + 1; e < e1_of[u]; ++e) {
            const int k = a.col_idx[e];
            const float w = a.weight[e];
            const bf16_t* p = pg.p + k * a.ss.t;
            float x0[8], x1[8];
            unpack8(*reinterpret_cast<const uint4*>(p), x0);
            unpack8(*reinterpret_cast<const uint4*>(p + a.ds / 2), x1);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              float y0 = x0[i], y1 = x1[i];
              if (is_k) {
                float cs, sn;
                rope_cs(f[i], k, cs, sn);
                y0 = x0[i] * cs + x1[i] * sn;
                y1 = x1[i] * cs - x0[i] * sn;
              }
              z0[i] += w * y0;
              z1[i] += w * y1;
            }
          }
        }
        const uint4 h0 = pack8(z0), h1 = pack8(z1);
        *reinterpret_cast<uint4*>(hi + r * kLDA + 8 * g) = h0;
        *reinterpret_cast<uint4*>(hi + r * kLDA + 64 + 8 * g) = h1;
        if (split) {
          float d0[8], d1[8];
          residual8(z0, h0, d0);
          residual8(z1, h1, d1);
          *reinterpret_cast<uint4*>(lo + r * kLDA + 8 * g) = pack8(d0);
          *reinterpret_cast<uint4*>(lo + r * kLDA + 64 + 8 * g) = pack8(d1);
        }
      }
    };

    fetch(0);
    transform(0, lds, lds + kPlane);
    if (nchunks > 1) fetch(1);
    __syncthreads();
    for (int c = 0; c < nchunks; ++c) {
      if (c + 1 < nchunks) {
        bf16_t* buf = lds + ((c + 1) % 2) * 2 * kPlane;
        transform(c + 1, buf, buf + kPlane);
        if (c + 2 < nchunks) fetch(c + 2);
      }
      __syncthreads();
    }
    return;
  }

  // =========================== consumers ===========================
  const int lane = tid & 63;
  const int cw = (tid - kProducers) >> 6;  // consumer wave 0..3
  const int npb = a.dout / 64;
  const int pb = nt * 4 + cw;
  const bool wave_on = pb < npb;
  const int per_head = a.dt / 64;
  const int hp = wave_on ? pb / per_head : 0;
  const int q = wave_on ? pb % per_head : 0;
  const int c0 = hp * a.dt + 32 * q;   // first feature of the low half
  const int c1 = c0 + a.dt / 2;        // its RoPE partners
  const int KSALL = a.din / 16;
  const bf16x8* w0p =
      a.wp[kv] + (static_cast<int64_t>(l) * (a.dout / 32) + c0 / 32) * KSALL * 64 + lane;
  const bf16x8* w1p =
      a.wp[kv] + (static_cast<int64_t>(l) * (a.dout / 32) + c1 / 32) * KSALL * 64 + lane;

  f32x16 acc[4][2];
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int p = 0; p < 2; ++p)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[m][p][v] = 0.f;

  bf16x8 wf[8][2];
  auto load_w = [&](int c) {
    if (!wave_on) return;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      wf[ks][0] = w0p[(c * 8 + ks) * 64];
      wf[ks][1] = w1p[(c * 8 + ks) * 64];
    }
  };

  load_w(0);
  __syncthreads();
  const int trow = lane % 32;
  const int tcol = 8 * (lane / 32);
  for (int c = 0; c < nchunks; ++c) {
    const bf16_t* hi = lds + (c % 2) * 2 * kPlane;
    const bf16_t* lo = hi + kPlane;
    if (wave_on) {
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const int off = (m * 32 + trow) * kLDA + ks * 16 + tcol;
          const bf16x8 zh = *reinterpret_cast<const bf16x8*>(hi + off);
          acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks][0], zh, acc[m][0], 0, 0, 0);
          acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks][1], zh, acc[m][1], 0, 0, 0);
          if (split) {
            const bf16x8 zl = *reinterpret_cast<const bf16x8*>(lo + off);
            acc[m][0] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks][0], zl, acc[m][0], 0, 0, 0);
            acc[m][1] =
                __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks][1], zl, acc[m][1], 0, 0, 0);
          }
        }
      }
      if (c + 1 < nchunks) load_w(c + 1);
    }
    __syncthreads();
  }
  if (!wave_on) return;

  // ---- epilogue: bias, target RoPE on K, bf16, direct 8-byte stores ----
  // lane holds, for token column lane%32 of token block m, the features
  // f = 8*(v/4) + 4*(lane/32) + v%4 (v < 16) of blocks c0 and c1.
  const float* bl = a.bias[kv] + static_cast<int64_t>(l) * a.dout;
  bf16_t* dst = a.tgt[kv] + l * a.ts.l + b * a.ts.b;
  const int fq = 4 * (lane / 32);
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int t = t0 + m * 32 + lane % 32;
    if (t >= tt) continue;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      float u0[4], u1[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int fo = 8 * g4 + fq + i;  // feature offset within the 32-block
        u0[i] = acc[m][0][4 * g4 + i] + bl[c0 + fo];
        u1[i] = acc[m][1][4 * g4 + i] + bl[c1 + fo];
        if (is_k) {
          float cs, sn;
          rope_cs(a.ft[32 * q + fo], t, cs, sn);
          const float y0 = u0[i] * cs - u1[i] * sn;
          const float y1 = u1[i] * cs + u0[i] * sn;
          u0[i] = y0;
          u1[i] = y1;
        }
      }
      typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
      const bf16x2 p00 = {static_cast<__bf16>(u0[0]), static_cast<__bf16>(u0[1])};
      const bf16x2 p01 = {static_cast<__bf16>(u0[2]), static_cast<__bf16>(u0[3])};
      const bf16x2 p10 = {static_cast<__bf16>(u1[0]), static_cast<__bf16>(u1[1])};
      const bf16x2 p11 = {static_cast<__bf16>(u1[2]), static_cast<__bf16>(u1[3])};
      const int d0 = 32 * q + 8 * g4 + fq;  // dim within target head hp
      bf16_t* rowp = dst + hp * a.ts.h + t * a.ts.t;
      *reinterpret_cast<uint2*>(rowp + d0) =
          make_uint2(__builtin_bit_cast(uint32_t, p00), __builtin_bit_cast(uint32_t, p01));
      *reinterpret_cast<uint2*>(rowp + a.dt / 2 + d0) =
          make_uint2(__builtin_bit_cast(uint32_t, p10), __builtin_bit_cast(uint32_t, p11));
    }
  }
}

}  // namespace kvx
