// kernel_mfma.h -- fused bf16 translation kernel on the gfx950 matrix cores.
//
// One workgroup (4 waves) owns (target layer l, K|V, a tile of MT = 128 target
// rows of one context, an N tile of 256 output features).  The reduction runs
// over K-chunks of one source head (DS features) of one mixed source layer:
//
//   prologue   each thread gathers 16-byte pieces of the source rows named by
//              the alignment entries of its target rows, undoes the source
//              RoPE at each source position (fp64-reduced angle), pools with
//              the entry weights in fp32, and writes the chunk to LDS as bf16
//              -- as hi = bf16(z), lo = bf16(z - hi) when the operand is a
//              computed value and the plan asks for the split;
//   body       v_mfma_f32_32x32x16_bf16 over the chunk: A fragments from LDS,
//              B fragments (weights) straight from global memory, pre-packed
//              at plan time so each fragment is one contiguous 1 KiB load;
//   epilogue   bias, target RoPE on K (each lane holds both members of every
//              rotation pair, see below), round to bf16, stage through LDS
//              and write whole rows into the target cache layout.
//
// N tiling: output features are grouped in "pair blocks" of 64 features --
// 32 consecutive features c0..c0+31 of a target head and their RoPE partners
// c0+Dt/2..c0+Dt/2+31.  Wave w of N tile nt owns pair block 4*nt + w, so in
// the 32x32 accumulator layout (lane = column) a lane holds u_i and u_{i+Dt/2}
// for the same rows in the same register slot.  Requires Dt % 64 == 0.
//
// Accumulator layout of v_mfma_f32_32x32x16_bf16 (checked on the device):
//   A: lane l holds A[l%32][8*(l/32) + j], j < 8
//   B: lane l holds B[8*(l/32) + j][l%32]
//   D: register v of lane l holds D[8*(v/4) + 4*(l/32) + v%4][l%32]
#pragma once

#include "common.h"

namespace kvx {

constexpr int kMT = 128;       // target rows per tile
constexpr int kNT = 256;       // output features per tile (4 pair blocks)
constexpr int kThreads = 256;  // 4 waves
constexpr int kStagePad = 8;   // bf16 padding per staged output row

struct FusedArgs {
  const bf16_t* src[2];
  Strides ss;
  bf16_t* tgt[2];
  Strides ts;
  const bf16x8* wp[2];      // packed B fragments [Lt][dout/32][din/16][64 lanes]
  const float* bias[2];     // [Lt][dout]
  const int32_t* layer_map; // [Lt][mix]
  int32_t mix, hs, ht, dt, din, dout;
  const double* fs;         // [DS/2] source theta_i / 2pi
  const double* ft;         // [dt/2] target theta_i / 2pi
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const float* weight;
  int32_t identity;
  int32_t split_k;          // split the (de-rotated) K operand
  int32_t split_v;          // split the (pooled) V operand
  int32_t n_tiles;          // N tiles per (layer, K|V)
  int32_t row_tiles;        // row tiles of this launch (all contexts)
  BatchArgs ba;
};

// LDS bytes the kernel needs for a source head_dim DS.
template <int DS>
constexpr int fused_lds_bytes() {
  constexpr int a = 2 * kMT * (DS + 8) * 2;
  constexpr int o = kMT * (kNT + kStagePad) * 2;
  return a > o ? a : o;
}

// Linear block id -> logical tile, so each XCD (blocks are dealt round-robin
// to the 8 XCDs) sweeps one contiguous range of logical tiles and the weights
// of a (layer, K|V) stay in that XCD's L2.
__device__ __forceinline__ int xcd_remap(int id, int total) {
  const int q = total / 8, r = total % 8;
  const int x = id % 8, slot = id / 8;
  return x * q + min(x, r) + slot;
}

template <int DS>
__global__ void __launch_bounds__(kThreads) fused_kernel(FusedArgs a) {
  constexpr int LDA = DS + 8;           // LDS row stride (bf16) of the A planes
  constexpr int G = DS / 16;            // 8-wide groups per half head
  constexpr int UNITS = kMT * G / kThreads;  // (row, group) units per thread
  constexpr int KS = DS / 16;           // MFMA K-steps per chunk
  static_assert(kMT * G % kThreads == 0, "units must divide evenly");

  __shared__ __attribute__((aligned(16))) bf16_t lds[fused_lds_bytes<DS>() / 2];
  bf16_t* a_hi = lds;
  bf16_t* a_lo = lds + kMT * LDA;

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

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const bool is_k = (kv == 0);
  const bool split = is_k ? a.split_k : a.split_v;

  // this wave's pair block
  const int npb = a.dout / 64;
  const int pb = nt * 4 + wave;
  const bool wave_on = pb < npb;
  const int per_head = a.dt / 64;
  const int hp = wave_on ? pb / per_head : 0;
  const int q = wave_on ? pb % per_head : 0;
  const int c0 = hp * a.dt + 32 * q;    // first feature of the low half
  const int c1 = c0 + a.dt / 2;         // its RoPE partners
  const int NB = a.dout / 32;
  const int KSALL = a.din / 16;
  const bf16x8* wp = a.wp[kv] + static_cast<int64_t>(l) * NB * KSALL * 64;

  f32x16 acc[4][2];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
#pragma unroll
    for (int p = 0; p < 2; ++p) {
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[m][p][v] = 0.f;
    }
  }

  const bf16_t* src = a.src[kv];
  const int nchunks = a.mix * a.hs;
  for (int kc = 0; kc < nchunks; ++kc) {
    const int j = kc / a.hs;
    const int h = kc % a.hs;
    const int ls = a.layer_map[l * a.mix + j];
    const bf16_t* base = src + ls * a.ss.l + b * a.ss.b + h * a.ss.h;

    // B fragments of this chunk, issued before the prologue so their latency
    // overlaps it.
    bf16x8 bfr[KS][2];
    if (wave_on) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const int kg = kc * KS + ks;
        bfr[ks][0] = wp[(static_cast<int64_t>(c0 / 32) * KSALL + kg) * 64 + lane];
        bfr[ks][1] = wp[(static_cast<int64_t>(c1 / 32) * KSALL + kg) * 64 + lane];
      }
    }

    // ---- prologue: gather, de-rotate, pool, split -> LDS ----
#pragma unroll
    for (int u = 0; u < UNITS; ++u) {
      const int unit = tid + u * kThreads;
      const int r = unit / G;
      const int g = unit % G;
      const int t = t0 + r;
      float z0[8], z1[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) z0[i] = z1[i] = 0.f;
      if (t < tt) {
        int e0 = 0, e1 = 1;
        if (!a.identity) {
          e0 = a.row_ptr[row_base + t];
          e1 = a.row_ptr[row_base + t + 1];
        }
        for (int e = e0; e < e1; ++e) {
          const int k = a.identity ? t : a.col_idx[e];
          const float w = a.identity ? 1.f : a.weight[e];
          const bf16_t* p = base + k * a.ss.t + 8 * g;
          const uint4 v0 = *reinterpret_cast<const uint4*>(p);
          const uint4 v1 = *reinterpret_cast<const uint4*>(p + DS / 2);
          const uint32_t w0[4] = {v0.x, v0.y, v0.z, v0.w};
          const uint32_t w1[4] = {v1.x, v1.y, v1.z, v1.w};
          float x0[8], x1[8];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            x0[2 * i] = __uint_as_float(w0[i] << 16);
            x0[2 * i + 1] = __uint_as_float(w0[i] & 0xffff0000u);
            x1[2 * i] = __uint_as_float(w1[i] << 16);
            x1[2 * i + 1] = __uint_as_float(w1[i] & 0xffff0000u);
          }
          if (is_k) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              float c, s;
              rope_cs(a.fs[8 * g + i], k, c, s);
              const float y0 = x0[i] * c + x1[i] * s;
              const float y1 = x1[i] * c - x0[i] * s;
              x0[i] = y0;
              x1[i] = y1;
            }
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            z0[i] += w * x0[i];
            z1[i] += w * x1[i];
          }
        }
      }
      uint32_t h0[4], h1[4], l0[4], l1[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bf16_t a0 = f32_to_bf16(z0[2 * i]), a1 = f32_to_bf16(z0[2 * i + 1]);
        const bf16_t b0 = f32_to_bf16(z1[2 * i]), b1 = f32_to_bf16(z1[2 * i + 1]);
        h0[i] = a0 | (static_cast<uint32_t>(a1) << 16);
        h1[i] = b0 | (static_cast<uint32_t>(b1) << 16);
        const bf16_t la0 = f32_to_bf16(z0[2 * i] - bf16_to_f32(a0));
        const bf16_t la1 = f32_to_bf16(z0[2 * i + 1] - bf16_to_f32(a1));
        const bf16_t lb0 = f32_to_bf16(z1[2 * i] - bf16_to_f32(b0));
        const bf16_t lb1 = f32_to_bf16(z1[2 * i + 1] - bf16_to_f32(b1));
        l0[i] = la0 | (static_cast<uint32_t>(la1) << 16);
        l1[i] = lb0 | (static_cast<uint32_t>(lb1) << 16);
      }
      *reinterpret_cast<uint4*>(a_hi + r * LDA + 8 * g) = make_uint4(h0[0], h0[1], h0[2], h0[3]);
      *reinterpret_cast<uint4*>(a_hi + r * LDA + DS / 2 + 8 * g) =
          make_uint4(h1[0], h1[1], h1[2], h1[3]);
      if (split) {
        *reinterpret_cast<uint4*>(a_lo + r * LDA + 8 * g) =
            make_uint4(l0[0], l0[1], l0[2], l0[3]);
        *reinterpret_cast<uint4*>(a_lo + r * LDA + DS / 2 + 8 * g) =
            make_uint4(l1[0], l1[1], l1[2], l1[3]);
      }
    }
    __syncthreads();

    // ---- body: MFMA over the chunk ----
    if (wave_on) {
      const int arow = lane % 32;
      const int acol = 8 * (lane / 32);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const bf16x8 ah =
              *reinterpret_cast<const bf16x8*>(a_hi + (m * 32 + arow) * LDA + ks * 16 + acol);
          acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bfr[ks][0], acc[m][0], 0, 0, 0);
          acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah, bfr[ks][1], acc[m][1], 0, 0, 0);
          if (split) {
            const bf16x8 al =
                *reinterpret_cast<const bf16x8*>(a_lo + (m * 32 + arow) * LDA + ks * 16 + acol);
            acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bfr[ks][0], acc[m][0], 0, 0, 0);
            acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al, bfr[ks][1], acc[m][1], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();
  }

  // ---- epilogue: bias, target RoPE, bf16, stage in LDS ----
  constexpr int LDO = kNT + kStagePad;
  bf16_t* stage = lds;
  if (wave_on) {
    const int col = lane % 32;
    const float* bl = a.bias[kv] + static_cast<int64_t>(l) * a.dout;
    const float bias0 = bl[c0 + col], bias1 = bl[c1 + col];
    const double f = a.ft[32 * q + col];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int row = m * 32 + 8 * (v / 4) + 4 * (lane / 32) + (v % 4);
        float u0 = acc[m][0][v] + bias0;
        float u1 = acc[m][1][v] + bias1;
        if (is_k) {
          float c, s;
          rope_cs(f, t0 + row, c, s);
          const float y0 = u0 * c - u1 * s;
          const float y1 = u1 * c + u0 * s;
          u0 = y0;
          u1 = y1;
        }
        stage[row * LDO + wave * 64 + col] = f32_to_bf16(u0);
        stage[row * LDO + wave * 64 + 32 + col] = f32_to_bf16(u1);
      }
    }
  }
  __syncthreads();

  // ---- store whole 16-byte pieces of target rows ----
  bf16_t* dst = a.tgt[kv] + l * a.ts.l + b * a.ts.b;
  constexpr int PIECES = kMT * kNT / 8;  // 16-byte pieces in the tile
  for (int pc = tid; pc < PIECES; pc += kThreads) {
    const int r = pc / (kNT / 8);
    const int sc8 = pc % (kNT / 8);      // staged column / 8
    const int w = sc8 / 8;               // owning wave (pair block)
    const int pbw = nt * 4 + w;
    const int t = t0 + r;
    if (t >= tt || pbw >= npb) continue;
    const int half = (sc8 / 4) % 2;
    const int hpw = pbw / per_head;
    const int qw = pbw % per_head;
    const int colg = hpw * a.dt + 32 * qw + half * (a.dt / 2) + (sc8 % 4) * 8;
    const int hd = colg / a.dt;
    const int d = colg % a.dt;
    *reinterpret_cast<uint4*>(dst + hd * a.ts.h + t * a.ts.t + d) =
        *reinterpret_cast<const uint4*>(stage + r * LDO + sc8 * 8);
  }
}

}  // namespace kvx
