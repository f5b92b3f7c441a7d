// fit.hip -- translator fit (kvx_fit.h): ridge least squares of the affine
// per-layer translator from paired caches (the Section 5 objective with the
// squared Frobenius distance).
//
// Device pipeline per batch of paired caches and group of target layers:
//   fit_prepare  Z (pooled, source-de-rotated rows) and Y (target rows
//                de-rotated by the target RoPE) as bf16 planes hi (and lo,
//                unless the values are exact bf16) of X^T[plane][feature][row],
//                stored in matrix-core fragment order (xfrag); adds the
//                column sums of Z and Y
//                and the row count (the bias column's entries) to the
//                accumulators;
//   fit_gram     acc[i][j] += sum_r X[r][i] X[r][j] for i over the Z features
//                and j >= i over Z and Y (upper Z^T Z blocks and Z^T Y),
//                v_mfma_f32_32x32x16_bf16 with hi*hi (+ hi*lo + lo*hi);
// and once per solve:
//   fit_solve    per system: A = Z^T Z + lam D (fp64), blocked Cholesky,
//                forward and backward substitution for the Z^T Y columns,
//                W = X^T[:din], b = X^T[din].
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "common.h"
#include "kvx_fit.h"

using namespace kvx;

namespace {

constexpr int kFB = 128;       // Gram block edge (features)
constexpr int kSlab = 32;      // rows per LDS slab of the Gram kernel
constexpr int kPrepRows = 64;   // rows per block of fit_prepare (rows padded to it)
constexpr int kPrepBlocks = 4;  // row blocks per workgroup of fit_prepare

// X^T (features x rows, per plane) is stored in the order the Gram's MFMA
// fragments read it: for each block of 32 features and each 16-row K step,
// the 64 lanes' fragments (lane l: feature l % 32, rows 8 (l / 32) .. +7) as
// one contiguous KiB.  A fragment is then one coalesced 1 KiB read, and a
// 16-byte-per-lane copy of it into LDS lands lane-linear, so the waves'
// fragment reads from LDS are free of bank conflicts.  Element offset of the
// 8 rows r .. r+7 (r % 8 == 0) of feature f, rp rows per plane:
__host__ __device__ constexpr int64_t xfrag(int64_t f, int64_t r, int64_t rp) {
  return (((f / 32) * (rp / 16) + r / 16) * 64 + f % 32 + 32 * ((r / 8) % 2)) * 8;
}
constexpr int kFitBatch = 64;  // contexts per launch

kvx_status fit_hip_fail(hipError_t e) { return hip_status(e); }

#define FIT_HIP(x)                                \
  do {                                            \
    hipError_t e_ = (x);                          \
    if (e_ != hipSuccess) return fit_hip_fail(e_); \
  } while (0)

int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Contexts of one launch: rows are concatenated per context.
struct FitCtx {
  int32_t n;
  int32_t row0[kFitBatch + 1];  // first row (within the launch) of each context
  int32_t csr0[kFitBatch];      // first CSR row of each context
};

struct PrepArgs {
  const void* src[2];
  Strides ss;
  const void* tgt[2];
  Strides ts;
  const int32_t* row_ptr;  // nullptr: identity alignment
  const int32_t* col_idx;
  const float* weight;
  const int32_t* layer_map;
  const double* fs;  // source theta / 2pi (zeros without RoPE)
  const double* ft;  // target theta / 2pi
  int32_t mix, hs, ds, ht, dt;
  int32_t din, dout, din_z, dout_p, F2, rp, nrows, l0;
  int32_t tz, ty;          // job tiles of Z pairs and of Y pairs (then padding tiles)
  int32_t pz[2], py[2];    // planes written per K|V: 2 (hi, lo) or 1 (exact bf16)
  int32_t src_rope, tgt_rope, vec;
  bf16_t* xt;  // [sys][2][F2 x rp in xfrag order], sys = (l - l0) * 2 + kv
  // bias sums (fit_bias): Z column sums into acc[sys][f][din], Y column sums
  // into acc[sys][din][din_p + c], the row count into acc[sys][din][din]
  float* acc;
  int32_t din_p, F, sys0, fit_bias;
  FitCtx ctx;
};

__device__ __forceinline__ int ctx_of(const FitCtx& c, int r) {
  int lo = 0, hi = c.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (c.row0[mid] <= r) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Eight consecutive elements as fp32: one 16-byte load (bf16) or two (fp32)
// when `vec`, else element by element.
template <typename T>
__device__ __forceinline__ void load8(const T* p, bool vec, float (&x)[8]);
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, bool vec, float (&x)[8]) {
  if (vec) {
    const uint4 r = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = bf16_to_f32(p[i]);
  }
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, bool vec, float (&x)[8]) {
  if (vec) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = p[i];
  }
}

// Feature (row of X^T) of local feature q of job tile jt, or -1: Z tiles hold
// 64 RoPE pairs of the flattened (mixed layer, source head, frequency) list
// (first members q < 64, second members 64 + q), Y tiles 64 pairs of the
// (target head, frequency) list after the din_z Z features, padding tiles
// 128 zero features (Z padding din .. din_z - 1, then Y padding).
__device__ __forceinline__ int tile_feature(const PrepArgs& a, int jt, int q) {
  const int m = q % 64, second = q / 64;
  if (jt < a.tz) {
    const int p = 64 * jt + m;
    if (p >= a.din / 2) return -1;
    const int half = a.ds / 2;
    return (p / half) * a.ds + p % half + second * half;
  }
  if (jt < a.tz + a.ty) {
    const int p = 64 * (jt - a.tz) + m;
    if (p >= a.dout / 2) return -1;
    const int half = a.dt / 2;
    return a.din_z + (p / half) * a.dt + p % half + second * half;
  }
  int idx = 128 * (jt - a.tz - a.ty) + q;
  if (idx < a.din_z - a.din) return a.din + idx;
  idx -= a.din_z - a.din;
  if (idx < a.dout_p - a.dout) return a.din_z + a.dout + idx;
  return -1;
}

// One workgroup: one job tile (128 features) x kPrepBlocks blocks of 64 rows
// of one system.  Per block, the rows are formed token-major (16-byte loads of
// 8 pairs, 8 lanes per 128-byte row segment), transposed through LDS, and
// written in fragment order (xfrag), 8 lanes per 128-byte run of 8 features.
// Each feature's sum over the workgroup's rows goes to the bias accumulators
// in one atomic add.  grid: (job tiles, rp / (64 kPrepBlocks), systems of the
// group).
template <typename T>
__global__ void __launch_bounds__(256, 4) fit_prepare(PrepArgs a) {
  __shared__ float tr[128][65];  // [local feature][row]
  const int jt = blockIdx.x, sys = blockIdx.z;
  const int l = a.l0 + sys / 2, kv = sys % 2;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const bool vec = a.vec != 0;
  const int64_t plane = static_cast<int64_t>(a.F2) * a.rp;
  bf16_t* base = a.xt + static_cast<int64_t>(sys) * 2 * plane;
  float bsum[4] = {0.f, 0.f, 0.f, 0.f};  // this lane's octets of its 4 pieces, over the blocks
  // the lane's 8 pairs (the same in every row block)
  const bool isz = jt < a.tz;
  const int g = lane % 8;
  const int npairs = isz ? a.din / 2 : a.dout / 2;
  const int p0 = 64 * (isz ? jt : jt - a.tz) + 8 * g;  // 8 pairs of one head
  const int half = (isz ? a.ds : a.dt) / 2;
  const int hp = p0 / half, i0 = p0 % half;
  const int j = hp / a.hs, hz = hp % a.hs;  // Z: mixed layer, source head
  const bool job = jt < a.tz + a.ty;
  const T* zb = job && isz ? static_cast<const T*>(a.src[kv]) +
                                 a.layer_map[l * a.mix + (p0 < npairs ? j : 0)] * a.ss.l +
                                 hz * a.ss.h + i0
                           : nullptr;
  const T* yb = job && !isz ? static_cast<const T*>(a.tgt[kv]) + l * a.ts.l + hp * a.ts.h + i0
                            : nullptr;
  const bool rot = job && kv == 0 && (isz ? a.src_rope : a.tgt_rope);
  // frequencies in registers (loads per use would wait behind the stores)
  double fr[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) fr[q] = rot && p0 < npairs ? (isz ? a.fs : a.ft)[i0 + q] : 0.0;
#pragma unroll 1
  for (int rb = 0; rb < kPrepBlocks; ++rb) {
  const int r0 = (blockIdx.y * kPrepBlocks + rb) * kPrepRows;
  if (r0 >= a.rp) break;  // uniform
  if (rb > 0) __syncthreads();  // the previous block's reads of tr are done
  if (job) {
    if (!isz || !a.row_ptr) {
      // one row per unit (native target rows, identity-aligned source rows):
      // both units' loads are issued before either is used
      const T* ptr[2];
      int pos[2];
      bool ok[2];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int r = r0 + lane / 8 + 8 * w + 32 * u;
        ok[u] = r < a.nrows && p0 < npairs;
        const int b = ctx_of(a.ctx, ok[u] ? r : 0);
        const int t = ok[u] ? r - a.ctx.row0[b] : 0;
        pos[u] = t;
        ptr[u] = isz ? zb + b * a.ss.b + t * a.ss.t : yb + b * a.ts.b + t * a.ts.t;
      }
      float x[2][2][8];
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (ok[u]) {
          load8<T>(ptr[u], vec, x[u][0]);
          load8<T>(ptr[u] + half, vec, x[u][1]);
        } else {
#pragma unroll
          for (int q = 0; q < 8; ++q) x[u][0][q] = x[u][1][q] = 0.f;
        }
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int i = lane / 8 + 8 * w + 32 * u;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          float y1 = x[u][0][q], y2 = x[u][1][q];
          if (rot) {
            float c, sn;
            rope_cs(fr[q], pos[u], c, sn);
            y1 = x[u][0][q] * c + x[u][1][q] * sn;
            y2 = x[u][1][q] * c - x[u][0][q] * sn;
          }
          tr[8 * g + q][i] = y1;
          tr[64 + 8 * g + q][i] = y2;
        }
      }
    } else {
      // pooled source rows (span alignment): entries of the CSR row
#pragma unroll 1
      for (int u = 0; u < 2; ++u) {
        const int i = lane / 8 + 8 * w + 32 * u;
        const int r = r0 + i;
        float v1[8], v2[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) v1[q] = v2[q] = 0.f;
        if (r < a.nrows && p0 < npairs) {
          const int b = ctx_of(a.ctx, r);
          const int t = r - a.ctx.row0[b];
          const T* sb = zb + b * a.ss.b;
          const int e0 = a.row_ptr[a.ctx.csr0[b] + t];
          const int e1 = a.row_ptr[a.ctx.csr0[b] + t + 1];
          for (int e = e0; e < e1; ++e) {
            const int k = a.col_idx[e];
            const float wt = a.weight[e];
            float x1[8], x2[8];
            load8<T>(sb + k * a.ss.t, vec, x1);
            load8<T>(sb + k * a.ss.t + half, vec, x2);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
              float y1 = x1[q], y2 = x2[q];
              if (rot) {
                float c, sn;
                rope_cs(fr[q], k, c, sn);
                y1 = x1[q] * c + x2[q] * sn;
                y2 = x2[q] * c - x1[q] * sn;
              }
              v1[q] += wt * y1;
              v2[q] += wt * y2;
            }
          }
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          tr[8 * g + q][i] = v1[q];
          tr[64 + 8 * g + q][i] = v2[q];
        }
      }
    }
  } else {
    for (int idx = tid; idx < 128 * 64; idx += 256) tr[idx / 64][idx % 64] = 0.f;
  }
  __syncthreads();
  // fragment-order output: piece = (local feature, 8-row octet)
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int piece = tid + 256 * k;
    const int q = piece / 8, oct = piece % 8;
    const int f = tile_feature(a, jt, q);
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = tr[q][8 * oct + e];
#pragma unroll
    for (int e = 0; e < 8; ++e) bsum[k] += v[e];
    if (f < 0) continue;
    const bool zf = f < a.din_z;
    const bool two = (zf ? a.pz[kv] : a.py[kv]) == 2;
    uint32_t h[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bf16_t h0 = f32_to_bf16(v[2 * i]), h1 = f32_to_bf16(v[2 * i + 1]);
      const bf16_t l0 = f32_to_bf16(v[2 * i] - bf16_to_f32(h0));
      const bf16_t l1 = f32_to_bf16(v[2 * i + 1] - bf16_to_f32(h1));
      h[i] = static_cast<uint32_t>(h0) | (static_cast<uint32_t>(h1) << 16);
      lo[i] = static_cast<uint32_t>(l0) | (static_cast<uint32_t>(l1) << 16);
    }
    bf16_t* dst = base + xfrag(f, r0 + 8 * oct, a.rp);
    *reinterpret_cast<uint4*>(dst) = make_uint4(h[0], h[1], h[2], h[3]);
    if (two) *reinterpret_cast<uint4*>(dst + plane) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
  }
  }
  if (!a.fit_bias) return;
  // each feature's sum over the workgroup's rows: its 8 octet lanes are adjacent
  float* acc = a.acc + static_cast<int64_t>(a.sys0 + sys) * a.din_p * a.F;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    float sum = bsum[k];
    sum += __shfl_xor(sum, 1);
    sum += __shfl_xor(sum, 2);
    sum += __shfl_xor(sum, 4);
    const int piece = tid + 256 * k;
    const int f = tile_feature(a, jt, piece / 8);
    if (f < 0 || piece % 8 != 0 || jt >= a.tz + a.ty) continue;
    if (f < a.din_z)
      atomicAdd(acc + static_cast<int64_t>(f) * a.F + a.din, sum);
    else
      atomicAdd(acc + static_cast<int64_t>(a.din) * a.F + a.din_p + (f - a.din_z), sum);
  }
  if (jt == 0 && blockIdx.y == 0 && tid == 0)
    atomicAdd(acc + static_cast<int64_t>(a.din) * a.F + a.din, static_cast<float>(a.nrows));
}

struct GramArgs {
  const bf16_t* xt;   // [sys][2][F2 x rp in xfrag order]
  float* acc;         // [sys_total][din_p][F]; this group starts at sys0
  int32_t F2, rp, nbi, nbj, sys0, nblk;
  int32_t din_z, din_p, F;
  int32_t pz[2], py[2];  // operand planes per K|V (1: exact bf16, lo plane absent)
};

typedef __attribute__((address_space(3))) char lds_char;

// One workgroup: one 128 x 128 block (bi, bj >= bi) of one system, all rows:
// bi over the Z features, bj over Z and Y (the bias column's sums come from
// fit_prepare).  One launch covers the K (kv = 0) or the V (kv = 1) systems
// of a layer group, whose operands have PZ planes on the Z side and PY on the
// Y side (1: exact bf16, lo plane absent), and LDS is sized for the planes
// there are.  Work items are system-major and each XCD takes a contiguous
// range, so the workgroups that re-read one system's operands share that
// XCD's L2.
// Slabs of 32 rows (two K steps) of both feature blocks are copied from HBM
// straight into LDS (16 bytes per lane, lane-linear: the fragments' own
// order), kSt deep (as many 16-32 KiB stages as fit 64 KiB, 2 to 4), the copy
// of slab s + kSt - 1 issued as slab s is computed.  Four waves: wave pair p (0, 1) takes K step p of every slab and
// each wave of a pair 64 of the block's rows x all 128 columns (2 x 4 MFMA
// tiles), so a K step reads 6 fragments (per plane) for 8 tile products; the
// pairs' partial sums are added through LDS at the end, in a fixed order.
// Products: hi*hi, plus hi*lo and lo*hi when the B and the A operand have a
// lo plane.
// s_waitcnt immediate that waits until at most n vector-memory operations of
// this wave are outstanding (LDS and export counters left alone)
constexpr int vmcnt_le(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Workgroup barrier for LDS hand-offs that leaves vector-memory operations in
// flight (__syncthreads() would wait for all of them, the copies of later
// slabs included); the memory clobber keeps the compiler's LDS accesses on
// their side of it.
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

template <int PZ, int PY>
__global__ void __launch_bounds__(256, 2) fit_gram(GramArgs a, int kv) {
  constexpr int PA = PZ, PB = PZ > PY ? PZ : PY;  // planes staged per side
  constexpr int kChunk = 64 * 8;                  // bf16 of one fragment (1 KiB)
  constexpr int kStage = (PA + PB) * 8 * kChunk;  // bf16 per slab: [A planes | B planes][4 fb][2 ks]
  constexpr int kRed = 2 * 2 * 2 * 16 * 64;       // floats of one half of a pair's sums
  constexpr int kSt = 32768 / kStage < 2 ? 2 : (32768 / kStage > 4 ? 4 : 32768 / kStage);
  constexpr int kBytes = kSt * kStage * 2 > kRed * 4 ? kSt * kStage * 2 : kRed * 4;
  // copies per wave and slab (fewer when the B block has no lo plane)
  constexpr int kCopies = (PA + PB) * 2 - (PB == 2 && PZ != PY ? 2 : 0);
  __shared__ __attribute__((aligned(16))) char lds[kBytes];
  const int wid = xcd_remap(blockIdx.x, gridDim.x);
  const int sys = 2 * (wid / a.nblk) + kv;  // system within the layer group
  int x = wid % a.nblk;
  int bi = 0;
  while (x >= a.nbj - bi) {
    x -= a.nbj - bi;
    ++bi;
  }
  const int bj = bi + x;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int pk = w / 2, wi = w % 2;  // K step of the slab, 64-row half of the block
  const bf16_t* xs = a.xt + static_cast<int64_t>(sys) * 2 * a.F2 * a.rp;
  const int64_t plane = static_cast<int64_t>(a.F2) * a.rp;
  const int ksn = a.rp / 16;
  constexpr bool lo_a = PZ == 2;
  const bool lo_b = (bj * kFB < a.din_z ? PZ : PY) == 2;

  // copy of slab s into stage st: chunk c (wave w takes c = w + 4 m) is
  // side A (c < 8 PA) or B, plane pl, feature block fbl, K step ksl
  lds_char* const lds3 = (lds_char*)(lds);  // the LDS address space (sets M0 for the copies)
  auto copy_slab = [&](int s, int st) __attribute__((always_inline)) {
#pragma unroll
    for (int m = 0; m < (PA + PB) * 2; ++m) {
      const int c = w + 4 * m;
      const bool isb = c >= PA * 8;
      const int cc = isb ? c - PA * 8 : c;
      const int pl = cc / 8, fbl = (cc % 8) / 2, ksl = cc % 2;
      if (isb && pl == 1 && !lo_b) continue;
      const int fb = (isb ? bj : bi) * 4 + fbl;
      const bf16_t* g =
          xs + pl * plane + (static_cast<int64_t>(fb) * ksn + 2 * s + ksl) * kChunk + lane * 8;
      __builtin_amdgcn_global_load_lds(g, lds3 + (st * kStage + c * kChunk) * 2, 16, 0, 0);
    }
  };

  f32x16 acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const int nslab = a.rp / kSlab;
#pragma unroll
  for (int s = 0; s + 1 < kSt; ++s)
    if (s < nslab) copy_slab(s, s);
  // slab 0 has landed: the copies of the kSt - 2 slabs after it may still be
  // in flight, at least kCopies each; with fewer slabs, wait for all
  if (nslab >= kSt - 1)
    __builtin_amdgcn_s_waitcnt(vmcnt_le((kSt - 2) * kCopies));
  else
    __builtin_amdgcn_s_waitcnt(vmcnt_le(0));
  lds_sync();
  const bf16x8* frag = reinterpret_cast<const bf16x8*>(lds);
  for (int s = 0; s < nslab; ++s) {
    const int st = s % kSt;
    // this wave's fragments of the slab, then the next copy, then the MFMAs
    bf16x8 fa[2][PA], fb[4][PB];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int pl = 0; pl < PA; ++pl)
        fa[t][pl] = frag[(st * kStage) / 8 + ((pl * 4 + 2 * wi + t) * 2 + pk) * 64 + lane];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int pl = 0; pl < PB; ++pl)
        if (pl == 0 || lo_b)
          fb[j][pl] = frag[(st * kStage) / 8 + (PA * 8 + (pl * 4 + j) * 2 + pk) * 64 + lane];
    if (s + kSt - 1 < nslab) copy_slab(s + kSt - 1, (s + kSt - 1) % kSt);
    // hi*hi, hi*lo, lo*hi; consecutive MFMAs use different accumulators
#pragma unroll
    for (int term = 0; term < 3; ++term)
      if (term == 0 || (term == 1 ? lo_b : lo_a))
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                fa[i][term == 2 ? PA - 1 : 0], fb[j][term == 1 ? PB - 1 : 0], acc[i][j], 0, 0, 0);
    // the copies of slab s + 1 have landed and every wave is done with stage
    // st.  While this iteration issued a copy, the kSt - 2 slabs after s + 1
    // have theirs in flight, at least kCopies each, all issued after slab
    // s + 1's; at the end, wait for all.  The MFMAs stay before the wait:
    // they are what hides the copies.
    __builtin_amdgcn_sched_barrier(0);
    if (s + kSt - 1 < nslab)
      __builtin_amdgcn_s_waitcnt(vmcnt_le((kSt - 2) * kCopies));
    else
      __builtin_amdgcn_s_waitcnt(vmcnt_le(0));
    lds_sync();
  }
  __builtin_amdgcn_s_waitcnt(vmcnt_le(0));
  // pair 1 hands its sums to pair 0 through LDS, half the columns at a time
  // (lane-linear, [wi][i][jj][v][lane]); pair 0 adds them and updates the
  // accumulators: D register v of lane l is row 8(v/4) + 4(l/32) + v%4,
  // column l%32 of its tile
  float* red = reinterpret_cast<float*>(lds);
  float* out = a.acc + static_cast<int64_t>(a.sys0 + sys) * a.din_p * a.F;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (pk == 1) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            red[(((wi * 2 + i) * 2 + jj) * 16 + v) * 64 + lane] = acc[i][2 * h + jj][v];
    }
    __syncthreads();
    if (pk == 0) {
      // per tile: its 16 accumulator loads first, then the stores
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int f = bj * kFB + (2 * h + jj) * 32 + lane % 32;  // feature of X^T
          const int col = f < a.din_z ? f : a.din_p + (f - a.din_z);
          float* q = out + static_cast<int64_t>(bi * kFB + wi * 64 + i * 32 + 4 * (lane / 32)) * a.F + col;
          float old[16];
#pragma unroll
          for (int v = 0; v < 16; ++v) old[v] = q[static_cast<int64_t>(8 * (v / 4) + v % 4) * a.F];
#pragma unroll
          for (int v = 0; v < 16; ++v)
            q[static_cast<int64_t>(8 * (v / 4) + v % 4) * a.F] =
                old[v] + (acc[i][2 * h + jj][v] + red[(((wi * 2 + i) * 2 + jj) * 16 + v) * 64 + lane]);
        }
    }
    __syncthreads();
  }
}

struct SolveArgs {
  const float* acc;  // [sys][din_p][F]
  double* A;         // [group][n][n] workspace, one per system of the launch
  double* X;         // [group][n][dout] workspace (right-hand sides, then solution)
  int32_t sys0;      // first system of the launch: system sys0 + blockIdx.y (.x)
  float* w[2];       // [Lt][dout][din]
  float* b[2];       // [Lt][dout] or nullptr
  int32_t* status;   // set to 1 if a pivot is not positive
  double lam;
  int32_t n, din, dout, din_p, F, fit_bias;
  int32_t np;  // n rounded up to the panel width: the padding unknowns get an
               // identity block and zero right-hand sides (so they solve to 0)
};

// The solve of each (layer, K|V) system, A = Zt^T Zt + lam D and
// L L^T X = Zt^T Y in fp64, as a blocked right-looking Cholesky spread over
// many workgroups: per 32-wide panel, one workgroup per system factors the
// diagonal block, solves the panel's rows below it and the panel's rows of
// the forward substitution (L Y = B); then 64 x 64 tiles of the trailing
// matrix and of the right-hand sides are updated by one workgroup each.  The
// backward substitution (L^T X = Y) runs panel by panel from the last, again
// with one workgroup per system for the diagonal block and tiles for the
// updates of the rows above.
constexpr int kSB = 32;  // panel width
constexpr int kST = 64;  // update tile edge

__device__ __forceinline__ double* sys_A(const SolveArgs& a, int g) {
  return a.A + static_cast<int64_t>(g) * a.np * a.np;
}
__device__ __forceinline__ double* sys_X(const SolveArgs& a, int g) {
  return a.X + static_cast<int64_t>(g) * a.np * a.dout;
}

// Lower triangle of A (ridge on the din weight unknowns, not the bias) and
// X = Zt^T Y from the upper accumulator blocks.  grid: (chunks, systems).
__global__ void __launch_bounds__(256) solve_build(SolveArgs a) {
  const int g = blockIdx.y;
  const float* acc = a.acc + static_cast<int64_t>(a.sys0 + g) * a.din_p * a.F;
  double* A = sys_A(a, g);
  double* X = sys_X(a, g);
  const int np = a.np;
  const int64_t nn = static_cast<int64_t>(np) * np;
  const int64_t total = nn + static_cast<int64_t>(np) * a.dout;
  for (int64_t idx = blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    if (idx < nn) {
      const int i = static_cast<int>(idx / np), j = static_cast<int>(idx % np);
      double v = 0.0;
      if (i >= a.n || j >= a.n) {
        v = i == j ? 1.0 : 0.0;
      } else if (j <= i) {
        v = acc[static_cast<int64_t>(j) * a.F + i];
        if (i == j && i < a.din) v += a.lam;
      }
      A[idx] = v;
    } else {
      const int64_t k = idx - nn;
      const int i = static_cast<int>(k / a.dout), c = static_cast<int>(k % a.dout);
      X[k] = i < a.n ? acc[static_cast<int64_t>(i) * a.F + a.din_p + c] : 0.0;
    }
  }
}

// Panel kb: factor the diagonal block in LDS and write L_kk back.
// grid: (systems).
__global__ void __launch_bounds__(256) solve_panel(SolveArgs a, int kb) {
  __shared__ double pk[kSB][kSB + 1];
  const int g = blockIdx.x, tid = threadIdx.x;
  const int n = a.np;
  constexpr int kw = kSB;
  double* A = sys_A(a, g);
  for (int idx = tid; idx < kSB * kSB; idx += 256) {
    const int i = idx / kSB, j = idx % kSB;
    pk[i][j] = (i < kw && j <= i) ? A[static_cast<int64_t>(kb + i) * n + kb + j] : 0.0;
  }
  __syncthreads();
  bool bad = false;
  for (int k = 0; k < kw; ++k) {
    const double dkk = pk[k][k];
    const bool ok = dkk > 0.0 && isfinite(dkk);
    bad |= !ok;
    const double d = ok ? sqrt(dkk) : 1.0;
    __syncthreads();
    if (tid == 0) pk[k][k] = d;
    for (int i = k + 1 + tid; i < kw; i += 256) pk[i][k] /= d;
    __syncthreads();
    for (int idx = tid; idx < kSB * kSB; idx += 256) {
      const int i = idx / kSB, j = idx % kSB;
      if (i > k && j > k && j <= i && i < kw) pk[i][j] -= pk[i][k] * pk[j][k];
    }
    __syncthreads();
  }
  if (bad && tid == 0) a.status[0] = 1;
  for (int idx = tid; idx < kSB * kSB; idx += 256) {
    const int i = idx / kSB, j = idx % kSB;
    if (i < kw && j <= i) A[static_cast<int64_t>(kb + i) * n + kb + j] = pk[i][j];
  }
}

// Panel kb, after its factor, `rhs` false: each thread one row below the
// diagonal block, L[i][kb..] = A[i][kb..] L_kk^-T; `rhs` true: each thread
// one right-hand side column of the panel's rows of L Y = B (X_k already
// holds B_k minus the earlier panels' terms).  Separate instantiations, so
// the compiler does not keep the factor's values live across both.
// grid: (ceil(items / 256), systems).
template <bool RHS>
__global__ void __launch_bounds__(256) solve_panel_rows(SolveArgs a, int kb) {
  __shared__ double pk[kSB][kSB + 1];
  const int g = blockIdx.y, tid = threadIdx.x;
  const int n = a.np, m = a.dout;
  constexpr int kw = kSB;
  double* A = sys_A(a, g);
  double* X = sys_X(a, g);
  for (int idx = tid; idx < kSB * kSB; idx += 256) {
    const int i = idx / kSB, j = idx % kSB;
    pk[i][j] = (i < kw && j <= i) ? A[static_cast<int64_t>(kb + i) * n + kb + j]
                                  : (i == j ? 1.0 : 0.0);
  }
  __syncthreads();
  const int item = blockIdx.x * 256 + tid;
  if (item >= (RHS ? m : n - kb - kw)) return;
  double* base = RHS ? X + static_cast<int64_t>(kb) * m + item
                     : A + static_cast<int64_t>(kb + kw + item) * n + kb;
  const int64_t step = RHS ? m : 1;
  double r[kSB];
#pragma unroll
  for (int q = 0; q < kSB; ++q) r[q] = q < kw ? base[q * step] : 0.0;
  // column by column: r_q is final once the earlier columns are subtracted
#pragma unroll
  for (int q = 0; q < kSB; ++q) {
    r[q] /= pk[q][q];
#pragma unroll
    for (int p = q + 1; p < kSB; ++p) r[p] -= pk[p][q] * r[q];
  }
#pragma unroll
  for (int q = 0; q < kSB; ++q)
    if (q < kw) base[q * step] = r[q];
}

// Trailing update after panel kb: 64 x 64 tiles of the lower triangle of
// A[t0:, t0:] (A[i][j] -= sum_q L[i][kb+q] L[j][kb+q]) and of X[t0:, :]
// (X[i][c] -= sum_q L[i][kb+q] Y[kb+q][c]), t0 = kb + 32.  Thread: a 4 x 4
// block of the tile.  grid: (tiles, systems).
__global__ void __launch_bounds__(256) solve_update(SolveArgs a, int kb) {
  __shared__ double P[kST][kSB + 1];  // L rows of the tile's rows
  __shared__ double Q[kST][kSB + 1];  // L rows of the tile's columns, or Y_k transposed
  const int g = blockIdx.y, tid = threadIdx.x;
  const int n = a.np, m = a.dout;
  constexpr int kw = kSB;
  const int t0 = kb + kw;
  const int nt = (n - t0 + kST - 1) / kST;
  const int ntri = nt * (nt + 1) / 2;
  const int nct = (m + kST - 1) / kST;
  int tile = blockIdx.x;
  if (tile >= ntri + nt * nct) return;
  double* A = sys_A(a, g);
  double* X = sys_X(a, g);
  const bool onA = tile < ntri;
  int ti, tj;
  if (onA) {
    ti = 0;
    while ((ti + 1) * (ti + 2) / 2 <= tile) ++ti;
    tj = tile - ti * (ti + 1) / 2;
  } else {
    tile -= ntri;
    ti = tile / nct;
    tj = tile % nct;
  }
  const int i0 = t0 + ti * kST;
  const int j0 = onA ? t0 + tj * kST : tj * kST;
  for (int idx = tid; idx < kST * kSB; idx += 256) {
    const int r = idx / kSB, q = idx % kSB;
    P[r][q] = (i0 + r < n && q < kw) ? A[static_cast<int64_t>(i0 + r) * n + kb + q] : 0.0;
    if (onA)
      Q[r][q] = (j0 + r < n && q < kw) ? A[static_cast<int64_t>(j0 + r) * n + kb + q] : 0.0;
    else  // Q[c][q] = Y[kb + q][j0 + c]
      Q[r][q] = (j0 + r < m && q < kw) ? X[static_cast<int64_t>(kb + q) * m + j0 + r] : 0.0;
  }
  __syncthreads();
  const int rb = (tid / 16) * 4, cb = (tid % 16) * 4;
  double s[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) s[x][y] = 0.0;
#pragma unroll 4
  for (int q = 0; q < kw; ++q) {
    double pv[4], qv[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      pv[x] = P[rb + x][q];
      qv[x] = Q[cb + x][q];
    }
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) s[x][y] += pv[x] * qv[y];
  }
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int i = i0 + rb + x, j = j0 + cb + y;
      if (onA) {
        if (i < n && j <= i) A[static_cast<int64_t>(i) * n + j] -= s[x][y];
      } else if (i < n && j < m) {
        X[static_cast<int64_t>(i) * m + j] -= s[x][y];
      }
    }
}

// Backward substitution, panel kb (from the last): L_kk^T X_k = X_k, one
// right-hand side column per thread.  grid: (ceil(dout / 256), systems).
__global__ void __launch_bounds__(256) solve_back_diag(SolveArgs a, int kb) {
  __shared__ double pk[kSB][kSB + 1];
  const int g = blockIdx.y, tid = threadIdx.x;
  const int n = a.np, m = a.dout;
  constexpr int kw = kSB;
  const double* A = sys_A(a, g);
  double* X = sys_X(a, g);
  for (int idx = tid; idx < kSB * kSB; idx += 256) {
    const int i = idx / kSB, j = idx % kSB;
    pk[i][j] = (i < kw && j <= i) ? A[static_cast<int64_t>(kb + i) * n + kb + j]
                                  : (i == j ? 1.0 : 0.0);
  }
  __syncthreads();
  const int c = blockIdx.x * 256 + tid;
  if (c >= m) return;
  double x[kSB];
#pragma unroll
  for (int q = 0; q < kSB; ++q) x[q] = q < kw ? X[static_cast<int64_t>(kb + q) * m + c] : 0.0;
#pragma unroll
  for (int q = kSB - 1; q >= 0; --q) {
    double v = x[q];
#pragma unroll
    for (int p = q + 1; p < kSB; ++p) v -= pk[p][q] * x[p];
    x[q] = v / pk[q][q];
  }
#pragma unroll
  for (int q = 0; q < kSB; ++q)
    if (q < kw) X[static_cast<int64_t>(kb + q) * m + c] = x[q];
}

// Backward update after panel kb: rows above it, X[j][c] -= sum_q
// L[kb+q][j] X[kb+q][c] for j < kb, in 64 x 64 tiles.  grid: (tiles, systems).
__global__ void __launch_bounds__(256) solve_back_update(SolveArgs a, int kb) {
  __shared__ double P[kST][kSB + 1];  // P[r][q] = L[kb + q][j0 + r]
  __shared__ double Q[kST][kSB + 1];  // Q[c][q] = X[kb + q][c0 + c]
  const int g = blockIdx.y, tid = threadIdx.x;
  const int n = a.np, m = a.dout;
  constexpr int kw = kSB;
  const int nct = (m + kST - 1) / kST;
  const int nrt = (kb + kST - 1) / kST;
  if (static_cast<int>(blockIdx.x) >= nrt * nct) return;
  const double* A = sys_A(a, g);
  double* X = sys_X(a, g);
  const int j0 = (blockIdx.x / nct) * kST, c0 = (blockIdx.x % nct) * kST;
  for (int idx = tid; idx < kST * kSB; idx += 256) {
    const int q = idx / kST, r = idx % kST;
    P[r][q] = (q < kw && j0 + r < kb) ? A[static_cast<int64_t>(kb + q) * n + j0 + r] : 0.0;
    Q[r][q] = (q < kw && c0 + r < m) ? X[static_cast<int64_t>(kb + q) * m + c0 + r] : 0.0;
  }
  __syncthreads();
  const int rb = (tid / 16) * 4, cb = (tid % 16) * 4;
  double s[4][4];
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) s[x][y] = 0.0;
#pragma unroll 4
  for (int q = 0; q < kw; ++q) {
    double pv[4], qv[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      pv[x] = P[rb + x][q];
      qv[x] = Q[cb + x][q];
    }
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
      for (int y = 0; y < 4; ++y) s[x][y] += pv[x] * qv[y];
  }
#pragma unroll
  for (int x = 0; x < 4; ++x)
#pragma unroll
    for (int y = 0; y < 4; ++y) {
      const int j = j0 + rb + x, c = c0 + cb + y;
      if (j < kb && c < m) X[static_cast<int64_t>(j) * m + c] -= s[x][y];
    }
}

// W = X[:din]^T (nn.Linear order) and b = X[din].  grid: (chunks, systems).
__global__ void __launch_bounds__(256) solve_write(SolveArgs a) {
  const int g = blockIdx.y;
  const int sys = a.sys0 + g;
  const int l = sys / 2, kv = sys % 2, m = a.dout;
  const double* X = sys_X(a, g);
  float* w = a.w[kv] + static_cast<int64_t>(l) * m * a.din;
  const int64_t total = static_cast<int64_t>(m) * a.din;
  for (int64_t idx = blockIdx.x * 256 + threadIdx.x; idx < total;
       idx += static_cast<int64_t>(gridDim.x) * 256) {
    const int c = static_cast<int>(idx / a.din), i = static_cast<int>(idx % a.din);
    w[idx] = static_cast<float>(X[static_cast<int64_t>(i) * m + c]);
  }
  if (a.b[kv] && blockIdx.x == 0)
    for (int c = threadIdx.x; c < m; c += 256)
      a.b[kv][static_cast<int64_t>(l) * m + c] =
          a.fit_bias ? static_cast<float>(X[static_cast<int64_t>(a.din) * m + c]) : 0.f;
}

// Enqueue the solve of `ng` systems (sa.sys0 ..) whose workspaces start at
// sa.A and sa.X.
kvx_status enqueue_solve(const SolveArgs& sa, int ng, hipStream_t st) {
  const int n = sa.np, m = sa.dout;
  const unsigned chunks = static_cast<unsigned>(
      std::min<int64_t>(1024, (int64_t(n) * (n + m) + 2047) / 2048));
  solve_build<<<dim3(chunks, ng), dim3(256), 0, st>>>(sa);
  FIT_HIP(hipGetLastError());
  const int nct = (m + kST - 1) / kST;
  for (int kb = 0; kb < n; kb += kSB) {
    solve_panel<<<dim3(ng), dim3(256), 0, st>>>(sa, kb);
    FIT_HIP(hipGetLastError());
    const int t0 = kb + std::min(kSB, n - kb);
    if (t0 < n) {
      solve_panel_rows<false><<<dim3((n - t0 + 255) / 256, ng), dim3(256), 0, st>>>(sa, kb);
      FIT_HIP(hipGetLastError());
    }
    solve_panel_rows<true><<<dim3((m + 255) / 256, ng), dim3(256), 0, st>>>(sa, kb);
    FIT_HIP(hipGetLastError());
    if (t0 < n) {
      const int nt = (n - t0 + kST - 1) / kST;
      solve_update<<<dim3(nt * (nt + 1) / 2 + nt * nct, ng), dim3(256), 0, st>>>(sa, kb);
      FIT_HIP(hipGetLastError());
    }
  }
  for (int kb = (n - 1) / kSB * kSB; kb >= 0; kb -= kSB) {
    solve_back_diag<<<dim3((m + 255) / 256, ng), dim3(256), 0, st>>>(sa, kb);
    FIT_HIP(hipGetLastError());
    if (kb > 0) {
      solve_back_update<<<dim3(((kb + kST - 1) / kST) * nct, ng), dim3(256), 0, st>>>(sa, kb);
      FIT_HIP(hipGetLastError());
    }
  }
  const unsigned wchunks = static_cast<unsigned>(
      std::min<int64_t>(256, (int64_t(m) * sa.din + 2047) / 2048));
  solve_write<<<dim3(std::max(1u, wchunks), ng), dim3(256), 0, st>>>(sa);
  FIT_HIP(hipGetLastError());
  return KVX_OK;
}

// Status flag of a solve: cleared by a kernel (not a memset) before the
// solve's launches.
__global__ void __launch_bounds__(64) clear_status(int32_t* status) {
  if (threadIdx.x == 0) status[0] = 0;
}

// Workspace of kvx_fit_solve_noalloc, held by every device the library runs
// on until the process ends: the fp64 matrices A and right-hand sides X of as
// many systems as fit, then the status flag.  Host code reaches it only
// through the per-device address from hipGetSymbolAddress (solve_workspace):
// the array's name in host code is a host-side stand-in, not a device
// address.
constexpr size_t kSolveWorkspaceBytes = size_t(128) << 20;
constexpr size_t kStatusBytes = 256;
static __device__ __align__(256) double scratch[kSolveWorkspaceBytes / sizeof(double)];

constexpr int kMaxDevices = 64;
std::mutex g_ws_mu;
void* g_ws[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per
// device (with that device current).
kvx_status solve_workspace(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e);
  if (dev < 0 || dev >= kMaxDevices) return KVX_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_ws_mu);
  if (!g_ws[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e);
    g_ws[dev] = p;
  }
  *out = g_ws[dev];
  return KVX_OK;
}

bool valid_side(const kvx_model& m) {
  return m.n_layers > 0 && m.n_kv_heads > 0 && m.head_dim > 0 && std::isfinite(m.rope_base);
}

std::vector<double> theta_table(const kvx_model& m) {
  std::vector<double> f(m.head_dim / 2, 0.0);
  const double two_pi = 6.283185307179586476925286766559;
  for (int i = 0; i < m.head_dim / 2; ++i) {
    double th = 0.0;
    if (m.inv_freq)
      th = m.inv_freq[i];
    else if (m.rope_base > 0.0)
      th = std::pow(m.rope_base, -2.0 * i / m.head_dim);
    f[i] = th / two_pi;
  }
  return f;
}

}  // namespace

struct kvx_fit {
  int device = 0;
  kvx_model src{}, tgt{};
  int32_t mix = 1, dtype = KVX_BF16, fit_bias = 1;
  int32_t din = 0, dout = 0, din_p = 0, dout_p = 0, F = 0, n = 0;
  int32_t din_z = 0, F2 = 0;  // prepared operands: Z features (padded), Z + Y
  int32_t src_rope = 0, tgt_rope = 0;
  int32_t* layer_map = nullptr;
  double* fs = nullptr;
  double* ft = nullptr;
  float* acc = nullptr;        // [Lt * 2][din_p][F]
  void* prep = nullptr;        // prepared operands X^T
  size_t prep_bytes = 0;
  void* solve_buf = nullptr;
  size_t solve_bytes = 0;
  int64_t rows = 0;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> timed;  // KVX_FIT_TIMING=1
};

extern "C" {

kvx_status kvx_fit_create(const kvx_fit_desc* d, kvx_fit** out) {
  if (out) *out = nullptr;
  if (!d || !out || !d->layer_map) return KVX_EINVAL;
  if (!valid_side(d->src) || !valid_side(d->tgt) || d->mix < 1) return KVX_EINVAL;
  if (d->dtype != KVX_F32 && d->dtype != KVX_BF16) return KVX_EINVAL;
  if (d->fit_bias != 0 && d->fit_bias != 1) return KVX_EINVAL;
  // 8 RoPE pairs per 16-byte piece of a head
  if (d->src.head_dim % 16 || d->tgt.head_dim % 16) return KVX_EUNSUPPORTED;
  const int64_t lt = d->tgt.n_layers;
  for (int64_t i = 0; i < lt * d->mix; ++i)
    if (d->layer_map[i] < 0 || d->layer_map[i] >= d->src.n_layers) return KVX_EINVAL;
  const int64_t din = int64_t(d->mix) * d->src.n_kv_heads * d->src.head_dim;
  const int64_t dout = int64_t(d->tgt.n_kv_heads) * d->tgt.head_dim;
  if (din > 16384 || dout > 16384) return KVX_ESHAPE;
  for (const kvx_model* m : {&d->src, &d->tgt})
    if (m->inv_freq)
      for (int i = 0; i < m->head_dim / 2; ++i)
        if (!std::isfinite(m->inv_freq[i])) return KVX_EINVAL;

  kvx_fit* f = new (std::nothrow) kvx_fit();
  if (!f) return KVX_ENOMEM;
  auto fail = [&](kvx_status s) {
    kvx_fit_destroy(f);
    return s;
  };
  f->src = d->src;
  f->tgt = d->tgt;
  f->src.inv_freq = f->tgt.inv_freq = nullptr;
  f->mix = d->mix;
  f->dtype = d->dtype;
  f->fit_bias = d->fit_bias;
  f->din = static_cast<int32_t>(din);
  f->dout = static_cast<int32_t>(dout);
  f->n = f->din + f->fit_bias;
  f->din_p = static_cast<int32_t>(round_up(f->n, kFB));
  f->dout_p = static_cast<int32_t>(round_up(dout, kFB));
  f->F = f->din_p + f->dout_p;
  f->din_z = static_cast<int32_t>(round_up(f->din, kFB));
  f->F2 = f->din_z + f->dout_p;
  f->src_rope = (d->src.inv_freq || d->src.rope_base > 0) ? 1 : 0;
  f->tgt_rope = (d->tgt.inv_freq || d->tgt.rope_base > 0) ? 1 : 0;
  hipError_t e = hipGetDevice(&f->device);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  const size_t mb = size_t(lt) * d->mix * sizeof(int32_t);
  e = hipMalloc(&f->layer_map, mb);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipMemcpy(f->layer_map, d->layer_map, mb, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  std::vector<double> fsv = theta_table(d->src), ftv = theta_table(d->tgt);
  e = hipMalloc(&f->fs, fsv.size() * sizeof(double));
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipMalloc(&f->ft, ftv.size() * sizeof(double));
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipMemcpy(f->fs, fsv.data(), fsv.size() * sizeof(double), hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipMemcpy(f->ft, ftv.data(), ftv.size() * sizeof(double), hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  const size_t ab = size_t(lt) * 2 * f->din_p * f->F * sizeof(float);
  e = hipMalloc(&f->acc, ab);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipMemset(f->acc, 0, ab);
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return fail(fit_hip_fail(e));
  *out = f;
  return KVX_OK;
}

kvx_status kvx_fit_accumulate(kvx_fit* f, const kvx_fit_io* io_in, void* stream) {
  if (!f || !io_in) return KVX_EINVAL;
  kvx_fit_io io = *io_in;
  if (io.batch < 0 || io.src_tokens < 0 || io.tgt_capacity < 0) return KVX_EINVAL;
  if (io.batch == 0) return KVX_OK;
  const bool identity = io.tgt_tokens == nullptr;
  std::vector<int32_t> tt(io.batch);
  int64_t rows = 0;
  for (int b = 0; b < io.batch; ++b) {
    const int32_t t = identity ? io.src_tokens : io.tgt_tokens[b];
    if (t < 0) return KVX_EINVAL;
    if (t > io.tgt_capacity) return KVX_ESHAPE;
    tt[b] = t;
    rows += t;
  }
  if (rows == 0) return KVX_OK;
  if (!io.src_k || !io.src_v || !io.tgt_k || !io.tgt_v) return KVX_EINVAL;
  if (!identity && (!io.row_ptr || !io.col_idx || !io.weight)) return KVX_EINVAL;
  if (rows > INT32_MAX / 2) return KVX_ESHAPE;
  const int64_t Hs = f->src.n_kv_heads, Ds = f->src.head_dim;
  const int64_t Lt = f->tgt.n_layers, Ht = f->tgt.n_kv_heads, Dt = f->tgt.head_dim;
  const int64_t B = io.batch;
  auto all_zero = [](const int64_t* s) { return !s[0] && !s[1] && !s[2] && !s[3]; };
  if (all_zero(io.src_stride)) {
    io.src_stride[3] = Ds;
    io.src_stride[2] = Ds * io.src_tokens;
    io.src_stride[1] = Hs * io.src_stride[2];
    io.src_stride[0] = B * io.src_stride[1];
  }
  if (all_zero(io.tgt_stride)) {
    io.tgt_stride[3] = Dt;
    io.tgt_stride[2] = Dt * int64_t(io.tgt_capacity);
    io.tgt_stride[1] = Ht * io.tgt_stride[2];
    io.tgt_stride[0] = B * io.tgt_stride[1];
  }
  for (int i = 0; i < 4; ++i)
    if (io.src_stride[i] < 0 || io.tgt_stride[i] < 0) return KVX_ESHAPE;
  if ((io.src_stride[3] < Ds && io.src_tokens > 1) ||
      (io.tgt_stride[3] < Dt && io.tgt_capacity > 1))
    return KVX_ESHAPE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int esz = f->dtype == KVX_F32 ? 4 : 2;
  // 16-byte loads of 8 pairs need 8-element aligned rows and buffers
  bool vec = (reinterpret_cast<uintptr_t>(io.src_k) | reinterpret_cast<uintptr_t>(io.src_v) |
              reinterpret_cast<uintptr_t>(io.tgt_k) | reinterpret_cast<uintptr_t>(io.tgt_v)) %
                 16 == 0;
  for (int i = 0; i < 4; ++i)
    if (io.src_stride[i] % 8 || io.tgt_stride[i] % 8) vec = false;
  // operand planes: bf16 values that are exact (identity-aligned, unrotated
  // source rows; unrotated native rows) need no lo plane
  int planes_z[2], planes_y[2];
  for (int kv = 0; kv < 2; ++kv) {
    const bool bf = f->dtype == KVX_BF16;
    planes_z[kv] = bf && identity && (kv == 1 || !f->src_rope) ? 1 : 2;
    planes_y[kv] = bf && (kv == 1 || !f->tgt_rope) ? 1 : 2;
  }
  const char* tenv = std::getenv("KVX_FIT_TIMING");
  const bool timing = tenv && tenv[0] == '1';

  int64_t row_base = 0;
  for (int64_t b0 = 0; b0 < B; b0 += kFitBatch) {
    const int nb = static_cast<int>(std::min<int64_t>(kFitBatch, B - b0));
    FitCtx ctx{};
    ctx.n = nb;
    int32_t r = 0;
    for (int i = 0; i < nb; ++i) {
      ctx.row0[i] = r;
      ctx.csr0[i] = static_cast<int32_t>(row_base);
      r += tt[b0 + i];
      row_base += tt[b0 + i];
    }
    ctx.row0[nb] = r;
    if (r == 0) continue;
    const int32_t rp = static_cast<int32_t>(round_up(r, kPrepRows));
    // layer groups sized so the prepared operands fit in 1 GiB
    const size_t per_layer = size_t(2) * 2 * f->F2 * rp * sizeof(bf16_t);
    const int64_t lg = std::max<int64_t>(1, std::min<int64_t>(Lt, (size_t(1) << 30) / per_layer));
    const size_t need = per_layer * lg;
    if (need > f->prep_bytes) {
      if (f->prep) {
        FIT_HIP(hipStreamSynchronize(st));
        FIT_HIP(hipFree(f->prep));
        f->prep = nullptr;
        f->prep_bytes = 0;
      }
      FIT_HIP(hipMalloc(&f->prep, need));
      f->prep_bytes = need;
    }
    const Strides ss{io.src_stride[0], io.src_stride[1], io.src_stride[2], io.src_stride[3]};
    const Strides ts{io.tgt_stride[0], io.tgt_stride[1], io.tgt_stride[2], io.tgt_stride[3]};
    for (int64_t l0 = 0; l0 < Lt; l0 += lg) {
      const int nl = static_cast<int>(std::min<int64_t>(lg, Lt - l0));
      PrepArgs pa{};
      pa.src[0] = static_cast<const char*>(io.src_k) + b0 * io.src_stride[1] * esz;
      pa.src[1] = static_cast<const char*>(io.src_v) + b0 * io.src_stride[1] * esz;
      pa.ss = ss;
      pa.tgt[0] = static_cast<const char*>(io.tgt_k) + b0 * io.tgt_stride[1] * esz;
      pa.tgt[1] = static_cast<const char*>(io.tgt_v) + b0 * io.tgt_stride[1] * esz;
      pa.ts = ts;
      pa.row_ptr = identity ? nullptr : io.row_ptr;
      pa.col_idx = io.col_idx;
      pa.weight = io.weight;
      pa.layer_map = f->layer_map;
      pa.fs = f->fs;
      pa.ft = f->ft;
      pa.mix = f->mix;
      pa.hs = static_cast<int32_t>(Hs);
      pa.ds = static_cast<int32_t>(Ds);
      pa.ht = static_cast<int32_t>(Ht);
      pa.dt = static_cast<int32_t>(Dt);
      pa.din = f->din;
      pa.dout = f->dout;
      pa.din_z = f->din_z;
      pa.dout_p = f->dout_p;
      pa.F2 = f->F2;
      pa.rp = rp;
      pa.nrows = r;
      pa.l0 = static_cast<int32_t>(l0);
      pa.tz = (f->din / 2 + 63) / 64;
      pa.ty = (f->dout / 2 + 63) / 64;
      for (int kv = 0; kv < 2; ++kv) {
        pa.pz[kv] = planes_z[kv];
        pa.py[kv] = planes_y[kv];
      }
      pa.src_rope = f->src_rope;
      pa.tgt_rope = f->tgt_rope;
      pa.vec = vec ? 1 : 0;
      pa.xt = static_cast<bf16_t*>(f->prep);
      pa.acc = f->acc;
      pa.din_p = f->din_p;
      pa.F = f->F;
      pa.sys0 = static_cast<int32_t>(l0 * 2);
      pa.fit_bias = f->fit_bias;
      pa.ctx = ctx;
      const int npad = (f->din_z - f->din) + (f->dout_p - f->dout);
      const int rows_wg = kPrepRows * kPrepBlocks;
      const dim3 pg(pa.tz + pa.ty + (npad + 127) / 128, (rp + rows_wg - 1) / rows_wg, nl * 2);
      if (f->dtype == KVX_F32)
        fit_prepare<float><<<pg, dim3(256), 0, st>>>(pa);
      else
        fit_prepare<bf16_t><<<pg, dim3(256), 0, st>>>(pa);
      FIT_HIP(hipGetLastError());
      GramArgs ga{};
      ga.xt = static_cast<const bf16_t*>(f->prep);
      ga.acc = f->acc;
      ga.F2 = f->F2;
      ga.rp = rp;
      ga.nbi = f->din_z / kFB;
      ga.nbj = f->F2 / kFB;
      ga.din_z = f->din_z;
      ga.din_p = f->din_p;
      ga.F = f->F;
      for (int kv = 0; kv < 2; ++kv) {
        ga.pz[kv] = planes_z[kv];
        ga.py[kv] = planes_y[kv];
      }
      ga.sys0 = static_cast<int32_t>(l0 * 2);
      int nblk = 0;
      for (int bi = 0; bi < ga.nbi; ++bi) nblk += ga.nbj - bi;
      ga.nblk = nblk;
      hipEvent_t ev[2] = {nullptr, nullptr};
      if (timing) {
        FIT_HIP(hipEventCreate(&ev[0]));
        FIT_HIP(hipEventCreate(&ev[1]));
        FIT_HIP(hipEventRecord(ev[0], st));
      }
      // one launch for the K systems and one for the V systems of the group,
      // each instantiated for its operands' planes
      for (int kv = 0; kv < 2; ++kv) {
        const dim3 gg(nblk * nl);
        const int pz = planes_z[kv], py = planes_y[kv];
        if (pz == 2 && py == 2)
          fit_gram<2, 2><<<gg, dim3(256), 0, st>>>(ga, kv);
        else if (pz == 2)
          fit_gram<2, 1><<<gg, dim3(256), 0, st>>>(ga, kv);
        else if (py == 2)
          fit_gram<1, 2><<<gg, dim3(256), 0, st>>>(ga, kv);
        else
          fit_gram<1, 1><<<gg, dim3(256), 0, st>>>(ga, kv);
        FIT_HIP(hipGetLastError());
      }
      if (timing) {
        FIT_HIP(hipEventRecord(ev[1], st));
        f->timed.emplace_back(ev[0], ev[1]);
      }
    }
  }
  f->rows += rows;
  return KVX_OK;
}

kvx_status kvx_fit_solve(kvx_fit* f, double lambda, float* w_k, float* w_v, float* b_k,
                         float* b_v, void* stream) {
  if (!f || !w_k || !w_v || !std::isfinite(lambda) || lambda < 0) return KVX_EINVAL;
  if (f->fit_bias && (!b_k || !b_v)) return KVX_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t nsys = int64_t(f->tgt.n_layers) * 2;
  const int32_t np = static_cast<int32_t>(round_up(f->n, kSB));
  const size_t abytes = size_t(nsys) * np * np * sizeof(double);
  const size_t xbytes = size_t(nsys) * np * f->dout * sizeof(double);
  const size_t need = abytes + xbytes + 256;
  if (need > f->solve_bytes) {
    if (f->solve_buf) {
      FIT_HIP(hipStreamSynchronize(st));
      FIT_HIP(hipFree(f->solve_buf));
      f->solve_buf = nullptr;
      f->solve_bytes = 0;
    }
    FIT_HIP(hipMalloc(&f->solve_buf, need));
    f->solve_bytes = need;
  }
  char* base = static_cast<char*>(f->solve_buf);
  int32_t* status = reinterpret_cast<int32_t*>(base + abytes + xbytes);
  clear_status<<<dim3(1), dim3(64), 0, st>>>(status);
  FIT_HIP(hipGetLastError());
  SolveArgs sa{};
  sa.acc = f->acc;
  sa.A = reinterpret_cast<double*>(base);
  sa.X = reinterpret_cast<double*>(base + abytes);
  sa.sys0 = 0;
  sa.w[0] = w_k;
  sa.w[1] = w_v;
  sa.b[0] = b_k;
  sa.b[1] = b_v;
  sa.status = status;
  sa.lam = lambda;
  sa.n = f->n;
  sa.din = f->din;
  sa.dout = f->dout;
  sa.din_p = f->din_p;
  sa.F = f->F;
  sa.fit_bias = f->fit_bias;
  sa.np = np;
  const kvx_status es = enqueue_solve(sa, static_cast<int>(nsys), st);
  if (es != KVX_OK) return es;
  int32_t h = 0;
  FIT_HIP(hipMemcpyAsync(&h, status, sizeof h, hipMemcpyDeviceToHost, st));
  FIT_HIP(hipStreamSynchronize(st));
  return h ? KVX_EDATA : KVX_OK;
}

kvx_status kvx_fit_solve_noalloc(kvx_fit* f, double lambda, float* w_k, float* w_v, float* b_k,
                                 float* b_v, void* stream) {
  if (!f || !w_k || !w_v || !std::isfinite(lambda) || lambda < 0) return KVX_EINVAL;
  if (f->fit_bias && (!b_k || !b_v)) return KVX_EINVAL;
  int dev = 0;
  FIT_HIP(hipGetDevice(&dev));
  if (dev != f->device) return KVX_EINVAL;
  const int32_t np = static_cast<int32_t>(round_up(f->n, kSB));
  const size_t per_sys = (size_t(np) * np + size_t(np) * f->dout) * sizeof(double);
  const int64_t group = int64_t((kSolveWorkspaceBytes - kStatusBytes) / per_sys);
  if (group < 1) return KVX_EUNSUPPORTED;
  void* ws = nullptr;
  const kvx_status s = solve_workspace(&ws);
  if (s != KVX_OK) return s;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t nsys = int64_t(f->tgt.n_layers) * 2;
  const int64_t g = std::min(group, nsys);
  char* base = static_cast<char*>(ws);
  int32_t* status = reinterpret_cast<int32_t*>(base + kSolveWorkspaceBytes - kStatusBytes);
  clear_status<<<dim3(1), dim3(64), 0, st>>>(status);
  FIT_HIP(hipGetLastError());
  SolveArgs sa{};
  sa.acc = f->acc;
  sa.A = reinterpret_cast<double*>(base);
  sa.X = reinterpret_cast<double*>(base + size_t(g) * np * np * sizeof(double));
  sa.w[0] = w_k;
  sa.w[1] = w_v;
  sa.b[0] = b_k;
  sa.b[1] = b_v;
  sa.status = status;
  sa.lam = lambda;
  sa.n = f->n;
  sa.din = f->din;
  sa.dout = f->dout;
  sa.din_p = f->din_p;
  sa.F = f->F;
  sa.fit_bias = f->fit_bias;
  sa.np = np;
  // groups of systems in stream order reuse the same workspace
  for (int64_t s0 = 0; s0 < nsys; s0 += g) {
    sa.sys0 = static_cast<int32_t>(s0);
    const kvx_status es = enqueue_solve(sa, static_cast<int>(std::min(g, nsys - s0)), st);
    if (es != KVX_OK) return es;
  }
  int32_t h = 0;
  FIT_HIP(hipMemcpyAsync(&h, status, sizeof h, hipMemcpyDeviceToHost, st));
  FIT_HIP(hipStreamSynchronize(st));
  return h ? KVX_EDATA : KVX_OK;
}

kvx_status kvx_fit_reset(kvx_fit* f, void* stream) {
  if (!f) return KVX_EINVAL;
  const size_t ab = size_t(f->tgt.n_layers) * 2 * f->din_p * f->F * sizeof(float);
  FIT_HIP(hipMemsetAsync(f->acc, 0, ab, static_cast<hipStream_t>(stream)));
  f->rows = 0;
  return KVX_OK;
}

int64_t kvx_fit_rows(const kvx_fit* f) { return f ? f->rows : 0; }

kvx_status kvx_fit_query(kvx_fit* f, kvx_fit_info* info) {
  if (!f || !info) return KVX_EINVAL;
  *info = kvx_fit_info{};
  info->systems = 2 * f->tgt.n_layers;
  info->n = f->n;
  const int nbi = f->din_z / kFB, nbj = f->F2 / kFB;
  for (int bi = 0; bi < nbi; ++bi) info->gram_blocks += nbj - bi;
  info->rows = f->rows;
  info->device_bytes = static_cast<int64_t>(size_t(f->tgt.n_layers) * 2 * f->din_p * f->F *
                                            sizeof(float) + f->prep_bytes + f->solve_bytes);
  double ms = 0.0;
  kvx_status rc = KVX_OK;
  for (auto& p : f->timed) {
    float t = 0.f;
    hipError_t e = hipEventSynchronize(p.second);
    if (e == hipSuccess) e = hipEventElapsedTime(&t, p.first, p.second);
    if (e != hipSuccess) rc = fit_hip_fail(e);
    ms += t;
    (void)hipEventDestroy(p.first);
    (void)hipEventDestroy(p.second);
  }
  info->gram_launches = static_cast<int32_t>(f->timed.size());
  info->gram_ms = ms;
  f->timed.clear();
  return rc;
}

void kvx_fit_destroy(kvx_fit* f) {
  if (!f) return;
  for (auto& p : f->timed) {
    (void)hipEventDestroy(p.first);
    (void)hipEventDestroy(p.second);
  }
  if (f->layer_map) (void)hipFree(f->layer_map);
  if (f->fs) (void)hipFree(f->fs);
  if (f->ft) (void)hipFree(f->ft);
  if (f->acc) (void)hipFree(f->acc);
  if (f->prep) (void)hipFree(f->prep);
  if (f->solve_buf) (void)hipFree(f->solve_buf);
  delete f;
}

}  // extern "C"
