// kernel_mfma.h -- fused bf16 translation kernel on the gfx950 matrix cores.
//
// Work unit ("tile"): (target layer l, K|V, 128 target rows of one context,
// 256 output features).  The kernel is persistent: one workgroup per compute
// unit, each XCD owning a contiguous range of tiles (so the weights of a
// layer stay in that XCD's L2) that its workgroups take either in contiguous
// pieces or round-robin (decode_tile), and its 8 waves run in two roles over
// the concatenated sequence of K-chunks of all its tiles:
//
//   producers (waves 0-3)  gather 16-byte pieces of the source rows named by
//       the alignment entries of each target row, undo the source RoPE at
//       each source position (fp64-reduced angle), pool with the entry
//       weights in fp32, and write the chunk into one of two LDS buffers as
//       bf16 -- as hi = bf16(z), lo = bf16(z - hi) when the operand is a
//       computed value and the plan asks for the split.  Raw source data is
//       prefetched a chunk ahead, across tile boundaries.
//   consumers (waves 4-7)  contract the chunk on v_mfma_f32_32x32x16_bf16:
//       weight fragments (pre-packed at plan time, one contiguous 1 KiB load
//       each) straight from global memory, token fragments from LDS; the
//       accumulators hold U^T = W Z^T (rows = output features, columns =
//       tokens).  After a tile's last chunk they add the bias, apply the
//       target RoPE to K, round to bf16 and store 8-byte pieces of target
//       rows directly from registers.
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

// Lambdas in kernels must be inlined: an outlined call spills its captured
// state to the stack.
#define KVX_INLINE __attribute__((always_inline))

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
  const bf16x8* wp[2];      // packed bf16 fragments [Lt][dout/32][din/16][64 lanes]
  const bf16x8* wh[2];      // the same as fp16 bit patterns (precision mode F16)
  const float* bias[2];     // [Lt][dout]
  const int32_t* layer_map; // [Lt][mix]
  int32_t mix, hs, ds, ht, dt, din, dout, lt;
  const double* fs;         // [ds/2] source theta_i / 2pi
  const double* ft;         // [dt/2] target theta_i / 2pi
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const float* weight;
  int32_t n_tiles;          // N tiles per (layer, K|V)
  int32_t row_tiles;        // row tiles of this launch (all contexts)
  int32_t total_tiles;      // row_tiles * n_tiles * 2 * Lt
  int32_t interleave;       // tile order and assignment (decode_tile); selects the variant
  const bf16_t* zsink;      // kSinkBytes of zeros: source of lanes without data
  bf16_t* trash;            // kSinkBytes never read: target of lanes without a row
  Paging pg;                // optional paged target layout
  // split table of precision BF16X2_OUTLIER: bit ks of entry
  // (l * 2 + kv) * (din / 128) + c marks k-step ks of chunk c as split;
  // NULL: every k-step of a computed operand is split
  const uint8_t* split_mask;
  BatchArgs ba;
};

// Size of each of the two sink areas: covers the second member of a pair
// group (Ds/2 + 8 elements) for Ds <= 2*kMaxHalfDim, and one 16-byte store.
constexpr int kSinkBytes = 2048;

constexpr int fused_lds_bytes() { return 2 * 2 * kPlane * 2; }
constexpr int kMaxLayerMap = 1024;  // target layers * mix held in LDS
constexpr int kMaxHalfDim = 256;    // source head_dim / 2 held in LDS
constexpr int kDTab = 3;            // relative source rotations held in LDS: |d| <= 3
constexpr int kTabHalf = 64;        // ... for source head_dim <= 128

struct Tile {
  int l, kv, nt, b, t0, tt, rb, rt;
  int tau;  // linear tile index
};

// The launch's context table, copied to LDS at kernel start so the step
// loop can index it (a dynamic index into the kernel argument would make the
// compiler copy the whole argument block to scratch memory).
struct CtxTable {
  int32_t tile_start[kMaxBatch + 1];
  int32_t t_tgt[kMaxBatch];
  int32_t row_base[kMaxBatch];
};

// Two tile orders, chosen per launch (FusedArgs::interleave):
//  * contiguous (0): layer slowest, then row tile, then N tile, K|V fastest;
//    each workgroup walks a contiguous range, so it alternates K and V tiles
//    (balancing their different costs) and re-reads a row tile's source rows
//    for its N tiles while they are still in its XCD's L2.
//  * interleaved (1): layer slowest, then K|V, then row tile, N tile
//    fastest; each XCD's range is dealt round-robin to its workgroups, which
//    then run neighbouring tiles at the same time.  They share one layer's
//    K or V translator in the L2, which pays when a tile's weight slice is
//    large (long contractions), where contiguous ranges would put several
//    layers' translators in flight per XCD and re-read them from HBM.
__device__ __forceinline__ void tile_context(int n_ctx, const CtxTable& cx, Tile& T) {
  // uniform values: keep them in scalar registers
  int b = 0;
  while (b + 1 < n_ctx && __builtin_amdgcn_readfirstlane(cx.tile_start[b + 1]) <= T.rt) ++b;
  T.b = b;
  T.t0 = (T.rt - __builtin_amdgcn_readfirstlane(cx.tile_start[b])) * kMT;
  T.tt = __builtin_amdgcn_readfirstlane(cx.t_tgt[b]);
  T.rb = __builtin_amdgcn_readfirstlane(cx.row_base[b]);
}
__device__ __forceinline__ Tile decode_tile(int order, int tau, int n_tiles, int row_tiles,
                                            int n_ctx, const CtxTable& cx) {
  Tile T;
  T.tau = tau;
  if (order == 2) {
    // resident: layer slowest, then row tile, then K|V, N tile fastest
    T.nt = tau % n_tiles;
    int rest = tau / n_tiles;
    T.kv = rest & 1;
    rest >>= 1;
    T.rt = rest % row_tiles;
    T.l = rest / row_tiles;
  } else if (order == 1) {
    T.nt = tau % n_tiles;
    int rest = tau / n_tiles;
    T.rt = rest % row_tiles;
    rest /= row_tiles;
    T.kv = rest & 1;
    T.l = rest >> 1;
  } else {
    T.kv = tau & 1;
    int rest = tau >> 1;
    T.nt = rest % n_tiles;
    rest /= n_tiles;
    T.rt = rest % row_tiles;
    T.l = rest / row_tiles;
  }
  tile_context(n_ctx, cx, T);
  return T;
}
// The next tile of a contiguous range (resident order: N tile fastest, then
// K|V, then row tile).
__device__ __forceinline__ void advance_tile_res(int n_tiles, int row_tiles, int n_ctx,
                                                 const CtxTable& cx, Tile& T) {
  ++T.tau;
  if (++T.nt < n_tiles) return;
  T.nt = 0;
  if (T.kv == 0) {
    T.kv = 1;
    return;
  }
  T.kv = 0;
  if (++T.rt == row_tiles) {
    T.rt = 0;
    ++T.l;
  }
  tile_context(n_ctx, cx, T);
}
// The next tile of a contiguous range.
__device__ __forceinline__ void advance_tile(int n_tiles, int row_tiles, int n_ctx,
                                             const CtxTable& cx, Tile& T) {
  ++T.tau;
  if (T.kv == 0) {
    T.kv = 1;
    return;
  }
  T.kv = 0;
  if (++T.nt < n_tiles) return;
  T.nt = 0;
  if (++T.rt == row_tiles) {
    T.rt = 0;
    ++T.l;
  }
  tile_context(n_ctx, cx, T);
}
// Interleaved order: advance T by `step` tiles, given step = dr * n_tiles +
// dn (dn < n_tiles); scalar additions and carries only, no division.
__device__ __forceinline__ void step_tile(int dn, int dr, int n_tiles, int row_tiles, int n_ctx,
                                          const CtxTable& cx, Tile& T) {
  T.tau += dr * n_tiles + dn;
  T.nt += dn;
  int r = dr;
  if (T.nt >= n_tiles) {
    T.nt -= n_tiles;
    ++r;
  }
  int lk = 2 * T.l + T.kv;
  T.rt += r;
  while (T.rt >= row_tiles) {
    T.rt -= row_tiles;
    ++lk;
  }
  T.kv = lk & 1;
  T.l = lk >> 1;
  tile_context(n_ctx, cx, T);
}

// Workgroup barrier that orders LDS only: waits for this wave's LDS (and
// scalar-load) counters, not for its outstanding global loads, so prefetched
// data can stay in flight across steps.  The memory clobber keeps the
// compiler from moving memory accesses across it.  (__syncthreads() would
// also wait for every outstanding global load and store.)
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ void unpack8(const uint4 v, float* x) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = __uint_as_float(w[i] << 16);
    x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Streaming (non-temporal) 16-byte load and store: source KV rows are read
// once and target rows written once, so they should not displace the
// translator weights, which every tile of a layer re-reads, from the L2.
__device__ __forceinline__ uint4 ld_stream(const bf16_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
// Source row load: streaming when every source row is read by one tile only
// (one N tile, or the resident order), cached when several N tiles re-read it.
template <bool STREAM>
__device__ __forceinline__ uint4 ld_src(const bf16_t* p) {
  if constexpr (STREAM)
    return ld_stream(p);
  else
    return *reinterpret_cast<const uint4*>(p);
}
__device__ __forceinline__ void st_stream(bf16_t* p, const uint4 v) {
  u32x4 w;
  w.x = v.x;
  w.y = v.y;
  w.z = v.z;
  w.w = v.w;
  __builtin_nontemporal_store(w, reinterpret_cast<u32x4*>(p));
}

// Target row piece store of the span-map epilogue (paged layout).  Cached
// even when the source loads stream: the pieces of one 128-byte line come
// from several store instructions, which the L2 merges before writing back
// (measured with non-temporal stores: 1.45x the bytes written, 2x slower).
__device__ __forceinline__ void st_out(bf16_t* p, const u32x4 v) {
  *reinterpret_cast<u32x4*>(p) = v;
}

// Round 8 floats to bf16 (hardware round-to-nearest-even) and pack.
__device__ __forceinline__ uint4 pack8(const float* z) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bf16x2 p = {static_cast<__bf16>(z[2 * i]), static_cast<__bf16>(z[2 * i + 1])};
    o[i] = __builtin_bit_cast(uint32_t, p);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

typedef __attribute__((__vector_size__(2 * sizeof(_Float16)))) _Float16 f16x2;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;

// Round 8 floats to fp16 (hardware round-to-nearest-even) and pack.
__device__ __forceinline__ uint4 pack8_f16(const float* z) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f16x2 p = {static_cast<_Float16>(z[2 * i]), static_cast<_Float16>(z[2 * i + 1])};
    o[i] = __builtin_bit_cast(uint32_t, p);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

// Operand precision of computed operands (de-rotated K, pooled V).
enum Prec { kBF16X2 = 0, kBF16 = 1, kF16 = 2 };

__device__ __forceinline__ void residual8(const float* z, const uint4 hi, float* r) {
  float h[8];
  unpack8(hi, h);
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = z[i] - h[i];
}

// First members of an 8-pair group (8 consecutive pairs of the flattened
// (j, h, d) list) at token 0; second members at p + ds/2.
struct PairGroup {
  const bf16_t* p;
  int i0;  // frequency index of the first pair
};


// Alignment entries of the units of one producer thread within one tile.
struct RowInfo {
  int e0[kUnits], e1[kUnits], k0[kUnits];
  float w0[kUnits];
};

// Store pieces per producer thread and tile: the rows of thread `it` are
// it / 32 + 8 i, i < kRowsPerThread.
constexpr int kRowsPerThread = kMT * kNT / 8 / 256;

// Physical blocks of this thread's rows of tile Tc (paged layout), loaded a
// tile ahead of the stores (unconditional loads: rows past the context's end
// read the last row's entry).
template <bool PAGED>
__device__ __forceinline__ void load_blocks(const FusedArgs& a, const Tile& Tc, int it,
                                            int32_t (&blk)[kRowsPerThread]) {
  if constexpr (PAGED) {
#pragma unroll
    for (int i = 0; i < kRowsPerThread; ++i) {
      const int t = Tc.t0 + it / 32 + 8 * i;
      const int tc = t < Tc.tt ? t : Tc.tt - 1;
      blk[i] = a.pg.table[Tc.b * a.pg.max_blocks + tc / a.pg.block_size];
    }
  }
}

// Staging layout of a finished tile.  Producer thread `it` stores the
// 16-byte pieces (row r = it / 32 + 8 j, staged column group
// (it % 32) ^ stage_swz(r)), j < 16; piece j lives in the A-buffer slot that
// the same thread fills in its transform (plane j / 8, unit (j % 8) / 2,
// half j % 2).  A producer therefore reads all of its staged pieces before
// its next transform overwrites them, without any other thread touching them
// in between, and the stores can run in the step after the staging.  Staged
// column w*64 + p*32 + e holds feature c_p + e of pair block 4*nt + w.
// The swizzle, an XOR of the column group by row bits 1-2 (placed at column
// bits 3-4), spreads the 32 rows that one staging write of a consumer wave
// covers over the LDS banks: a half-wave of 8-byte writes then touches each
// bank it can reach at most twice, the least for writes that fill half of
// each 16-byte piece.  It leaves column bit 2 alone (the consumers' second
// 8-byte write goes to the piece owned by thread it + 4) and uses row bits
// 0-4 only (so the stores can form a thread's column groups once).  A store
// still covers whole rows, so its coalescing is unchanged.
__device__ __forceinline__ int stage_swz(int row) { return (row & 6) << 2; }

__device__ __forceinline__ int stage_slot(int it, int j) {
  return (j / 8) * kPlane + (it / 8 + 32 * ((j % 8) / 2)) * kLDA + 64 * (j % 2) + 8 * (it % 8);
}

// Whole 16-byte pieces of target rows from the staged tile Tc; thread `it`
// of 256.
template <bool PAGED>
__device__ __forceinline__ void store_rows(const FusedArgs& a, const Tile& Tc, const bf16_t* st,
                                           int it, const int32_t (&blk)[kRowsPerThread]) {
  const int npb = a.dout / 64;
  const int per_head = a.dt / 64;
  bf16_t* dst = a.tgt[Tc.kv] + Tc.l * a.ts.l;
  // Piece i of this thread is row r = it / 32 + 8 i of the tile, staged
  // column group (it % 32) ^ stage_swz(r).  stage_swz reads row bits 0-4
  // only, and r agrees with it / 32 + 8 (i % 4) there, so the column part of
  // the address takes at most four values, formed once.  A staged column
  // group lies within one target head (the pair block's 32 features and
  // their partners dt/2 further on).
  int64_t coff[4];
  bool con[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int sc8 = (it % 32) ^ stage_swz(it / 32 + 8 * q);  // staged column / 8
    const int pbw = Tc.nt * 4 + sc8 / 8;   // pair block of the owning consumer wave
    const int half = (sc8 / 4) % 2;
    const int hd = pbw / per_head;         // target head
    const int d = 32 * (pbw - hd * per_head) + half * (a.dt / 2) + (sc8 % 4) * 8;
    coff[q] = static_cast<int64_t>(hd) * a.ts.h + d;
    con[q] = pbw < npb;  // pair blocks past dout go to the trash area
  }
  const int r0 = it / 32;
  const int64_t row0 =
      static_cast<int64_t>(Tc.b) * a.ts.b + static_cast<int64_t>(Tc.t0 + r0) * a.ts.t;
#pragma unroll
  for (int i = 0; i < kRowsPerThread; ++i) {
    const int t = Tc.t0 + r0 + 8 * i;
    const int64_t row = PAGED ? static_cast<int64_t>(blk[i]) * a.ts.b +
                                    static_cast<int64_t>(t % a.pg.block_size) * a.ts.t
                              : row0 + static_cast<int64_t>(8 * i) * a.ts.t;
    bf16_t* q = dst + coff[i % 4] + row;
    // rows past the context's end go to the trash area too, so the store is
    // unconditional
    q = (t < Tc.tt && con[i % 4]) ? q : a.trash;
    st_stream(q, *reinterpret_cast<const uint4*>(st + stage_slot(it, i)));
  }
}

// IDENT: identity alignment.  CS_CACHE: the RoPE angles of a unit do not
// change across the chunks of a tile (identity alignment and Ds = 128, where
// every chunk is one head at the same frequencies), so they are computed once
// per tile.
//
// Step schedule.  Each tile takes nch chunk steps followed by one epilogue
// step; every step ends with a workgroup barrier and step s owns LDS buffer
// s % 2.  In a chunk step the consumers contract the buffer the producers
// filled during the previous step.  In the epilogue step the consumers stage
// the finished tile in their buffer while the producers fill the other
// buffer with the next tile's first chunk; the producers write the staged
// rows either after a mid-step barrier or at the start of the following
// step, each from its own slots, before its transform reuses them.
// Producers prefetch raw source data two or three chunks ahead into
// registers.
//
// PREC: how computed operands (de-rotated K, pooled V) reach the matrix
// cores -- split into two bf16 terms (kBF16X2), rounded once to bf16 (kBF16)
// or rounded once to fp16 and contracted against fp16 weights (kF16).  With
// identity alignment V is already bf16 and goes through unchanged, except in
// kF16 where every operand is fp16 (bf16 -> fp16 is exact in fp16's normal
// range) so the consumers run a single contraction type.
//
// STREAM: source rows are read with streaming loads (one N tile, so no tile
// re-reads them).  PAGED: target rows go through the block table.
template <bool IDENT, bool CS_CACHE, int PREC, bool STREAM, bool PAGED, int ORDER>
__global__ void __launch_bounds__(kThreads) fused_kernel(FusedArgs a) {
  // Identity alignment: the consumers stage a finished tile in LDS and the
  // producers store its rows in the step after.  Span maps: the consumers
  // store the rows straight from their accumulators (kDirect), so the LDS
  // buffers hold only operands -- which lets the resident order (ORDER 2)
  // keep a row tile's chunks in them for all of its N tiles.
  constexpr bool kDirect = !IDENT;
  constexpr bool RES = ORDER == 2;
  static_assert(!RES || kDirect, "the resident order needs direct stores");
  __shared__ __attribute__((aligned(16))) bf16_t lds[fused_lds_bytes() / 2];
  // layer map and source RoPE frequencies: per-lane lookups go to LDS, so no
  // vector load inside the step loop can queue behind outstanding stores
  __shared__ int32_t lmap[kMaxLayerMap];
  __shared__ double fsl[kMaxHalfDim];
  // span maps: cos / sin of the source rotation by d = -kDTab .. kDTab
  // positions, [d + kDTab][i] for i < kTabHalf (source head_dim <= 128)
  __shared__ float2 rotd[(2 * kDTab + 1) * kTabHalf];
  // target RoPE: theta_i / 2pi, and cos/sin of the rotation by 32 positions
  __shared__ double ftl[kMaxHalfDim];
  __shared__ float2 rot32[kMaxHalfDim];
  // bias of the tile being finished, in staging-column order (tile parity)
  __shared__ __attribute__((aligned(16))) float biasl[2][kNT];
  __shared__ CtxTable ctx;

  // Workgroups are dispatched to the 8 XCDs round-robin (block id mod 8).
  // Each XCD owns a contiguous range of tiles, in proportion to the
  // workgroups it holds.  Contiguous order: the range is split into one
  // contiguous piece per workgroup.  Interleaved order: it is dealt
  // round-robin, workgroup `slot` of the XCD taking tiles xbeg + slot,
  // xbeg + slot + nq, ...
  constexpr bool inter = ORDER == 1;  // a.interleave, as a template argument
  const int G = gridDim.x;
  const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
  const int nq = G / 8 + (xcd < G % 8 ? 1 : 0);          // workgroups on this XCD
  const int wfirst = xcd * (G / 8) + min(xcd, G % 8);     // and their rank in the grid
  auto part = [&](int w) KVX_INLINE {
    return static_cast<int>(static_cast<int64_t>(w) * a.total_tiles / G);
  };
  const int xbeg = part(wfirst), xend = part(wfirst + nq);
  const int tfirst = inter ? xbeg + slot : part(wfirst + slot);
  const int ntw = inter ? (slot < xend - xbeg ? (xend - xbeg - slot + nq - 1) / nq : 0)
                        : part(wfirst + slot + 1) - tfirst;  // tiles of this workgroup
  const int nch = a.din / 128;
  const int spt = nch + 1;            // steps per tile
  const int nchunks = ntw * nch;      // chunk steps of this workgroup
  const int nsteps = ntw * spt;
  if (nsteps == 0) return;
  const int tid = threadIdx.x;
  for (int i = tid; i < a.lt * a.mix; i += kThreads) lmap[i] = a.layer_map[i];
  for (int i = tid; i <= a.ba.n; i += kThreads) {
    ctx.tile_start[i] = a.ba.tile_start[i];
    if (i < a.ba.n) {
      ctx.t_tgt[i] = a.ba.t_tgt[i];
      ctx.row_base[i] = a.ba.row_base[i];
    }
  }
  const int n_tiles = a.n_tiles, row_tiles = a.row_tiles, n_ctx = a.ba.n;
  auto tile_at = [&](int tau) KVX_INLINE {
    return decode_tile(ORDER, tau, n_tiles, row_tiles, n_ctx, ctx);
  };
  // the workgroup's next tile (called only while one remains)
  const int step_dn = nq % n_tiles, step_dr = nq / n_tiles;
  auto next_tile = [&](Tile& T) KVX_INLINE {
    if constexpr (inter)
      step_tile(step_dn, step_dr, n_tiles, row_tiles, n_ctx, ctx, T);
    else if constexpr (RES)
      advance_tile_res(n_tiles, row_tiles, n_ctx, ctx, T);
    else
      advance_tile(n_tiles, row_tiles, n_ctx, ctx, T);
  };
  for (int i = tid; i < a.ds / 2; i += kThreads) fsl[i] = a.fs[i];
  const bool dtab = a.ds <= 2 * kTabHalf;
  if constexpr (!IDENT) {
    for (int i = tid; i < (2 * kDTab + 1) * kTabHalf; i += kThreads) {
      float c = 1.f, sn = 0.f;
      if (i % kTabHalf < a.ds / 2) rope_cs(a.fs[i % kTabHalf], i / kTabHalf - kDTab, c, sn);
      rotd[i] = make_float2(c, sn);
    }
  }
  for (int i = tid; i < a.dt / 2; i += kThreads) {
    ftl[i] = a.ft[i];
    float c, sn;
    rope_cs(a.ft[i], 32, c, sn);
    rot32[i] = make_float2(c, sn);
  }
  __syncthreads();

  if (tid < kProducers) {
    // =========================== producers ===========================
    const int g = tid % 8;  // 8-pair group within a chunk

    auto row_info = [&](const Tile& T, RowInfo& ri) KVX_INLINE {
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        const int t = T.t0 + tid / 8 + 32 * u;
        if (IDENT) {
          ri.e0[u] = 0;
          ri.e1[u] = t < T.tt ? 1 : 0;
          ri.k0[u] = t;
          ri.w0[u] = 1.f;
        } else {
          // unconditional loads: rows past the context's end read the last
          // row's pointers (a tile holds at least one row) and are then
          // emptied; empty rows read their first entry from the zero sink
          const int tc = t < T.tt ? t : T.tt - 1;
          const int e0 = a.row_ptr[T.rb + tc];
          int e1 = a.row_ptr[T.rb + tc + 1];
          e1 = t < T.tt ? e1 : e0;
          const bool any = e1 > e0;
          const int32_t* ci = any ? a.col_idx + e0 : reinterpret_cast<const int32_t*>(a.zsink);
          const float* wi = any ? a.weight + e0 : reinterpret_cast<const float*>(a.zsink);
          ri.e0[u] = e0;
          ri.e1[u] = e1;
          ri.k0[u] = *ci;
          ri.w0[u] = *wi;
        }
      }
    };

    // Raw first-entry data of a chunk (global chunk index cs) and the row
    // info it was fetched with.  With identity alignment three sets rotate
    // (cs mod 3), so two chunks stay in flight while one is transformed; the
    // span-map path (more registers per set: alignment entries) and the paged
    // path (block ids of the next tile) use two.
    constexpr int kDepth = IDENT && !PAGED ? 3 : 2;
    struct Raw {
      uint4 x0[kUnits], x1[kUnits];
      RowInfo ri;
    };
    Raw rA, rB, rC;
    // This thread's 8-pair group at chunk 0 of any tile: mixed layer j0,
    // source head h0, first frequency i00 (pair 8 g of the flattened list).
    const int half = a.ds / 2;
    const int hp0 = (8 * g) / half;
    const int j0 = hp0 / a.hs, h0 = hp0 % a.hs, i00 = (8 * g) % half;
    // Position of a chunk: its tile, chunk index in the tile, this thread's
    // group; advanced one chunk at a time (no divisions in the step loop).
    // ord: tile ordinal within this workgroup's range (resident order: of the
    // first tile of the chunk's row-tile group in the range)
    struct ChunkPos {
      Tile T;
      int c, j, h, i0, ord;
    };
    auto advance_pos = [&](ChunkPos& P) KVX_INLINE {
      if (++P.c == nch) {
        P.c = 0;
        if constexpr (RES) {
          // the next (layer, row tile, K|V) group: skip this group's other N tiles
          const int k = n_tiles - P.T.nt;
          P.ord += k;
          if (P.ord < ntw)
            for (int i = 0; i < k; ++i) next_tile(P.T);
        } else {
          ++P.ord;
          if (P.ord < ntw) next_tile(P.T);
        }
        P.j = j0;
        P.h = h0;
        P.i0 = i00;
        return;
      }
      P.i0 += 64;  // a chunk holds 64 pairs
      while (P.i0 >= half) {
        P.i0 -= half;
        if (++P.h == a.hs) {
          P.h = 0;
          ++P.j;
        }
      }
    };
    auto group_ptr = [&](const ChunkPos& P) KVX_INLINE -> const bf16_t* {
      const int ls = lmap[P.T.l * a.mix + P.j];
      return a.src[P.T.kv] + ls * a.ss.l + P.T.b * a.ss.b + P.h * a.ss.h + P.i0;
    };
    // chunks this workgroup's producers transform: one per chunk step, or, in
    // the resident order, nch per row-tile group its range touches
    const int nprod = RES ? (tile_at(tfirst).nt + ntw + n_tiles - 1) / n_tiles * nch : nchunks;
    ChunkPos fpos;
    fpos.T = tile_at(tfirst);
    fpos.c = 0;
    fpos.j = j0;
    fpos.h = h0;
    fpos.i0 = i00;
    fpos.ord = 0;
    ChunkPos tpos = fpos;  // transform position
    Tile ftile = fpos.T;
    RowInfo fri;
    const bf16_t* fgp = nullptr;
    // Address of the next chunk's first 8-pair group for this thread (and
    // the tile's row info); `more` false: no further chunk, the previous
    // address is returned (its loads read the zero sink).  Done before the
    // step's LDS writes: its LDS and scalar lookups then do not wait for
    // those writes to drain.
    auto fetch_addr = [&](bool more) KVX_INLINE -> const bf16_t* {
      if (more) {
        if (fpos.c == 0) {
          ftile = fpos.T;
          if (!IDENT) row_info(ftile, fri);
        }
        fgp = group_ptr(fpos);
        advance_pos(fpos);
      }
      return fgp;
    };
    // `more` false: there is no such chunk; the loads still issue (from the
    // zero sink), so every step issues the same loads.
    auto fetch_issue = [&](const bf16_t* gp, Raw& R, bool more) KVX_INLINE {
      if (!IDENT) R.ri = fri;
      PairGroup pg;
      pg.p = gp;
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        const int t = ftile.t0 + tid / 8 + 32 * u;  // identity: source token = t
        const bool any = more && (IDENT ? t < ftile.tt : fri.e1[u] > fri.e0[u]);
        // a unit without data reads zeros from the sink: the loads stay
        // unconditional, so the compiler can count them exactly
        const bf16_t* p = any ? pg.p + (IDENT ? t : fri.k0[u]) * a.ss.t : a.zsink;
        R.x0[u] = ld_src<STREAM>(p);
        R.x1[u] = ld_src<STREAM>(p + a.ds / 2);
      }
    };

    float csc[CS_CACHE ? kUnits : 1][8], css[CS_CACHE ? kUnits : 1][8];

    // Span map, contiguous target: second-entry data of the chunk at tpos
    // (the next one to be transformed), requested at the end of the previous
    // chunk's transform so that a whole step covers its latency.  (The paged
    // variant, which holds its block ids as well, reads second entries in
    // the transform like later ones: the prefetch would spill there.)
    constexpr bool kPrefetch2 = !IDENT && !PAGED;
    uint4 yb0[kPrefetch2 ? kUnits : 1], yb1[kPrefetch2 ? kUnits : 1];
    float ybw[kPrefetch2 ? kUnits : 1];  // its pooling weight (0: no second entry)
    int ybk[kPrefetch2 ? kUnits : 1];    // and source token
    auto second_issue = [&](const Raw& R, bool exists) KVX_INLINE {
      if constexpr (kPrefetch2) {
        const bf16_t* gp = group_ptr(tpos);
        // the second entries' tokens and weights are those of the tile:
        // (re)read at its first chunk only
        if (tpos.c == 0) {
#pragma unroll
          for (int u = 0; u < kUnits; ++u) {
            // unconditional loads from valid addresses: without a second
            // entry the token and weight come from the zero sink
            const bool two = R.ri.e1[u] - R.ri.e0[u] >= 2;
            const int32_t* ci = two ? a.col_idx + R.ri.e0[u] + 1
                                    : reinterpret_cast<const int32_t*>(a.zsink);
            const float* wi = two ? a.weight + R.ri.e0[u] + 1
                                  : reinterpret_cast<const float*>(a.zsink);
            ybk[u] = *ci;
            ybw[u] = *wi;
          }
        }
#pragma unroll
        for (int u = 0; u < kUnits; ++u) {
          const bool two = exists && R.ri.e1[u] - R.ri.e0[u] >= 2;
          const bf16_t* q = two ? gp + ybk[u] * a.ss.t : a.zsink;
          yb0[u] = ld_src<STREAM>(q);
          yb1[u] = ld_src<STREAM>(q + a.ds / 2);
        }
      }
    };

    // Transform the chunk at tpos (chunks are transformed in order).
    auto transform = [&](const Raw& R, bf16_t* hi, bf16_t* lo) KVX_INLINE {
      const Tile T = tpos.T;
      const int c = tpos.c;
      const bool is_k = T.kv == 0;
      if (IDENT && !is_k && PREC != kF16) {
        // identity-aligned V: the bf16 source rows are the operand
#pragma unroll
        for (int u = 0; u < kUnits; ++u) {
          const int r = tid / 8 + 32 * u;
          *reinterpret_cast<uint4*>(hi + r * kLDA + 8 * g) = R.x0[u];
          *reinterpret_cast<uint4*>(hi + r * kLDA + 64 + 8 * g) = R.x1[u];
        }
        advance_pos(tpos);
        return;
      }
      PairGroup pg;
      pg.p = group_ptr(tpos);
      pg.i0 = tpos.i0;
      double f[8];
      if (is_k && (!CS_CACHE || c == 0)) {
#pragma unroll
        for (int i = 0; i < 8; ++i) f[i] = fsl[pg.i0 + i];
      }
      if (CS_CACHE && is_k && c == 0) {
#pragma unroll
        for (int u = 0; u < kUnits; ++u)
#pragma unroll
          for (int i = 0; i < 8; ++i)
            rope_cs(f[i], T.t0 + tid / 8 + 32 * u, csc[u][i], css[u][i]);
      }
      // span maps: the token and weight of each row's third entry, when it
      // has one, requested before any row's arithmetic (the entry's data is
      // then requested in the row's turn without a dependent index load)
      int k3[kPrefetch2 ? kUnits : 1];
      float w3[kPrefetch2 ? kUnits : 1];
      if constexpr (kPrefetch2) {
#pragma unroll
        for (int u = 0; u < kUnits; ++u) {
          k3[u] = 0;
          w3[u] = 0.f;
          if (R.ri.e1[u] - R.ri.e0[u] >= 3) {
            k3[u] = a.col_idx[R.ri.e0[u] + 2];
            w3[u] = a.weight[R.ri.e0[u] + 2];
          }
        }
      }
#pragma unroll
      for (int u = 0; u < kUnits; ++u) {
        const int r = tid / 8 + 32 * u;
        float z0[8], z1[8];
        if constexpr (kPrefetch2) {
          // First two entries.  For K they are pooled in the first entry's
          // frame, R(-k0) (w0 x_k0 + w1 R(-(k1 - k0)) x_k1) -- equal to
          // w0 R(-k0) x_k0 + w1 R(-k1) x_k1 -- so only the first entry needs
          // a fresh fp64-reduced angle: the relative rotation of a nearby
          // second token (|k1 - k0| <= kDTab, as in spans) comes from the
          // rotd table; a farther one is formed like any other angle.  A row
          // without a second entry has zero data and weight (and d = 0).
          const int k0 = R.ri.k0[u];
          const float w0 = R.ri.w0[u], w1 = ybw[u];
          float x0[8], x1[8], v0[8], v1[8];
          unpack8(R.x0[u], x0);
          unpack8(R.x1[u], x1);
          unpack8(yb0[u], v0);
          unpack8(yb1[u], v1);
          if (is_k) {
            const int d = R.ri.e1[u] - R.ri.e0[u] >= 2 ? ybk[u] - k0 : 0;
            const bool tab = dtab && d >= -kDTab && d <= kDTab;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              float cd, sd;
              if (tab) {
                const float2 t = rotd[(d + kDTab) * kTabHalf + pg.i0 + i];
                cd = t.x;
                sd = t.y;
              } else {
                rope_cs(f[i], d, cd, sd);
              }
              const float y0 = w0 * x0[i] + w1 * (v0[i] * cd + v1[i] * sd);
              const float y1 = w0 * x1[i] + w1 * (v1[i] * cd - v0[i] * sd);
              float cs_, sn;
              rope_cs(f[i], k0, cs_, sn);
              z0[i] = y0 * cs_ + y1 * sn;
              z1[i] = y1 * cs_ - y0 * sn;
            }
          } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              z0[i] = w0 * x0[i] + w1 * v0[i];
              z1[i] = w0 * x1[i] + w1 * v1[i];
            }
          }
        } else {
          float x0[8], x1[8];
          unpack8(R.x0[u], x0);
          unpack8(R.x1[u], x1);
          const int k = IDENT ? T.t0 + r : R.ri.k0[u];
          const float w = IDENT ? 1.f : R.ri.w0[u];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            float y0 = x0[i], y1 = x1[i];
            if (is_k) {
              float cs_, sn;
              if (CS_CACHE) {
                cs_ = csc[u][i];
                sn = css[u][i];
              } else {
                rope_cs(f[i], k, cs_, sn);
              }
              y0 = x0[i] * cs_ + x1[i] * sn;
              y1 = x1[i] * cs_ - x0[i] * sn;
            }
            z0[i] = w * y0;
            z1[i] = w * y1;
          }
        }
        if constexpr (!IDENT) {
          for (int e = R.ri.e0[u] + (kPrefetch2 ? 2 : 1); e < R.ri.e1[u]; ++e) {
            const bool third = kPrefetch2 && e == R.ri.e0[u] + 2;
            const int k = third ? k3[kPrefetch2 ? u : 0] : a.col_idx[e];
            const float w = third ? w3[kPrefetch2 ? u : 0] : a.weight[e];
            const bf16_t* p = pg.p + k * a.ss.t;
            float x0[8], x1[8];
            unpack8(ld_src<STREAM>(p), x0);
            unpack8(ld_src<STREAM>(p + a.ds / 2), x1);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              float y0 = x0[i], y1 = x1[i];
              if (is_k) {
                float cs_, sn;
                rope_cs(f[i], k, cs_, sn);
                y0 = x0[i] * cs_ + x1[i] * sn;
                y1 = x1[i] * cs_ - x0[i] * sn;
              }
              z0[i] += w * y0;
              z1[i] += w * y1;
            }
          }
        }
        if (PREC == kF16) {
          *reinterpret_cast<uint4*>(hi + r * kLDA + 8 * g) = pack8_f16(z0);
          *reinterpret_cast<uint4*>(hi + r * kLDA + 64 + 8 * g) = pack8_f16(z1);
          continue;
        }
        const uint4 h0 = pack8(z0), h1 = pack8(z1);
        *reinterpret_cast<uint4*>(hi + r * kLDA + 8 * g) = h0;
        *reinterpret_cast<uint4*>(hi + r * kLDA + 64 + 8 * g) = h1;
        if (PREC == kBF16X2) {
          float d0[8], d1[8];
          residual8(z0, h0, d0);
          residual8(z1, h1, d1);
          *reinterpret_cast<uint4*>(lo + r * kLDA + 8 * g) = pack8(d0);
          *reinterpret_cast<uint4*>(lo + r * kLDA + 64 + 8 * g) = pack8(d1);
        }
      }
      advance_pos(tpos);
    };

    // chunk cs is consumed at step (its tile ordinal) * spt + (its index in the
    // tile) and written into that step's buffer during the step before.
    fetch_issue(fetch_addr(true), rA, true);
    fetch_issue(fetch_addr(nprod > 1), rB, nprod > 1);
    if constexpr (kDepth == 3) fetch_issue(fetch_addr(nprod > 2), rC, nprod > 2);
    {
      const bf16_t* gp = fetch_addr(nprod > kDepth);
      second_issue(rA, true);
      transform(rA, lds, lds + kPlane);
      second_issue(rB, nprod > 1);
      fetch_issue(gp, rA, nprod > kDepth);
    }
    lds_barrier();
    // Step s ends with a barrier; in an epilogue step (sc == nch) the
    // consumers stage the finished tile in buffer s % 2 and the producers
    // write its rows (the consumers issue no global stores, so their weight
    // loads never wait behind stores).
    int s = 0;
    int sc = 0;    // s % spt
    int sord = 0;  // s / spt: tile ordinal of step s
    // tile whose rows are stored next, and the physical blocks of its rows
    Tile stT = tile_at(tfirst);
    int st_ord = 0;
    int32_t blk[kRowsPerThread];
    if constexpr (!kDirect) load_blocks<PAGED>(a, stT, tid, blk);
    // Bias entry `tid` of a tile in staging-column order (consumer wave
    // tid / 64, block tid / 32 % 2, feature tid % 32); pair blocks past dout
    // read the zero sink.
    auto bias_entry = [&](const Tile& Tb) KVX_INLINE -> float {
      const int pb = Tb.nt * 4 + tid / 64;
      const int npb = a.dout / 64, per_head = a.dt / 64;
      const int f = (pb / per_head) * a.dt + 32 * (pb % per_head) + ((tid / 32) % 2) * (a.dt / 2) +
                    tid % 32;
      const float* q = pb < npb ? a.bias[Tb.kv] + static_cast<int64_t>(Tb.l) * a.dout + f
                                : reinterpret_cast<const float*>(a.zsink);
      return *q;
    };
    // tile 0's bias now; each later tile's is loaded during the previous
    // tile's epilogue step and written at the end of its own first step
    biasl[0][tid] = bias_entry(stT);
    // at the epilogue step of tile k, biasT becomes tile k + 1 (the last
    // tile repeats itself) and its bias is loaded
    Tile biasT = stT;
    int bias_ord = 0;
    float bias_next = 0.f;
    // Rows of tile stT staged in buffer sb, then the block ids of the next.
    auto store_tile = [&](int sb) KVX_INLINE {
      store_rows<PAGED>(a, stT, lds + sb * 2 * kPlane, tid, blk);
      if (++st_ord < ntw) next_tile(stT);
      load_blocks<PAGED>(a, stT, tid, blk);
    };
    auto end_step = [&]() KVX_INLINE {
      if (sc == 0 && s > 0) biasl[sord & 1][tid] = bias_next;
      if (sc == nch) {
        if (bias_ord + 1 < ntw) {
          next_tile(biasT);
          ++bias_ord;
        }
        bias_next = bias_entry(biasT);
      }
      lds_barrier();
      ++s;
      if (++sc == spt) {
        sc = 0;
        ++sord;
      }
      // identity alignment: the tile staged in step s - 1, before this
      // thread's transform of step s reuses the slots
      if constexpr (!kDirect)
        if (sc == 0) store_tile((s - 1) & 1);
    };
    // Step in which the chunk at P is written: the step before its first use
    // (step ord * spt + c, buffer s % 2) -- or, in the resident order, where
    // chunk c of a group lives in buffer c, the step after the previous
    // group's last use of buffer c.
    auto write_step = [&](const ChunkPos& P) KVX_INLINE -> int {
      if constexpr (RES)
        return P.ord == 0 ? P.c - 1 : (P.ord - 1) * spt + P.c + 1;
      else
        return P.ord * spt + P.c - 1;
    };
    // Transform the next chunk (the one at tpos, written at write_step) from
    // raw set R, and
    // refill R with the chunk kDepth further on.  Called with the sets in turn
    // (chunk mod kDepth), so each set keeps its registers.
    auto produce = [&](int next, Raw& R, const Raw& Rn) KVX_INLINE {
      while (s < write_step(tpos)) end_step();  // steps with nothing to transform
      bf16_t* buf = lds + (RES ? tpos.c : (s + 1) & 1) * 2 * kPlane;
      const bool more = next + kDepth < nprod;
      const bf16_t* gp = fetch_addr(more);
      transform(R, buf, buf + kPlane);
      second_issue(Rn, next + 1 < nprod);  // Rn: the chunk after this one
      fetch_issue(gp, R, more);
      end_step();
    };
    int next = 1;
    if constexpr (kDepth == 3) {
      for (; next + 2 < nprod; next += 3) {
        produce(next, rB, rC);
        produce(next + 1, rC, rA);
        produce(next + 2, rA, rB);
      }
      if (next < nprod) produce(next, rB, rC);
      if (next + 1 < nprod) produce(next + 1, rC, rA);
    } else {
      for (; next + 1 < nprod; next += 2) {
        produce(next, rB, rA);
        produce(next + 1, rA, rB);
      }
      if (next < nprod) produce(next, rB, rA);
    }
    while (s < nsteps) end_step();
    return;
  }

  // =========================== consumers ===========================
  const int lane = tid & 63;
  const int ct = tid - kProducers;        // consumer thread 0..255
  const int cw = ct >> 6;                 // consumer wave 0..3
  const int npb = a.dout / 64;
  const int per_head = a.dt / 64;
  const int KSALL = a.din / 16;
  const int trow = lane % 32;
  const int tcol = 8 * (lane / 32);
  const int fq = 4 * (lane / 32);

  // The consumer wave's pair block of a tile, kept compact (registers are
  // scarce): its index pb = 4 nt + wave and the weight fragment pointer of
  // its first 32 features c0 = hp Dt + 32 q (target head hp, block q of the
  // head); the RoPE partners c1 = c0 + Dt/2 lie w1off fragments further.  A
  // pair block past dout (on() false) points at block 0 and stores nothing.
  struct Blocks {
    int pb;
    const bf16x8* w0p;
  };
  auto b_on = [&](const Blocks& B) KVX_INLINE { return B.pb < npb; };
  auto b_hp = [&](const Blocks& B) KVX_INLINE { return B.pb < npb ? B.pb / per_head : 0; };
  auto b_q = [&](const Blocks& B) KVX_INLINE { return B.pb < npb ? B.pb % per_head : 0; };
  const int64_t w1off = static_cast<int64_t>(a.dt / 64) * KSALL * 64;
  // weight fragment pointer of block c0 for tile T's layer and K|V
  auto rebase = [&](Blocks& B, const Tile& T) KVX_INLINE {
    const bf16x8* wsel = PREC == kF16 ? a.wh[T.kv] : a.wp[T.kv];
    const bf16x8* base = wsel + static_cast<int64_t>(T.l) * (a.dout / 32) * KSALL * 64;
    const int c0 = b_hp(B) * a.dt + 32 * b_q(B);
    B.w0p = base + static_cast<int64_t>(c0 / 32) * KSALL * 64 + lane;
  };
  auto blocks = [&](const Tile& T, int w) KVX_INLINE {
    Blocks B;
    B.pb = T.nt * 4 + w;
    rebase(B, T);
    return B;
  };

  f32x16 acc[4][2];
  // weight fragments of k-steps ks .. ks + 3 (ring of four)
  bf16x8 wf[4][2];
  auto load_w = [&](const Blocks& B, int c) KVX_INLINE {
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      wf[ks][0] = B.w0p[(c * 8 + ks) * 64];
      wf[ks][1] = B.w0p[w1off + (c * 8 + ks) * 64];
    }
  };

  // Bias, target RoPE on K, bf16, into the staging slots (stage_slot):
  // lane holds, for token column lane%32 of token block m, the features
  // 8*(v/4) + 4*(lane/32) + v%4 (v < 16) of blocks c0 and c1; staged at
  // column cw*64 + p*32 + feature offset.  Bias comes from the tile's LDS
  // copy; the RoPE angle is formed in fp64 for token block 0 and advanced by
  // 32 positions per block with the rotation by 32 positions.
  auto stage = [&](const Tile& Tc, const Blocks& B, bf16_t* st, const float* bias_t) KVX_INLINE {
    const bool is_k = Tc.kv == 0;
    const float* bl = bias_t + cw * 64 + fq;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(bl + 8 * g4);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(bl + 32 + 8 * g4);
      float cs[4], sn[4], c32[4], s32[4];
      if (is_k) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int fi = 32 * b_q(B) + 8 * g4 + fq + i;
          rope_cs(ftl[fi], Tc.t0 + lane % 32, cs[i], sn[i]);
          const float2 r = rot32[fi];
          c32[i] = r.x;
          s32[i] = r.y;
        }
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int row = m * 32 + lane % 32;
        float u0[4], u1[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          u0[i] = acc[m][0][4 * g4 + i] + b0[i];
          u1[i] = acc[m][1][4 * g4 + i] + b1[i];
        }
        if (is_k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float y0 = u0[i] * cs[i] - u1[i] * sn[i];
            const float y1 = u1[i] * cs[i] + u0[i] * sn[i];
            u0[i] = y0;
            u1[i] = y1;
            // angle of token block m + 1
            const float c2 = cs[i] * c32[i] - sn[i] * s32[i];
            sn[i] = sn[i] * c32[i] + cs[i] * s32[i];
            cs[i] = c2;
          }
        }
        const bf16x2 p00 = {static_cast<__bf16>(u0[0]), static_cast<__bf16>(u0[1])};
        const bf16x2 p01 = {static_cast<__bf16>(u0[2]), static_cast<__bf16>(u0[3])};
        const bf16x2 p10 = {static_cast<__bf16>(u1[0]), static_cast<__bf16>(u1[1])};
        const bf16x2 p11 = {static_cast<__bf16>(u1[2]), static_cast<__bf16>(u1[3])};
        // staged columns cw*64 + p*32 + 8*g4 + fq .. +3 of this row (p = 1:
        // piece owner it + 4 -- the swizzle leaves bit 2 alone -- whose slot
        // is 32 elements further)
        bf16_t* sp = st + stage_slot((row % 8) * 32 + ((cw * 8 + g4) ^ stage_swz(row)), row / 8) + fq;
        *reinterpret_cast<uint2*>(sp) =
            make_uint2(__builtin_bit_cast(uint32_t, p00), __builtin_bit_cast(uint32_t, p01));
        *reinterpret_cast<uint2*>(sp + 32) =
            make_uint2(__builtin_bit_cast(uint32_t, p10), __builtin_bit_cast(uint32_t, p11));
      }
    }
  };

  // Span maps (kDirect): the epilogue of a tile -- bias, target RoPE on K,
  // bf16 -- with the rows stored straight from the accumulators.  A lane holds, for token column lane%32 of
  // token block m, the features 8*(v/4) + 4*(lane/32) + v%4 (v < 16) of
  // blocks c0 and c1.  For each pair of 8-feature groups (g4 = 2gp, 2gp+1),
  // v_permlane32_swap gives lane l the upper half of group 2gp from lane
  // l + 32 and lane l + 32 the lower half of group 2gp+1 from lane l, so each
  // lane then holds one 16-byte piece (8 consecutive features) of its row and
  // the two lanes of a row store adjacent pieces.  Bias comes from the tile's
  // LDS copy; the RoPE angle is formed in fp64 for token block 0 and advanced
  // by 32 positions per block with the rotation by 32 positions.  Lanes past
  // the context's end, and pair blocks past dout, store to the trash area, so
  // the stores stay unconditional.
  // Feature groups 2gp and 2gp + 1 of every token block (gp = 0, 1).
  auto finish = [&](const Tile& Tc, const Blocks& B, const float* bias_t,
                    const int32_t (&blk)[4], const int gp) KVX_INLINE {
    const bool is_k = Tc.kv == 0;
    const int half = lane / 32;
    const float* bl = bias_t + cw * 64 + fq;
    bf16_t* dst = a.tgt[Tc.kv] + Tc.l * a.ts.l + static_cast<int64_t>(b_hp(B)) * a.ts.h;
    const int col = 32 * b_q(B) + 8 * (2 * gp + half);
    // Contiguous layout: this context's rows of the head as a buffer resource
    // whose size ends at row T_t (zero for a pair block past dout), so the
    // hardware drops the stores of rows past the context's end; offsets are
    // 32-bit (the host keeps a context's rows below 2^31 bytes).
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        dst + (PAGED ? 0 : static_cast<int64_t>(Tc.b) * a.ts.b), static_cast<short>(0),
        b_on(B) && !PAGED ? static_cast<int>(static_cast<int64_t>(Tc.tt) * a.ts.t * 2) : 0,
        0x00020000);
    // packed bf16 pairs of group 2gp, [token block][block c0|c1][dword]
    uint32_t w0[4][2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int g4 = 2 * gp + h;
      const f32x4 b0 = *reinterpret_cast<const f32x4*>(bl + 8 * g4);
      const f32x4 b1 = *reinterpret_cast<const f32x4*>(bl + 32 + 8 * g4);
      float cs[4], sn[4], c32[4], s32[4];
      if (is_k) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int fi = 32 * b_q(B) + 8 * g4 + fq + i;
          rope_cs(ftl[fi], Tc.t0 + lane % 32, cs[i], sn[i]);
          const float2 r = rot32[fi];
          c32[i] = r.x;
          s32[i] = r.y;
        }
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        float u0[4], u1[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          u0[i] = acc[m][0][4 * g4 + i] + b0[i];
          u1[i] = acc[m][1][4 * g4 + i] + b1[i];
        }
        if (is_k) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float y0 = u0[i] * cs[i] - u1[i] * sn[i];
            const float y1 = u1[i] * cs[i] + u0[i] * sn[i];
            u0[i] = y0;
            u1[i] = y1;
            // angle of token block m + 1
            const float c2 = cs[i] * c32[i] - sn[i] * s32[i];
            sn[i] = sn[i] * c32[i] + cs[i] * s32[i];
            cs[i] = c2;
          }
        }
        uint32_t q[2][2];  // [block c0|c1][dword]
#pragma unroll
        for (int d = 0; d < 2; ++d) {
          const bf16x2 q0 = {static_cast<__bf16>(u0[2 * d]), static_cast<__bf16>(u0[2 * d + 1])};
          const bf16x2 q1 = {static_cast<__bf16>(u1[2 * d]), static_cast<__bf16>(u1[2 * d + 1])};
          q[0][d] = __builtin_bit_cast(uint32_t, q0);
          q[1][d] = __builtin_bit_cast(uint32_t, q1);
        }
        if (h == 0) {
#pragma unroll
          for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int d = 0; d < 2; ++d) w0[m][p][d] = q[p][d];
          continue;
        }
        // trade halves with the partner lane, then store one piece per block
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int d = 0; d < 2; ++d) {
            const auto r = __builtin_amdgcn_permlane32_swap(w0[m][p][d], q[p][d], false, false);
            w0[m][p][d] = r[0];
            q[p][d] = r[1];
          }
        const int t = Tc.t0 + m * 32 + lane % 32;
        const u32x4 v0 = {w0[m][0][0], w0[m][0][1], q[0][0], q[0][1]};
        const u32x4 v1 = {w0[m][1][0], w0[m][1][1], q[1][0], q[1][1]};
        if constexpr (PAGED) {
          const int64_t row = static_cast<int64_t>(blk[m]) * a.ts.b +
                              static_cast<int64_t>(t % a.pg.block_size) * a.ts.t;
          const bool ok = t < Tc.tt && b_on(B);
          st_out(ok ? dst + row + col : a.trash, v0);
          st_out(ok ? dst + row + col + a.dt / 2 : a.trash, v1);
        } else {
          const int off = (t * static_cast<int>(a.ts.t) + col) * 2;
          __builtin_amdgcn_raw_buffer_store_b128(v0, rs, off, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b128(v1, rs, off + a.dt, 0, 0);
        }
      }
    }
  };
  // Physical blocks of this lane's rows (token lane%32 of each token block)
  // of tile Tc, loaded when the consumers start the tile (unconditional
  // loads: rows past the context's end read the last row's entry).
  auto tile_blocks = [&](const Tile& Tc, int32_t (&blk)[4]) KVX_INLINE {
    if constexpr (PAGED) {
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const int t = Tc.t0 + m * 32 + lane % 32;
        const int tc = t < Tc.tt ? t : Tc.tt - 1;
        blk[m] = a.pg.table[Tc.b * a.pg.max_blocks + tc / a.pg.block_size];
      }
    }
  };

  Tile T = tile_at(tfirst);
  Blocks B = blocks(T, cw);
  Tile Tn = T;      // next tile (decoded in the step that loads its weights)
  Blocks Bn = B;
  int32_t cblk[4] = {0, 0, 0, 0};  // paged span maps: blocks of this lane's rows of T
  load_w(B, 0);  // valid addresses even for a pair block past dout
  lds_barrier();
  int cs = 0;    // global chunk index
  int c = 0;     // chunk within the tile; c == nch: epilogue step
  int tpar = 0;  // tile parity (bias buffer)
  for (int s = 0; s < nsteps; ++s) {
    // resident order: chunk c of a row-tile group stays in buffer c for all of
    // the group's N tiles
    bf16_t* buf = lds + (RES ? c : s & 1) * 2 * kPlane;
    if (c < nch) {
      // ---------------- chunk step ----------------
      const bool computed = T.kv == 0 || !IDENT;
      if constexpr (kDirect && PAGED)
        if (c == 0) tile_blocks(T, cblk);
      // k-steps of this chunk that take the split operand (a uniform load)
      const int kmask =
          PREC == kBF16X2 && a.split_mask ? a.split_mask[(T.l * 2 + T.kv) * nch + c] : 0xFF;
      // weights four k-steps ahead (k-steps 4..7 of this chunk, then 0..3 of
      // the next chunk, possibly of the next tile): a ring slot is reloaded
      // as soon as the MFMAs of its k-step have issued
      const bool more = cs + 1 < nchunks;
      const int cn = more && c + 1 < nch ? c + 1 : 0;
      if (c == 0) Bn = B;
      if (more && cn == 0) {
        Tn = T;
        next_tile(Tn);
        if (Tn.nt == (B.pb >> 2)) {
          Bn = B;
          rebase(Bn, Tn);
        } else {
          Bn = blocks(Tn, cw);
        }
      }
      // unconditional (past the last chunk, or for a pair block past dout, the
      // addresses are still valid fragments): the compiler then counts the
      // outstanding loads exactly instead of draining them all
      // (span maps: the last chunk of a tile leaves k-steps 0..3 of the next
      // tile to the end of the epilogue, whose direct stores need the
      // registers)
      const bool hold = false;
      auto reload = [&](int ks) KVX_INLINE {
        if (ks < 4) {
          wf[ks][0] = B.w0p[(c * 8 + ks + 4) * 64];
          wf[ks][1] = B.w0p[w1off + (c * 8 + ks + 4) * 64];
        } else if (!hold) {
          wf[ks - 4][0] = Bn.w0p[(cn * 8 + ks - 4) * 64];
          wf[ks - 4][1] = Bn.w0p[w1off + (cn * 8 + ks - 4) * 64];
        }
      };
      if (b_on(B)) {
        const bf16_t* hi = buf;
        const bf16_t* lo = buf + kPlane;
        // MFMA groups run in the order (k-step, plane): the token fragments of
        // group g + 1 are read before the MFMAs of group g issue, so the LDS
        // latency hides behind eight MFMAs; the scheduling barriers keep the
        // compiler from sinking the reads next to their first use.
        auto frag = [&](const bf16_t* plane, int ks, bf16x8 (&z)[4]) KVX_INLINE {
#pragma unroll
          for (int m = 0; m < 4; ++m)
            z[m] = *reinterpret_cast<const bf16x8*>(plane + (m * 32 + trow) * kLDA + ks * 16 + tcol);
        };
        // `fresh`: the tile's first MFMAs, which start from zero accumulators
        // (an inline-constant source, so no register clearing)
        auto mfma8 = [&](int ks, const bf16x8 (&z)[4], bool fresh) KVX_INLINE {
          const f32x16 zero = {};
#pragma unroll
          for (int m = 0; m < 4; ++m) {
#pragma unroll
            for (int p = 0; p < 2; ++p) {
              const f32x16 cin = fresh ? zero : acc[m][p];
              if (PREC == kF16)
                acc[m][p] = __builtin_amdgcn_mfma_f32_32x32x16_f16(
                    __builtin_bit_cast(f16x8, wf[ks % 4][p]), __builtin_bit_cast(f16x8, z[m]), cin,
                    0, 0, 0);
              else
                acc[m][p] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[ks % 4][p], z[m], cin, 0, 0, 0);
            }
          }
        };
        const bool split = PREC == kBF16X2 && computed;
        bf16x8 za[4], zb[4];
        frag(hi, 0, za);
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          // unsplit k-steps prefetch the next k-step's fragments into zb
          // (idle without a split) and move them to za after the group
          const bool split_ks = split && ((kmask >> ks) & 1);
          if (split_ks) frag(lo, ks, zb);
          else if (ks + 1 < 8) frag(hi, ks + 1, zb);
          __builtin_amdgcn_sched_barrier(0);
          if (ks == 0 && c == 0) mfma8(ks, za, true);
          else mfma8(ks, za, false);
          __builtin_amdgcn_sched_barrier(0);
          if (split_ks && ks + 1 < 8) frag(hi, ks + 1, za);
          __builtin_amdgcn_sched_barrier(0);
          if (split_ks) {
            mfma8(ks, zb, false);
          } else if (ks + 1 < 8) {
#pragma unroll
            for (int m = 0; m < 4; ++m) za[m] = zb[m];
          }
          reload(ks);
          __builtin_amdgcn_sched_barrier(0);
        }
      } else if (!hold) {
        load_w(Bn, cn);
      }
      ++cs;
      ++c;
      lds_barrier();
    } else {
      // ---------------- epilogue step ----------------
      if constexpr (kDirect) {
        finish(T, B, biasl[tpar], cblk, 0);
        finish(T, B, biasl[tpar], cblk, 1);
      } else {
        if (b_on(B)) stage(T, B, buf, biasl[tpar]);
      }
      lds_barrier();
      if (cs < nchunks) {
        T = Tn;
        B = Bn;
      }
      c = 0;
      tpar ^= 1;
    }
  }
}

}  // namespace kvx
