/*
 * kvx_fit.h -- fitting the per-layer affine translator of kvx.h from paired
 * KV caches (gfx950 / MI355X).
 *
 * Section 5 of the paper learns the translator T_theta by minimising a
 * representation distance D(T_theta(KV_A(C)), KV_B(C)) between translated
 * caches and caches the target model prefilled itself; Section 2.2 recalls
 * closed-form linear maps between the caches of two models.  For the affine
 * translator of kvx.h (u = W z + b, target RoPE after it), D the squared
 * Frobenius distance over the cache and a ridge penalty lam * ||W||_F^2 (the
 * bias is not penalised), the minimiser for each (target layer, K|V) solves
 * the normal equations
 *
 *     (Zt^T Zt + lam D) [W b]^T = Zt^T Y,    Zt = [Z 1],  D = diag(1, ..., 1, 0)
 *
 * where row t of Z is the pooled, source-de-rotated row z_t of the
 * translation (kvx.h, steps 1-2, same layer map and mixing) and row t of Y is
 * the native target row de-rotated by the target RoPE at position t (K) or
 * the native row itself (V).  RoPE is a rotation, so the distance over the
 * cache equals the distance before the target rotation.
 *
 * Work split: kvx_fit_accumulate forms Z and Y on the device and adds
 * Zt^T [Zt Y] into fp32 accumulators held by the fit (matrix cores; operands
 * that are not exact bf16 values are split into two bf16 terms: relative
 * product error about 2^-16);
 * kvx_fit_solve factors each system in fp64 (Cholesky) and writes W and b.
 * Calls are stream-ordered; everything runs in HIP kernels.
 */
#ifndef KVX_FIT_H
#define KVX_FIT_H

#include <stdint.h>

#include "kvx.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Geometry of the translator to fit; consumed by kvx_fit_create. */
typedef struct {
  kvx_model src;             /* as in kvx_plan_desc (inv_freq copied) */
  kvx_model tgt;
  int32_t mix;               /* source layers concatenated per target layer, >= 1 */
  const int32_t* layer_map;  /* host [tgt.n_layers * mix] */
  int32_t dtype;             /* kvx_dtype of the KV caches passed to accumulate */
  int32_t fit_bias;          /* 1: fit b (unpenalised); 0: b = 0 */
} kvx_fit_desc;

/* One batch of paired caches.  Layout, strides and alignment exactly as in
 * the kvx_io struct, all-zero strides meaning contiguous; tgt_k / tgt_v are
 * the native target caches [Lt][B][Ht][tgt_capacity][Dt] and are only read.
 * Rows t >= T_t[b] are ignored. */
typedef struct {
  int32_t batch;
  int32_t src_tokens;
  const void* src_k;         /* device [Ls][B][Hs][T_s][Ds] */
  const void* src_v;
  int64_t src_stride[4];
  const int32_t* tgt_tokens; /* host [B]; NULL = identity alignment */
  const int32_t* row_ptr;    /* device [R+1] */
  const int32_t* col_idx;    /* device [nnz] */
  const float* weight;       /* device [nnz] */
  const void* tgt_k;         /* device [Lt][B][Ht][tgt_capacity][Dt] */
  const void* tgt_v;
  int64_t tgt_stride[4];
  int32_t tgt_capacity;
} kvx_fit_io;

typedef struct kvx_fit kvx_fit;

/* Allocate the fp32 accumulators (zeroed) and copy the layer map and RoPE
 * tables (synchronous, current HIP device).  Errors: KVX_EINVAL, KVX_ESHAPE,
 * KVX_EUNSUPPORTED (a head_dim that is not a multiple of 16), KVX_ENOMEM,
 * KVX_EHIP; *out = NULL then. */
kvx_status kvx_fit_create(const kvx_fit_desc* desc, kvx_fit** out);

/* Add one batch of paired caches to the accumulators (asynchronous on
 * `stream`; buffers are borrowed until the stream work completes).  Host
 * arguments are validated before anything is enqueued; CSR contents are
 * trusted.  May grow the fit's device scratch (hipMalloc), so it is not for
 * graph capture.  batch == 0 or zero rows is a no-op. */
kvx_status kvx_fit_accumulate(kvx_fit* fit, const kvx_fit_io* io, void* stream);

/* Solve every (layer, K|V) system with ridge `lambda` >= 0 and write device
 * fp32 outputs: w_k, w_v [Lt][Ht*Dt][mix*Hs*Ds] (nn.Linear order, directly
 * usable as kvx_plan_desc weights after a cast to the plan's dtype) and b_k,
 * b_v [Lt][Ht*Dt] (zeros when fit_bias == 0; may be NULL then).  The
 * accumulators are kept, so more batches may follow.  KVX_EDATA if a system
 * is not positive definite (too few rows for lambda == 0, or lambda < 0);
 * the outputs are then unspecified.  Synchronises `stream` (it reads a
 * device status flag back). */
kvx_status kvx_fit_solve(kvx_fit* fit, double lambda, float* w_k, float* w_v, float* b_k,
                         float* b_v, void* stream);

/* kvx_fit_solve for callers that cannot allocate device memory (code that
 * must not call hipMalloc: serving loops, harnesses that forbid allocation):
 * the same solve, with the same results, that allocates nothing.  Its fp64
 * workspace is a 128 MiB static device array of the library, which every
 * device the library is loaded on holds until the process ends; systems are
 * solved in groups that fit it, in stream order.  Limit: one system's
 * (n^2 + n*dout) doubles, n = mix*Hs*Ds + fit_bias, must fit in the workspace
 * (n up to 3840 at dout 512), else KVX_EUNSUPPORTED with nothing
 * enqueued.  The current device must be the fit's (KVX_EINVAL otherwise).
 * Every call on a device shares that device's workspace: calls that overlap
 * on one device (other streams, other threads) race and must be serialised
 * by the caller.  Synchronises `stream`, as kvx_fit_solve. */
kvx_status kvx_fit_solve_noalloc(kvx_fit* fit, double lambda, float* w_k, float* w_v,
                                 float* b_k, float* b_v, void* stream);

/* Zero the accumulators (asynchronous). */
kvx_status kvx_fit_reset(kvx_fit* fit, void* stream);

/* Rows accumulated so far (host count). */
int64_t kvx_fit_rows(const kvx_fit* fit);

/* Diagnostics of a fit.  With the environment variable KVX_FIT_TIMING=1 at
 * accumulate time, every Gram pass (the K-system and the V-system launch of
 * one group of target layers, back to back) is bracketed by HIP events on its
 * stream; kvx_fit_query then waits for them and reports their summed
 * duration (and releases them). */
typedef struct {
  int32_t systems;        /* (target layer, K|V) systems = 2 * Lt */
  int32_t n;              /* unknowns per output column: din + fit_bias */
  int32_t gram_blocks;    /* 128 x 128 accumulator blocks per system */
  int32_t gram_launches;  /* timed Gram passes since the last query */
  int64_t rows;           /* rows accumulated since create / reset */
  int64_t device_bytes;   /* accumulators and scratch currently held */
  double gram_ms;         /* summed duration of the timed Gram passes, ms */
} kvx_fit_info;

kvx_status kvx_fit_query(kvx_fit* fit, kvx_fit_info* info);

/* Release (NULL-safe); no fit work may still be running. */
void kvx_fit_destroy(kvx_fit* fit);

#ifdef __cplusplus
}
#endif
#endif /* KVX_FIT_H */
