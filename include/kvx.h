/*
 * kvx.h -- C-ABI of the cross-model KV-translation library (gfx950 / MI355X).
 *
 * The operator turns a source model's per-layer KV cache for a context into
 * the KV cache of a different target model, so the target can decode without
 * its own prefill:  KV^_B(C) = T_{A->B}(KV_A(C))  (paper Section 4, the
 * translation operator), with T = T_theta a parameterised translator
 * (Section 5).  Translation may work per layer or on groups of layers and per
 * KV head (Section 5, granularity), and source and target may differ in
 * layers, heads, hidden size and tokenizer (Section 4).  Concretely, for target
 * layer l, context b, target token t:
 *
 *   x_k  = concat_{j<mix, h<Hs} R_src(-k) K_src[layer_map[l*mix+j]][b][h][k]
 *          (V: the same concatenation without the rotation)
 *   z_t  = sum_{e in row t} weight[e] * x_{col_idx[e]}     (identity: z_t = x_t)
 *   u    = W[l] z_t + bias[l]
 *   K_tgt[l][b][h][t] = R_tgt(+t) u[h*Dt : (h+1)*Dt],   V_tgt: u[h*Dt : (h+1)*Dt]
 *
 * R(p) is rotate-half RoPE: the pair (i, i + D/2) of a head vector turns by
 * p * theta_i, theta_i = base^(-2i/D).  Positions are 0-based within each
 * context.  The translator's learned parameters theta of Section 5 are W and
 * bias, one pair per target layer and per K/V.
 *
 * Everything of the translation runs in HIP kernels on the caller's stream;
 * the host side validates, sizes the launch and enqueues.
 */
#ifndef KVX_H
#define KVX_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes.  No function throws across the ABI. */
typedef enum {
  KVX_OK = 0,
  KVX_EINVAL = 1,       /* NULL or out-of-range argument */
  KVX_ESHAPE = 2,       /* inconsistent dimensions, strides or capacity */
  KVX_EUNSUPPORTED = 3, /* valid but not supported by this library (e.g. odd head_dim) */
  KVX_ENOMEM = 4,       /* device allocation failed */
  KVX_EHIP = 5,         /* a HIP runtime call failed; see kvx_last_hip_error() */
  KVX_EDATA = 6         /* device CSR contents invalid (validation mode only) */
} kvx_status;

/* Storage dtype of KV tensors and translator weights. */
typedef enum { KVX_F32 = 0, KVX_BF16 = 1 } kvx_dtype;

/* Precision of the matrix-core operands (bf16 plans only; ignored for f32).
 * A "computed" operand is one the translation produces before the projection:
 * RoPE-de-rotated K, and pooled V rows when the tokenizers differ.  Source V
 * with identity alignment is already bf16 and always goes through unchanged.
 *  KVX_PREC_BF16X2: computed operands are split a = hi + lo into two bf16
 *                   values and contracted twice against the bf16 W (relative
 *                   operand error about 2^-17; no range limit).  Default.
 *  KVX_PREC_BF16:   computed operands rounded once to bf16 (2^-9).
 *  KVX_PREC_F16:    computed operands rounded once to fp16 and contracted
 *                   against an fp16 copy of W (2^-12, one contraction).
 *                   Range limit: a computed operand of magnitude >= 65520
 *                   overflows and makes the affected outputs non-finite;
 *                   kvx_plan_create returns KVX_EUNSUPPORTED if a weight
 *                   exceeds the fp16 range.
 *  KVX_PREC_BF16X2_OUTLIER: mixed precision by channel, in the manner of
 *                   LLM.int8() (Dettmers et al., 2022), which keeps outlier
 *                   features at higher precision: the computed operands of
 *                   the 16-feature k-steps that hold a source channel marked
 *                   in kvx_plan_desc.outlier_k / outlier_v are split as in
 *                   BF16X2, all others are rounded once as in BF16.  K's
 *                   de-rotation mixes the two members of a RoPE pair, so a
 *                   marked K channel also marks its partner (d + Ds/2 mod Ds).
 *                   With every channel marked it is BF16X2, with none BF16.
 * Accumulation is fp32 in every mode. */
typedef enum {
  KVX_PREC_BF16X2 = 0,
  KVX_PREC_BF16 = 1,
  KVX_PREC_F16 = 2,
  KVX_PREC_BF16X2_OUTLIER = 3
} kvx_precision;

/* One side of the translation (a model's KV-cache geometry). */
typedef struct {
  int32_t n_layers;        /* transformer layers */
  int32_t n_kv_heads;      /* KV heads per layer */
  int32_t head_dim;        /* even */
  double rope_base;        /* RoPE base; <= 0 disables RoPE on this side */
  const double* inv_freq;  /* optional host [head_dim/2], overrides base^(-2i/D);
                              copied by kvx_plan_create */
} kvx_model;

/* Translator and geometry; consumed once by kvx_plan_create. */
typedef struct {
  kvx_model src;
  kvx_model tgt;
  int32_t mix;               /* source layers concatenated per target layer, >= 1 */
  const int32_t* layer_map;  /* host [tgt.n_layers * mix], source layer ids;
                                input feature (j*Hs + h)*Ds + d of target layer l
                                is source layer layer_map[l*mix+j], head h, dim d */
  int32_t dtype;             /* kvx_dtype of KV tensors and weights */
  const void* w_k;           /* device [Lt][Ht*Dt][mix*Hs*Ds], nn.Linear [out][in] order */
  const void* w_v;
  const float* b_k;          /* device fp32 [Lt][Ht*Dt], or NULL for zero bias */
  const float* b_v;
  int32_t precision;         /* kvx_precision */
  /* Outlier channels of the source cache, read by KVX_PREC_BF16X2_OUTLIER
   * only (ignored otherwise): host [src.n_layers][src.n_kv_heads][src.head_dim],
   * nonzero marks channel (layer, head, dim) of source K (outlier_k) or V
   * (outlier_v); NULL marks none.  Copied into the plan's split table. */
  const uint8_t* outlier_k;
  const uint8_t* outlier_v;
} kvx_plan_desc;

/* One translation call.  Strides are in elements, for (layer, batch, head,
 * token); head_dim is unit-stride.  All-zero strides mean the contiguous
 * layout [L][B][H][T][D] (src: T = src_tokens; tgt: T = tgt_capacity). */
typedef struct {
  int32_t batch;             /* B independent contexts */
  int32_t src_tokens;        /* T_s, the same for all contexts */
  const void* src_k;         /* device, [Ls][B][Hs][T_s][Ds] */
  const void* src_v;
  int64_t src_stride[4];
  /* Token alignment (tokenizers differ).  tgt_tokens == NULL means identity
   * alignment: T_t = T_s and the CSR pointers are ignored. */
  const int32_t* tgt_tokens; /* host [B], T_t of each context */
  const int32_t* row_ptr;    /* device [R+1], R = sum T_t; rows concatenated per
                                context, row_ptr[0] = 0 */
  const int32_t* col_idx;    /* device [nnz], source token index within the context */
  const float* weight;       /* device [nnz], pooling weights */
  void* tgt_k;               /* device, [Lt][B][Ht][tgt_capacity][Dt] */
  void* tgt_v;
  int64_t tgt_stride[4];
  int32_t tgt_capacity;      /* >= max_b T_t[b]; rows t >= T_t[b] are left untouched */
  /* Paged target layout (optional; the cache assembly of a serving system
   * that pages its KV memory, Section 2.2 and Section 6.1).  block_table ==
   * NULL: the contiguous layout above.  Otherwise target token t of context b
   * is written to physical block block_table[b * max_blocks + t / block_size]
   * at slot t % block_size: tgt_stride then reads (layer, block, head, slot),
   * and all-zero strides mean [Lt][num_blocks][Ht][block_size][Dt].
   * tgt_capacity is not used; T_t[b] <= max_blocks * block_size is required.
   * Blocks and slots that no target token maps to are left untouched.  Block
   * ids are trusted unless KVX_VALIDATE=1 (then 0 <= id < num_blocks is
   * checked for every entry a target token uses; KVX_EDATA otherwise). */
  const int32_t* block_table; /* device [B][max_blocks] */
  int32_t block_size;         /* tokens per block, > 0 */
  int32_t max_blocks;         /* block_table entries per context, > 0 */
  int32_t num_blocks;         /* physical blocks in tgt_k / tgt_v, > 0 */
} kvx_io;

typedef struct kvx_plan kvx_plan;

/* Validate the descriptor, copy the layer map and RoPE tables, and repack the
 * weights into plan-owned device memory (synchronous; uses the current HIP
 * device).  The caller's weight and bias buffers may be freed on return.
 * Errors: KVX_EINVAL (NULL/out of range), KVX_ESHAPE, KVX_EUNSUPPORTED
 * (head_dim odd; or a plan the matrix-core kernel does not tile -- fp32, or
 * head_dim not a multiple of 16 (source) / 64 (target) or above 512 -- whose
 * contraction length mix*Hs*Ds exceeds 16384, the pooled rows the general
 * kernel keeps in LDS), KVX_ENOMEM, KVX_EHIP.  On error *out is set to NULL. */
kvx_status kvx_plan_create(const kvx_plan_desc* desc, kvx_plan** out);

/* Enqueue the translation on `stream` (a hipStream_t; NULL = default stream).
 * Asynchronous: KV and alignment buffers are borrowed and must stay valid
 * until the stream work completes.  Every host-visible argument is validated
 * before anything is enqueued; device-resident CSR contents are trusted unless
 * the environment sets KVX_VALIDATE=1 (then, after synchronising `stream`, they
 * are copied back and checked before any launch: row_ptr[0] == 0 and
 * monotone, col_idx in [0, src_tokens), no empty row, and each row's weights
 * summing to 1 within n_row * 2^-23 -- pooling rows partition unity; any
 * violation returns KVX_EDATA with nothing enqueued).  batch == 0 or an
 * empty output is a no-op returning KVX_OK.  The plan is immutable and holds no
 * per-call scratch, so concurrent calls on different streams are safe.
 * Fault injection: with KVX_FAULT=launch in the environment a call that passes
 * validation returns KVX_EHIP (kvx_last_hip_error() = hipErrorLaunchFailure)
 * without enqueuing anything, so a caller's recovery path -- the fallback to
 * native prefill when a translation is unavailable -- can be exercised. */
kvx_status kvx_translate(const kvx_plan* plan, const kvx_io* io, void* stream);

/* Translator variants, composed on the device into the plan's dense
 * per-layer W (and b) at plan creation.  Section 5 of the paper lists
 * low-dimensional latent adapters among the translation mechanisms and
 * Section 2.2 recalls a mixture of translator modules:
 *   KVX_FACTORS_LOWRANK  u = U[l] (V[l] z) + b[l]   ->  W[l] = U[l] V[l]
 *   KVX_FACTORS_MIXTURE  u = sum_k alpha_k (W_k[l] z + b_k[l])
 *                        ->  W[l] = sum_k alpha_k W_k[l], b[l] = sum_k alpha_k b_k[l]
 * The composition reads the factors in the plan's dtype, accumulates in fp32
 * and rounds W once to the plan's dtype (b stays fp32); the translation then
 * runs as for a dense plan, so the equality with the literal variant holds up
 * to that one rounding of W. */
typedef enum { KVX_FACTORS_LOWRANK = 1, KVX_FACTORS_MIXTURE = 2 } kvx_factors_kind;

typedef struct {
  int32_t kind;            /* kvx_factors_kind */
  int32_t rank;            /* LOWRANK: r >= 1 */
  const void* u_k;         /* LOWRANK: device [Lt][Ht*Dt][r], plan dtype */
  const void* u_v;
  const void* v_k;         /* LOWRANK: device [Lt][r][mix*Hs*Ds], plan dtype */
  const void* v_v;
  int32_t n_mix;           /* MIXTURE: 1 <= K <= 32 */
  const double* alpha;     /* MIXTURE: host [K], finite */
  const void* w_k;         /* MIXTURE: device [K][Lt][Ht*Dt][mix*Hs*Ds], plan dtype */
  const void* w_v;
  const float* b_k;        /* MIXTURE: device fp32 [K][Lt][Ht*Dt], or NULL for zero */
  const float* b_v;
} kvx_factors;

/* As kvx_plan_create, with W (and, for a mixture, b) composed from `f`;
 * desc->w_k / w_v are not read (may be NULL); desc->b_k / b_v give the bias
 * of a low-rank plan and are not read for a mixture.  Synchronous.  Errors as
 * kvx_plan_create, plus KVX_EINVAL for a bad kind, rank, K or alpha and
 * KVX_EUNSUPPORTED for K > 32. */
kvx_status kvx_plan_create_factored(const kvx_plan_desc* desc, const kvx_factors* f,
                                    kvx_plan** out);

/* Release a plan (NULL-safe).  The caller must ensure no translation that uses
 * it is still running. */
void kvx_plan_destroy(kvx_plan* plan);

/* Static description of a status code. */
const char* kvx_status_string(kvx_status s);

/* Last HIP error code seen by this thread (0 if none). */
int32_t kvx_last_hip_error(void);

/* Which kernel a plan dispatches to and its launch shape (diagnostics). */
typedef struct {
  int32_t kernel;        /* 0 = fp32 tiled kernel, 1 = bf16 MFMA fused kernel */
  int32_t tile_rows;     /* target rows per workgroup */
  int32_t tile_cols;     /* output features per workgroup */
  int32_t threads;       /* threads per workgroup */
  int32_t precision;     /* kvx_precision of the plan */
  int64_t weight_bytes;  /* device bytes held by the plan */
  /* KVX_PREC_BF16X2_OUTLIER on the fused kernel: of the `ksteps` 16-feature
   * k-steps of all target layers' K and V contractions, `split_ksteps` take
   * the split operand (when the operand is computed).  Both 0 otherwise. */
  int64_t split_ksteps;
  int64_t ksteps;
  /* Fused kernel: order in which the workgroups take the (layer, K|V, row
   * tile, N tile) work units.  0 = contiguous ranges (K and V alternate
   * within a workgroup); 1 = interleaved (each XCD's range dealt
   * round-robin, so the XCD's workgroups share one translator slice in its
   * L2), chosen when din >= 1024; 2 = resident (for span maps: a row tile's
   * pooled, de-rotated rows are formed once and kept in LDS for all of its
   * N tiles), chosen when din <= 256 and dout > 256 -- identity-aligned
   * calls of such a plan use 0.  0 for the tiled kernel. */
  int32_t tile_order;
} kvx_plan_info;

kvx_status kvx_plan_query(const kvx_plan* plan, kvx_plan_info* info);

/* Staged (unfused) translation: the operator of Section 4 as three launches
 * that pass their intermediates through a caller-provided device workspace,
 * for measuring each stage's memory throughput against the fused kernel and as
 * an independent path to check it:
 *   KVX_STAGE_POOL     source RoPE removal on K and pooling over each target
 *                      row's alignment entries (fp32), written to the
 *                      workspace as bf16 planes hi and, unless the plan's
 *                      precision is KVX_PREC_BF16 or the operand is an
 *                      identity-aligned V, lo = bf16(z - hi);
 *   KVX_STAGE_PROJECT  U = Z W^T per (target layer, K|V), fp32, on the
 *                      matrix cores;
 *   KVX_STAGE_STORE    bias, target RoPE on K, bf16 rounding, store into
 *                      the target cache (contiguous or paged).
 * Same arguments, layouts, validation and fault injection as kvx_translate, for plans on the
 * fused kernel (bf16) with precision BF16X2, BF16 or BF16X2_OUTLIER (the
 * latter computed as BF16X2); other plans return KVX_EUNSUPPORTED, as do
 * buffers or strides that are not 16-byte aligned.
 * Workspace: device memory, 16-byte aligned, owned by the caller, not read
 * before it is written; kvx_staged_workspace_bytes gives the bytes that
 * `layers` target layers take for this io (Z: 2 x 2 x rows x din bf16, U:
 * 2 x rows x dout fp32 per layer, rows = the target rows of up to 64
 * contexts, each rounded up to 128).  A smaller workspace runs the layers in
 * groups (KVX_ESHAPE if one layer does not fit).  stages: a non-zero subset
 * of KVX_STAGE_ALL; anything but KVX_STAGE_ALL requires a workspace for all
 * target layers and batch <= 64 (KVX_EINVAL otherwise), and later stages
 * must be called with the same io and workspace after the earlier ones
 * (stream order).  Calls sharing a workspace must not overlap. */
typedef enum {
  KVX_STAGE_POOL = 1,
  KVX_STAGE_PROJECT = 2,
  KVX_STAGE_STORE = 4,
  KVX_STAGE_ALL = 7
} kvx_stage;

kvx_status kvx_staged_workspace_bytes(const kvx_plan* plan, const kvx_io* io, int32_t layers,
                                      size_t* bytes);

kvx_status kvx_translate_staged(const kvx_plan* plan, const kvx_io* io, void* workspace,
                                size_t workspace_bytes, uint32_t stages, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* KVX_H */
