/*
 * kvx_oracle.h -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 CPU implementation of the cross-model KV-translation
 * operator  KV^_B(C) = T_{A->B}(KV_A(C))  (paper Section 4, the translation
 * operator; Section 5, the parameterised translator T_theta).  It exists to
 * check the GPU library against; nothing in the product path may call it.
 *
 * The operator computed, for target layer l, context b, target token t:
 *
 *   1. source row of token k: the concatenation over the mixed source layers
 *      j < mix (ids layer_map[l*mix + j]) and source heads h of the head
 *      vector K_s[ls][b][h][k], de-rotated by the source RoPE at position k
 *      (rotation by -k*theta_i on the pairs (i, i+D/2)); V rows unrotated;
 *   2. token alignment: z_t = sum_e weight[e] * x_{col_idx[e]} over the CSR
 *      row of t (identity alignment: z_t = x_t);
 *   3. projection: u = W[l] z_t + b[l]   (W in nn.Linear [out][in] order);
 *   4. target K head h: rotation of u[h*Dt .. (h+1)*Dt) by +t*theta_i;
 *      target V head h: u[h*Dt .. (h+1)*Dt).
 *
 * theta_i = base^(-2i/D) in fp64 unless an inv_freq table overrides it;
 * base <= 0 disables RoPE on that side.
 *
 * Inputs are read in their storage dtype (float32, or bfloat16 bit patterns)
 * and widened exactly to double; all arithmetic is double.
 */
#ifndef KVX_ORACLE_H
#define KVX_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { KVXO_F32 = 0, KVXO_BF16 = 1 };

typedef struct {
  int32_t n_layers;
  int32_t n_heads;       /* KV heads */
  int32_t head_dim;      /* even */
  double rope_base;      /* <= 0: no RoPE */
  const double* inv_freq;/* optional [head_dim/2] */
} kvxo_model;

typedef struct {
  kvxo_model src, tgt;
  int32_t mix;                 /* source layers per target layer, >= 1 */
  const int32_t* layer_map;    /* [tgt.n_layers * mix] */
  int32_t dtype;               /* KVXO_F32 or KVXO_BF16 (KV and W) */
  const void* w_k;             /* [Lt][Ht*Dt][mix*Hs*Ds] */
  const void* w_v;
  const float* b_k;            /* [Lt][Ht*Dt] or NULL */
  const float* b_v;
  int32_t batch;               /* B */
  int32_t src_tokens;          /* T_s */
  const void* src_k;           /* [Ls][B][Hs][T_s][Ds] contiguous */
  const void* src_v;
  const int32_t* tgt_tokens;   /* [B]; NULL = identity alignment (T_t = T_s) */
  const int32_t* row_ptr;      /* [R+1], rows concatenated per context */
  const int32_t* col_idx;      /* [nnz], source token within the context */
  const float* weight;         /* [nnz] */
} kvxo_problem;

/* y = R(pos) x for one head vector of length D (rotate-half pairing). */
void kvxo_rope(const double* x, double* y, int32_t D, double pos,
               double base, const double* inv_freq);

/* Compute n output rows (layer[i], b[i], t[i]); out_k/out_v are
 * [n][Ht*Dt] (heads concatenated).  Returns 0, or a negative code for an
 * invalid argument (-1 argument, -2 index out of range). */
int kvxo_rows(const kvxo_problem* p, int64_t n, const int32_t* layer,
              const int32_t* b, const int32_t* t, double* out_k, double* out_v);

/* Full operator into tgt_k/tgt_v [Lt][B][Ht][cap][Dt]; rows t >= T_t[b]
 * are left untouched.  Same return codes as kvxo_rows. */
int kvxo_translate(const kvxo_problem* p, int32_t cap, double* tgt_k, double* tgt_v);

/* Threads an OpenMP parallel region of the oracle uses. */
int kvxo_num_threads(void);

#ifdef __cplusplus
}
#endif
#endif
