/*
 * kvx_oracle.c -- TEST INFRASTRUCTURE ONLY: the fp64 CPU oracle of the
 * cross-model KV-translation operator.  See kvx_oracle.h for the definition.
 *
 * Written for obviousness, not speed: one output row at a time, plain loops,
 * no blocking, no BLAS.  Rows are independent, so an OpenMP loop spreads
 * them over host threads; it does not change any result.
 */
#include "kvx_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Exact widening of one stored element to double. */
static double load(const void* base, int32_t dtype, int64_t i) {
  if (dtype == KVXO_F32) return (double)((const float*)base)[i];
  uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* RoPE frequency theta_i of a model side (Section 4 translation operator;
 * the rotary frequencies are the usual base^(-2i/D)). */
static double freq(const kvxo_model* m, int32_t i) {
  if (m->inv_freq) return m->inv_freq[i];
  return pow(m->rope_base, -2.0 * (double)i / (double)m->head_dim);
}

static int has_rope(const kvxo_model* m) {
  return m->inv_freq != NULL || m->rope_base > 0.0;
}

/* Rotate-half RoPE: pair (i, i+D/2) is turned by angle pos*theta_i. */
static void rope_apply(const double* x, double* y, int32_t D, double pos,
                       const double* theta) {
  int32_t h = D / 2;
  for (int32_t i = 0; i < h; ++i) {
    double a = pos * theta[i];
    double c = cos(a), s = sin(a);
    double x0 = x[i], x1 = x[i + h];
    y[i] = x0 * c - x1 * s;
    y[i + h] = x1 * c + x0 * s;
  }
}

void kvxo_rope(const double* x, double* y, int32_t D, double pos, double base,
               const double* inv_freq) {
  kvxo_model m = {1, 1, D, base, inv_freq};
  double* th = (double*)malloc(sizeof(double) * (size_t)(D / 2 + 1));
  for (int32_t i = 0; i < D / 2; ++i) th[i] = freq(&m, i);
  rope_apply(x, y, D, pos, th);
  free(th);
}

int kvxo_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

static int check(const kvxo_problem* p) {
  if (!p || !p->layer_map || !p->w_k || !p->w_v || !p->src_k || !p->src_v) return -1;
  if (p->mix < 1 || p->batch < 0 || p->src_tokens < 0) return -1;
  if (p->src.head_dim <= 0 || p->src.head_dim % 2 || p->tgt.head_dim <= 0 ||
      p->tgt.head_dim % 2)
    return -1;
  for (int64_t i = 0; i < (int64_t)p->tgt.n_layers * p->mix; ++i)
    if (p->layer_map[i] < 0 || p->layer_map[i] >= p->src.n_layers) return -2;
  if (p->tgt_tokens && (!p->row_ptr || !p->col_idx || !p->weight)) return -1;
  return 0;
}

/* Per-thread work buffers. */
typedef struct {
  double *zk, *zv, *uk, *uv, *xk, *xv, *xr, *ths, *tht;
} scratch;

static scratch scratch_new(const kvxo_problem* p) {
  int64_t din = (int64_t)p->mix * p->src.n_heads * p->src.head_dim;
  int64_t dout = (int64_t)p->tgt.n_heads * p->tgt.head_dim;
  scratch s;
  s.zk = (double*)calloc((size_t)din, sizeof(double));
  s.zv = (double*)calloc((size_t)din, sizeof(double));
  s.uk = (double*)calloc((size_t)dout, sizeof(double));
  s.uv = (double*)calloc((size_t)dout, sizeof(double));
  s.xk = (double*)calloc((size_t)p->src.head_dim, sizeof(double));
  s.xv = (double*)calloc((size_t)p->src.head_dim, sizeof(double));
  s.xr = (double*)calloc((size_t)p->src.head_dim, sizeof(double));
  s.ths = (double*)calloc((size_t)p->src.head_dim / 2 + 1, sizeof(double));
  s.tht = (double*)calloc((size_t)p->tgt.head_dim / 2 + 1, sizeof(double));
  for (int32_t i = 0; i < p->src.head_dim / 2; ++i) s.ths[i] = freq(&p->src, i);
  for (int32_t i = 0; i < p->tgt.head_dim / 2; ++i) s.tht[i] = freq(&p->tgt, i);
  return s;
}

static void scratch_free(scratch* s) {
  free(s->zk); free(s->zv); free(s->uk); free(s->uv);
  free(s->xk); free(s->xv); free(s->xr); free(s->ths); free(s->tht);
}

/* One target row (l, b, t) of K and V; out_k/out_v hold Ht*Dt values.
 * row0 is the first CSR row of context b. */
static int one_row(const kvxo_problem* p, scratch* s, int32_t l, int32_t b, int32_t t,
                   int64_t row0, double* out_k, double* out_v) {
  const int32_t Hs = p->src.n_heads, Ds = p->src.head_dim;
  const int32_t Ht = p->tgt.n_heads, Dt = p->tgt.head_dim;
  const int32_t Ts = p->src_tokens, B = p->batch;
  const int64_t din = (int64_t)p->mix * Hs * Ds, dout = (int64_t)Ht * Dt;

  /* Step 2's entry list: a CSR row, or the single token t with weight 1. */
  int64_t e0 = 0, e1 = 1;
  if (p->tgt_tokens) {
    e0 = p->row_ptr[row0 + t];
    e1 = p->row_ptr[row0 + t + 1];
    if (e1 < e0) return -2;
  } else if (t >= Ts) {
    return -2;
  }

  memset(s->zk, 0, sizeof(double) * (size_t)din);
  memset(s->zv, 0, sizeof(double) * (size_t)din);

  /* Steps 1-2: de-rotate every source row of the span at its own position,
   * then pool with the alignment weights. */
  for (int64_t e = e0; e < e1; ++e) {
    int32_t k = p->tgt_tokens ? p->col_idx[e] : t;
    double w = p->tgt_tokens ? (double)p->weight[e] : 1.0;
    if (k < 0 || k >= Ts) return -2;
    for (int32_t j = 0; j < p->mix; ++j) {
      int64_t ls = p->layer_map[(int64_t)l * p->mix + j];
      for (int32_t h = 0; h < Hs; ++h) {
        int64_t src = (((ls * B + b) * Hs + h) * (int64_t)Ts + k) * Ds;
        for (int32_t d = 0; d < Ds; ++d) {
          s->xk[d] = load(p->src_k, p->dtype, src + d);
          s->xv[d] = load(p->src_v, p->dtype, src + d);
        }
        if (has_rope(&p->src))
          rope_apply(s->xk, s->xr, Ds, -(double)k, s->ths);
        else
          memcpy(s->xr, s->xk, sizeof(double) * (size_t)Ds);
        int64_t col = ((int64_t)j * Hs + h) * Ds;
        for (int32_t d = 0; d < Ds; ++d) {
          s->zk[col + d] += w * s->xr[d];
          s->zv[col + d] += w * s->xv[d];
        }
      }
    }
  }

  /* Step 3: u = W z + b, one dot product per output feature. */
  const int64_t wl = (int64_t)l * dout * din;
  for (int64_t o = 0; o < dout; ++o) {
    double ak = 0.0, av = 0.0;
    for (int64_t i = 0; i < din; ++i) {
      ak += load(p->w_k, p->dtype, wl + o * din + i) * s->zk[i];
      av += load(p->w_v, p->dtype, wl + o * din + i) * s->zv[i];
    }
    if (p->b_k) ak += (double)p->b_k[(int64_t)l * dout + o];
    if (p->b_v) av += (double)p->b_v[(int64_t)l * dout + o];
    s->uk[o] = ak;
    s->uv[o] = av;
  }

  /* Step 4: target RoPE on each K head at the target position t. */
  for (int32_t h = 0; h < Ht; ++h) {
    const double* u = s->uk + (int64_t)h * Dt;
    if (has_rope(&p->tgt))
      rope_apply(u, out_k + (int64_t)h * Dt, Dt, (double)t, s->tht);
    else
      memcpy(out_k + (int64_t)h * Dt, u, sizeof(double) * (size_t)Dt);
  }
  memcpy(out_v, s->uv, sizeof(double) * (size_t)dout);
  return 0;
}

static void row_offsets(const kvxo_problem* p, int64_t* off) {
  off[0] = 0;
  for (int32_t b = 0; b < p->batch; ++b)
    off[b + 1] = off[b] + (p->tgt_tokens ? p->tgt_tokens[b] : p->src_tokens);
}

int kvxo_rows(const kvxo_problem* p, int64_t n, const int32_t* layer, const int32_t* b,
              const int32_t* t, double* out_k, double* out_v) {
  int rc = check(p);
  if (rc) return rc;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(p->batch + 1));
  row_offsets(p, off);
  const int64_t dout = (int64_t)p->tgt.n_heads * p->tgt.head_dim;
  for (int64_t i = 0; i < n; ++i) {
    if (layer[i] < 0 || layer[i] >= p->tgt.n_layers || b[i] < 0 || b[i] >= p->batch ||
        t[i] < 0 || t[i] >= off[b[i] + 1] - off[b[i]]) {
      free(off);
      return -2;
    }
  }
  int err = 0;
#pragma omp parallel
  {
    scratch s = scratch_new(p);
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i) {
      int r = one_row(p, &s, layer[i], b[i], t[i], off[b[i]], out_k + i * dout,
                      out_v + i * dout);
      if (r) {
#pragma omp atomic write
        err = r;
      }
    }
    scratch_free(&s);
  }
  free(off);
  return err;
}

int kvxo_translate(const kvxo_problem* p, int32_t cap, double* tgt_k, double* tgt_v) {
  int rc = check(p);
  if (rc) return rc;
  const int32_t Lt = p->tgt.n_layers, Ht = p->tgt.n_heads, Dt = p->tgt.head_dim;
  const int32_t B = p->batch;
  int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B + 1));
  row_offsets(p, off);
  for (int32_t b = 0; b < B; ++b)
    if (off[b + 1] - off[b] > cap) {
      free(off);
      return -1;
    }
  const int64_t n = (int64_t)Lt * off[B];
  if (n == 0) {
    free(off);
    return 0;
  }
  int err = 0;
#pragma omp parallel
  {
    scratch s = scratch_new(p);
    double* rk = (double*)malloc(sizeof(double) * (size_t)Ht * Dt);
    double* rv = (double*)malloc(sizeof(double) * (size_t)Ht * Dt);
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < n; ++i) {
      int32_t l = (int32_t)(i / off[B]);
      int64_t r = i % off[B];
      int32_t b = 0;
      while (r >= off[b + 1]) ++b;
      int32_t t = (int32_t)(r - off[b]);
      int e = one_row(p, &s, l, b, t, off[b], rk, rv);
      if (e) {
#pragma omp atomic write
        err = e;
        continue;
      }
      for (int32_t h = 0; h < Ht; ++h) {
        int64_t dst = ((((int64_t)l * B + b) * Ht + h) * cap + t) * Dt;
        memcpy(tgt_k + dst, rk + (int64_t)h * Dt, sizeof(double) * (size_t)Dt);
        memcpy(tgt_v + dst, rv + (int64_t)h * Dt, sizeof(double) * (size_t)Dt);
      }
    }
    free(rk);
    free(rv);
    scratch_free(&s);
  }
  free(off);
  return err;
}
