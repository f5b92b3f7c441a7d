// kvx.hip -- C-ABI of the KV-translation library: plan creation (validation,
// weight packing, RoPE tables), translation (validation, launch), teardown.
// The declarations and their contracts are in include/kvx.h.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "kvx.h"
#include "common.h"
#include "kernel_mfma.h"
#include "fused_launch.h"
#include "kernel_tiled.h"
#include "staged.h"

using namespace kvx;

namespace {

thread_local int32_t g_last_hip = 0;

kvx_status hip_fail(hipError_t e) { return kvx::hip_status(e); }

#define KVX_HIP(x)                          \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return hip_fail(e_); \
  } while (0)

enum Kernel { kTiled = 0, kFused = 1 };

}  // namespace

kvx_status kvx::hip_status(hipError_t e) {
  if (e == hipSuccess) return KVX_OK;
  g_last_hip = static_cast<int32_t>(e);
  return e == hipErrorOutOfMemory ? KVX_ENOMEM : KVX_EHIP;
}

struct kvx_plan {
  int device = 0;
  kvx_model src{}, tgt{};
  int32_t mix = 1;
  int32_t dtype = KVX_BF16;
  int32_t precision = KVX_PREC_BF16X2;
  int32_t din = 0, dout = 0;
  int kernel = kTiled;
  int n_cu = 0;                  // compute units of the plan's device
  int64_t bytes = 0;
  // device memory owned by the plan
  int32_t* layer_map = nullptr;  // [Lt*mix]
  double* fs = nullptr;          // [Ds/2] theta_i / 2pi (zeros when RoPE is off)
  double* ft = nullptr;          // [Dt/2]
  void* w[2] = {nullptr, nullptr};  // tiled: [Lt][dout][din]; fused: packed fragments
  void* wh[2] = {nullptr, nullptr}; // fused, precision F16: packed fp16 fragments
  float* bias[2] = {nullptr, nullptr};
  // fused kernel: a zero area that lanes without data load from, and an area
  // that lanes without a valid output row store to (never read), so that
  // every global access of the kernel is unconditional
  void* zsink = nullptr;
  void* trash = nullptr;
  uint8_t* split_mask = nullptr; // precision BF16X2_OUTLIER: [Lt][2][din/128]
  int64_t split_ksteps = 0, ksteps = 0;
  // fused kernel: interleaved tile order (1) when one tile's weight slice
  // (din x 256 bf16) reaches 512 KiB; with contiguous ranges the workgroups
  // of an XCD would then keep several layers' translators in flight, more
  // than its 4 MiB L2 holds.  Resident order (2) when a row tile's whole
  // contraction (din <= 256) fits the kernel's two LDS buffers and the
  // output has several N tiles: the chunks are transformed once and kept
  // for all N tiles (span maps; identity-aligned calls use 0).
  int32_t tile_order = 0;
  void* block = nullptr;         // single allocation backing all of the above
};

namespace {

bool valid_model(const kvx_model& m) {
  return m.n_layers > 0 && m.n_kv_heads > 0 && m.head_dim > 0 && std::isfinite(m.rope_base);
}

// theta_i / (2 pi) for i < D/2 in fp64; all zero when the side has no RoPE.
std::vector<double> rope_table(const kvx_model& m) {
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

bool fused_supported(const kvx_plan& p) {
  return p.dtype == KVX_BF16 && p.src.head_dim % 16 == 0 && p.din % 128 == 0 &&
         p.tgt.head_dim % 64 == 0 && p.dout % 64 == 0 &&
         p.src.head_dim / 2 <= kMaxHalfDim && p.tgt.head_dim / 2 <= kMaxHalfDim &&
         int64_t(p.tgt.n_layers) * p.mix <= kMaxLayerMap;
}

// Target rows per workgroup of the tiled kernel, and the LDS its pooled rows
// take (rows x din fp32).
int tiled_rows(int din) {
  int r = 16384 / (din > 0 ? din : 1);
  return r < 1 ? 1 : (r > 16 ? 16 : r);
}
// dynamic LDS a launch gets without raising the kernel's limit (64 KiB):
// din <= 16384
constexpr size_t kMaxLdsBytes = 64 * 1024;
size_t tiled_lds_bytes(int din) { return size_t(tiled_rows(din)) * din * sizeof(float); }

// Input feature held in K-slot `k` of the fused kernel: chunk c = k / 128 holds
// the RoPE pairs 64c .. 64c+63 of the flattened (mixed layer, head, d < Ds/2)
// list, first members in slots 0..63, second members (d + Ds/2) in 64..127.
int64_t fused_feature_of_slot(int64_t k, int64_t ds) {
  const int64_t c = k / 128, s = k % 128;
  const int64_t pair = 64 * c + (s % 64);
  const int64_t half = ds / 2;
  const int64_t head = pair / half;  // (j * Hs + h)
  const int64_t d = pair % half + (s >= 64 ? half : 0);
  return head * ds + d;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

}  // namespace

extern "C" {

const char* kvx_status_string(kvx_status s) {
  switch (s) {
    case KVX_OK: return "ok";
    case KVX_EINVAL: return "invalid argument";
    case KVX_ESHAPE: return "inconsistent shape, stride or capacity";
    case KVX_EUNSUPPORTED: return "unsupported configuration";
    case KVX_ENOMEM: return "out of device memory";
    case KVX_EHIP: return "HIP runtime error";
    case KVX_EDATA: return "invalid alignment data";
  }
  return "unknown status";
}

int32_t kvx_last_hip_error(void) { return g_last_hip; }

kvx_status kvx_plan_create(const kvx_plan_desc* d, kvx_plan** out) {
  if (out) *out = nullptr;
  if (!d || !out || !d->layer_map || !d->w_k || !d->w_v) return KVX_EINVAL;
  if (!valid_model(d->src) || !valid_model(d->tgt) || d->mix < 1) return KVX_EINVAL;
  if (d->dtype != KVX_F32 && d->dtype != KVX_BF16) return KVX_EINVAL;
  if (d->precision != KVX_PREC_BF16X2 && d->precision != KVX_PREC_BF16 &&
      d->precision != KVX_PREC_F16 && d->precision != KVX_PREC_BF16X2_OUTLIER)
    return KVX_EINVAL;
  if (d->src.head_dim % 2 || d->tgt.head_dim % 2) return KVX_EUNSUPPORTED;
  const int64_t lt = d->tgt.n_layers;
  for (int64_t i = 0; i < lt * d->mix; ++i)
    if (d->layer_map[i] < 0 || d->layer_map[i] >= d->src.n_layers) return KVX_EINVAL;
  const int64_t din64 = int64_t(d->mix) * d->src.n_kv_heads * d->src.head_dim;
  const int64_t dout64 = int64_t(d->tgt.n_kv_heads) * d->tgt.head_dim;
  if (din64 > (1 << 20) || dout64 > (1 << 20)) return KVX_ESHAPE;
  if (d->src.inv_freq)
    for (int i = 0; i < d->src.head_dim / 2; ++i)
      if (!std::isfinite(d->src.inv_freq[i])) return KVX_EINVAL;
  if (d->tgt.inv_freq)
    for (int i = 0; i < d->tgt.head_dim / 2; ++i)
      if (!std::isfinite(d->tgt.inv_freq[i])) return KVX_EINVAL;

  kvx_plan* p = new (std::nothrow) kvx_plan();
  if (!p) return KVX_ENOMEM;
  p->src = d->src;
  p->tgt = d->tgt;
  p->src.inv_freq = p->tgt.inv_freq = nullptr;  // tables live on the device
  p->mix = d->mix;
  p->dtype = d->dtype;
  p->precision = d->precision;
  p->din = static_cast<int32_t>(din64);
  p->dout = static_cast<int32_t>(dout64);
  p->kernel = fused_supported(*p) ? kFused : kTiled;
  // the tiled kernel holds one pooled row (din fp32) per target row in LDS
  if (p->kernel == kTiled && tiled_lds_bytes(p->din) > kMaxLdsBytes) {
    delete p;
    return KVX_EUNSUPPORTED;
  }
  p->tile_order = p->kernel != kFused ? 0 : p->din >= 1024 ? 1 : (p->din <= 256 && p->dout > 256) ? 2 : 0;

  auto fail = [&](kvx_status s) {
    kvx_plan_destroy(p);
    return s;
  };

  hipError_t e = hipGetDevice(&p->device);
  if (e != hipSuccess) return fail(hip_fail(e));
  e = hipDeviceGetAttribute(&p->n_cu, hipDeviceAttributeMultiprocessorCount, p->device);
  if (e != hipSuccess) return fail(hip_fail(e));

  const size_t esz = d->dtype == KVX_F32 ? 4 : 2;
  const size_t wbytes = size_t(lt) * dout64 * din64 * esz;
  const size_t bbytes = size_t(lt) * dout64 * sizeof(float);
  const size_t mbytes = size_t(lt) * d->mix * sizeof(int32_t);
  const size_t fsb = d->src.head_dim / 2 * sizeof(double);
  const size_t ftb = d->tgt.head_dim / 2 * sizeof(double);
  const bool want_f16 = p->kernel == kFused && d->precision == KVX_PREC_F16;
  const size_t hbytes = want_f16 ? wbytes : 0;
  size_t off_w0 = 0, off_w1 = align256(wbytes);
  size_t off_h0 = off_w1 + align256(wbytes), off_h1 = off_h0 + align256(hbytes);
  size_t off_b0 = off_h1 + align256(hbytes);
  size_t off_b1 = off_b0 + align256(bbytes), off_m = off_b1 + align256(bbytes);
  size_t off_fs = off_m + align256(mbytes), off_ft = off_fs + align256(fsb);
  const bool want_mask = p->kernel == kFused && d->precision == KVX_PREC_BF16X2_OUTLIER;
  const int64_t nch = din64 / 128;
  const size_t smb = want_mask ? size_t(lt) * 2 * nch : 0;
  size_t off_sink = off_ft + align256(ftb);
  size_t off_sm = off_sink + 2 * kSinkBytes;
  size_t total = off_sm + align256(smb);
  e = hipMalloc(&p->block, total);
  if (e != hipSuccess) return fail(hip_fail(e));
  p->bytes = static_cast<int64_t>(total);
  char* base = static_cast<char*>(p->block);
  p->w[0] = base + off_w0;
  p->w[1] = base + off_w1;
  if (want_f16) {
    p->wh[0] = base + off_h0;
    p->wh[1] = base + off_h1;
  }
  p->bias[0] = reinterpret_cast<float*>(base + off_b0);
  p->bias[1] = reinterpret_cast<float*>(base + off_b1);
  p->layer_map = reinterpret_cast<int32_t*>(base + off_m);
  p->fs = reinterpret_cast<double*>(base + off_fs);
  p->ft = reinterpret_cast<double*>(base + off_ft);
  p->zsink = base + off_sink;
  p->trash = base + off_sink + kSinkBytes;
  if (want_mask) p->split_mask = reinterpret_cast<uint8_t*>(base + off_sm);
  e = hipMemset(p->zsink, 0, kSinkBytes);
  if (e != hipSuccess) return fail(hip_fail(e));

  // Weights: copy to the host, repack, upload.  Plan creation is once per
  // translator, so clarity wins over speed here.
  std::vector<char> host(wbytes), packed;
  const void* wsrc[2] = {d->w_k, d->w_v};
  for (int kv = 0; kv < 2; ++kv) {
    e = hipMemcpy(host.data(), wsrc[kv], wbytes, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(hip_fail(e));
    const void* up = host.data();
    if (p->kernel == kFused) {
      // A fragment (feature block nb, k-step ks) of v_mfma_f32_32x32x16_bf16:
      // lane holds W[nb*32 + lane%32][feature of slot ks*16 + 8*(lane/32) + j].
      packed.resize(wbytes);
      const uint16_t* wsrc16 = reinterpret_cast<const uint16_t*>(host.data());
      uint16_t* dst = reinterpret_cast<uint16_t*>(packed.data());
      const int64_t nb_n = dout64 / 32, ks_n = din64 / 16;
      std::vector<int64_t> feat(din64);
      for (int64_t k = 0; k < din64; ++k) feat[k] = fused_feature_of_slot(k, d->src.head_dim);
      for (int64_t l = 0; l < lt; ++l)
        for (int64_t nb = 0; nb < nb_n; ++nb)
          for (int64_t ks = 0; ks < ks_n; ++ks)
            for (int lanei = 0; lanei < 64; ++lanei)
              for (int jj = 0; jj < 8; ++jj) {
                const int64_t o = nb * 32 + lanei % 32;
                const int64_t i = feat[ks * 16 + 8 * (lanei / 32) + jj];
                dst[((((l * nb_n + nb) * ks_n + ks) * 64 + lanei) * 8) + jj] =
                    wsrc16[(l * dout64 + o) * din64 + i];
              }
      up = packed.data();
    }
    e = hipMemcpy(p->w[kv], up, wbytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(hip_fail(e));
    if (want_f16) {
      // the same fragments as fp16 (exact for bf16 values in the fp16 normal
      // range; smaller magnitudes round to the nearest fp16 subnormal)
      std::vector<uint16_t> h(wbytes / 2);
      const uint16_t* src16 = static_cast<const uint16_t*>(up);
      for (size_t i = 0; i < h.size(); ++i) {
        uint32_t u = static_cast<uint32_t>(src16[i]) << 16;
        float f;
        std::memcpy(&f, &u, sizeof f);
        if (!(std::fabs(f) <= 65504.0f)) return fail(KVX_EUNSUPPORTED);
        _Float16 hv = static_cast<_Float16>(f);
        std::memcpy(&h[i], &hv, sizeof hv);
      }
      e = hipMemcpy(p->wh[kv], h.data(), wbytes, hipMemcpyHostToDevice);
      if (e != hipSuccess) return fail(hip_fail(e));
    }
  }
  const float* bsrc[2] = {d->b_k, d->b_v};
  for (int kv = 0; kv < 2; ++kv) {
    if (bsrc[kv])
      e = hipMemcpy(p->bias[kv], bsrc[kv], bbytes, hipMemcpyDeviceToDevice);
    else
      e = hipMemset(p->bias[kv], 0, bbytes);
    if (e != hipSuccess) return fail(hip_fail(e));
  }
  e = hipMemcpy(p->layer_map, d->layer_map, mbytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(hip_fail(e));
  std::vector<double> fsv = rope_table(d->src), ftv = rope_table(d->tgt);
  e = hipMemcpy(p->fs, fsv.data(), fsb, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(hip_fail(e));
  e = hipMemcpy(p->ft, ftv.data(), ftb, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(hip_fail(e));
  if (want_mask) {
    // Bit ks of entry (l, kv, c): k-step ks of chunk c holds a marked channel
    // (for K, also a channel whose RoPE partner is marked).
    const int hs = d->src.n_kv_heads, ds = d->src.head_dim;
    std::vector<uint8_t> sm(smb, 0);
    const uint8_t* marks[2] = {d->outlier_k, d->outlier_v};
    for (int64_t l = 0; l < lt; ++l)
      for (int kv = 0; kv < 2; ++kv)
        for (int64_t k = 0; k < din64; ++k) {
          if (!marks[kv]) break;
          const int64_t f = fused_feature_of_slot(k, ds);
          const int64_t j = f / (int64_t(hs) * ds), h = (f / ds) % hs, dd = f % ds;
          const int64_t ls = d->layer_map[l * d->mix + j];
          const uint8_t* row = marks[kv] + (ls * hs + h) * ds;
          const bool hit = row[dd] != 0 || (kv == 0 && row[(dd + ds / 2) % ds] != 0);
          if (hit) sm[(l * 2 + kv) * nch + k / 128] |= uint8_t(1u << ((k % 128) / 16));
        }
    for (uint8_t b : sm)
      for (int i = 0; i < 8; ++i) p->split_ksteps += (b >> i) & 1;
    p->ksteps = int64_t(smb) * 8;
    e = hipMemcpy(p->split_mask, sm.data(), smb, hipMemcpyHostToDevice);
    if (e != hipSuccess) return fail(hip_fail(e));
  }
  e = hipDeviceSynchronize();
  if (e != hipSuccess) return fail(hip_fail(e));
  *out = p;
  return KVX_OK;
}

void kvx_plan_destroy(kvx_plan* p) {
  if (!p) return;
  if (p->block) (void)hipFree(p->block);
  delete p;
}

kvx_status kvx_plan_query(const kvx_plan* p, kvx_plan_info* info) {
  if (!p || !info) return KVX_EINVAL;
  info->kernel = p->kernel;
  info->tile_rows = p->kernel == kFused ? kMT : 0;
  info->tile_cols = p->kernel == kFused ? kNT : 0;
  info->threads = p->kernel == kFused ? kThreads : 256;
  info->precision = p->precision;
  info->weight_bytes = p->bytes;
  info->split_ksteps = p->split_ksteps;
  info->ksteps = p->ksteps;
  info->tile_order = p->tile_order;
  return KVX_OK;
}

}  // extern "C"

namespace {

void launch_fused(bool identity, bool ds128, int precision, int grid, hipStream_t st,
                  const FusedArgs& a) {
  switch (precision) {
    case KVX_PREC_BF16: launch_fused_bf16(identity, ds128, grid, st, a); break;
    case KVX_PREC_F16: launch_fused_f16(identity, ds128, grid, st, a); break;
    default: launch_fused_bf16x2(identity, ds128, grid, st, a); break;
  }
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Host-side check of device CSR contents (validation mode only).
kvx_status validate_csr(const kvx_io& io, int64_t rows, hipStream_t st) {
  std::vector<int32_t> rp(rows + 1);
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e);
  e = hipMemcpy(rp.data(), io.row_ptr, (rows + 1) * sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  if (rp[0] != 0) return KVX_EDATA;
  for (int64_t r = 0; r < rows; ++r)
    if (rp[r + 1] < rp[r]) return KVX_EDATA;
  const int64_t nnz = rp[rows];
  std::vector<int32_t> ci(nnz > 0 ? nnz : 1);
  if (nnz > 0) {
    e = hipMemcpy(ci.data(), io.col_idx, nnz * sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e);
  }
  for (int64_t i = 0; i < nnz; ++i)
    if (ci[i] < 0 || ci[i] >= io.src_tokens) return KVX_EDATA;
  // Pooling rows are a partition of unity: no empty row, and the weights of
  // each row sum to 1 within the rounding of its entries (each weight an fp32
  // value, so |sum - 1| <= n_row * 2^-23 for weights that round 1/n_row).
  std::vector<float> wv(nnz > 0 ? nnz : 1);
  if (nnz > 0) {
    e = hipMemcpy(wv.data(), io.weight, nnz * sizeof(float), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e);
  }
  for (int64_t r = 0; r < rows; ++r) {
    const int64_t n = int64_t(rp[r + 1]) - rp[r];
    if (n == 0) return KVX_EDATA;
    double sum = 0.0;
    for (int64_t i = rp[r]; i < rp[r + 1]; ++i) sum += double(wv[i]);
    if (!(std::fabs(sum - 1.0) <= double(n) * std::ldexp(1.0, -23))) return KVX_EDATA;
  }
  return KVX_OK;
}

// Host-side check of the block ids that target tokens use (validation mode).
kvx_status validate_blocks(const kvx_io& io, const std::vector<int32_t>& ttok, hipStream_t st) {
  std::vector<int32_t> bt(size_t(io.batch) * io.max_blocks);
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e);
  e = hipMemcpy(bt.data(), io.block_table, bt.size() * sizeof(int32_t), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  for (int b = 0; b < io.batch; ++b) {
    const int64_t used = (int64_t(ttok[b]) + io.block_size - 1) / io.block_size;
    for (int64_t j = 0; j < used; ++j) {
      const int32_t id = bt[size_t(b) * io.max_blocks + j];
      if (id < 0 || id >= io.num_blocks) return KVX_EDATA;
    }
  }
  return KVX_OK;
}

// A call's arguments with the default strides filled in and the target rows
// of every context; rows == 0: nothing to do.
struct Call {
  kvx_io io;
  bool identity = false, paged = false;
  std::vector<int32_t> ttok;
  int64_t rows = 0;
};

kvx_status prepare_call(const kvx_plan* p, const kvx_io* io_in, Call& c) {
  if (!p || !io_in) return KVX_EINVAL;
  kvx_io& io = c.io;
  io = *io_in;
  if (io.batch < 0 || io.src_tokens < 0 || io.tgt_capacity < 0) return KVX_EINVAL;
  if (io.batch == 0) return KVX_OK;
  const bool identity = io.tgt_tokens == nullptr;
  const bool paged = io.block_table != nullptr;
  c.identity = identity;
  c.paged = paged;
  if (paged && (io.block_size <= 0 || io.max_blocks <= 0 || io.num_blocks <= 0))
    return KVX_EINVAL;
  // rows a context may hold in the target layout
  const int64_t cap = paged ? int64_t(io.max_blocks) * io.block_size : io.tgt_capacity;
  c.ttok.assign(io.batch, 0);
  int64_t rows = 0;
  for (int b = 0; b < io.batch; ++b) {
    const int32_t t = identity ? io.src_tokens : io.tgt_tokens[b];
    if (t < 0) return KVX_EINVAL;
    if (t > cap) return KVX_ESHAPE;
    c.ttok[b] = t;
    rows += t;
  }
  if (rows == 0) return KVX_OK;
  if (!io.src_k || !io.src_v || !io.tgt_k || !io.tgt_v) return KVX_EINVAL;
  if (!identity && (!io.row_ptr || !io.col_idx || !io.weight)) return KVX_EINVAL;
  if (rows > INT32_MAX / 2) return KVX_ESHAPE;

  const int64_t Hs = p->src.n_kv_heads, Ds = p->src.head_dim;
  const int64_t Ht = p->tgt.n_kv_heads, Dt = p->tgt.head_dim;
  const int64_t B = io.batch;
  auto all_zero = [](const int64_t* s) { return !s[0] && !s[1] && !s[2] && !s[3]; };
  if (all_zero(io.src_stride)) {
    io.src_stride[3] = Ds;
    io.src_stride[2] = Ds * io.src_tokens;
    io.src_stride[1] = Hs * io.src_stride[2];
    io.src_stride[0] = B * io.src_stride[1];
  }
  if (all_zero(io.tgt_stride)) {
    // contiguous [Lt][B][Ht][tgt_capacity][Dt], or paged
    // [Lt][num_blocks][Ht][block_size][Dt]
    io.tgt_stride[3] = Dt;
    io.tgt_stride[2] = Dt * (paged ? int64_t(io.block_size) : int64_t(io.tgt_capacity));
    io.tgt_stride[1] = Ht * io.tgt_stride[2];
    io.tgt_stride[0] = (paged ? int64_t(io.num_blocks) : B) * io.tgt_stride[1];
  }
  for (int i = 0; i < 4; ++i)
    if (io.src_stride[i] < 0 || io.tgt_stride[i] < 0) return KVX_ESHAPE;
  // strides must keep one row (head_dim values) inside the next-outer step
  const int64_t tgt_rows = paged ? io.block_size : io.tgt_capacity;  // rows per token stride run
  if ((io.src_stride[3] < Ds && io.src_tokens > 1) || (io.tgt_stride[3] < Dt && tgt_rows > 1))
    return KVX_ESHAPE;
  c.rows = rows;
  return KVX_OK;
}

// KVX_VALIDATE=1: check the device-resident alignment map and block table.
kvx_status validate_call(const Call& c, bool csr, bool blocks, hipStream_t st) {
  const char* vmode = std::getenv("KVX_VALIDATE");
  if (!(vmode && vmode[0] == '1')) return KVX_OK;
  if (csr && !c.identity) {
    kvx_status s = validate_csr(c.io, c.rows, st);
    if (s != KVX_OK) return s;
  }
  if (blocks && c.paged) {
    kvx_status s = validate_blocks(c.io, c.ttok, st);
    if (s != KVX_OK) return s;
  }
  return KVX_OK;
}

// KVX_FAULT=launch: the call reports a failed launch (KVX_EHIP, with
// hipErrorLaunchFailure for kvx_last_hip_error) after its validation, with
// nothing enqueued -- so callers' recovery paths (the paper's fallback to
// native prefill) can be tested without making a kernel fail.
bool injected_launch_fault() {
  const char* f = std::getenv("KVX_FAULT");
  return f && std::strcmp(f, "launch") == 0;
}

// 16-byte vector access needs 16-byte aligned rows and buffers.
bool rows_aligned16(const kvx_io& io, int esz) {
  for (int i = 0; i < 4; ++i)
    if ((io.src_stride[i] * esz) % 16 || (io.tgt_stride[i] * esz) % 16) return false;
  return aligned16(io.src_k) && aligned16(io.src_v) && aligned16(io.tgt_k) && aligned16(io.tgt_v);
}

}  // namespace

extern "C" kvx_status kvx_translate(const kvx_plan* p, const kvx_io* io_in, void* stream) {
  Call call;
  kvx_status cs = prepare_call(p, io_in, call);
  if (cs != KVX_OK || call.rows == 0) return cs;
  const kvx_io& io = call.io;
  const bool identity = call.identity, paged = call.paged;
  const std::vector<int32_t>& ttok = call.ttok;
  const int64_t rows = call.rows;
  const int64_t Hs = p->src.n_kv_heads, Ds = p->src.head_dim;
  const int64_t Lt = p->tgt.n_layers, Ht = p->tgt.n_kv_heads, Dt = p->tgt.head_dim;
  const int64_t B = io.batch;
  hipStream_t st = static_cast<hipStream_t>(stream);
  cs = validate_call(call, true, true, st);
  if (cs != KVX_OK) return cs;
  if (injected_launch_fault()) return hip_fail(hipErrorLaunchFailure);

  const int esz = p->dtype == KVX_F32 ? 4 : 2;
  bool fused = p->kernel == kFused && rows_aligned16(io, esz);
  // the fused kernel addresses a context's rows of one head with 32-bit byte
  // offsets (contiguous layout)
  if (fused && !paged && int64_t(io.tgt_capacity) * io.tgt_stride[3] * esz > INT32_MAX)
    fused = false;
  if (p->kernel == kFused && !fused) return KVX_EUNSUPPORTED;

  const Strides ss{io.src_stride[0], io.src_stride[1], io.src_stride[2], io.src_stride[3]};
  const Strides ts{io.tgt_stride[0], io.tgt_stride[1], io.tgt_stride[2], io.tgt_stride[3]};
  int64_t row_base = 0;
  for (int64_t b0 = 0; b0 < B; b0 += kMaxBatch) {
    const int nb = static_cast<int>(B - b0 < kMaxBatch ? B - b0 : kMaxBatch);
    BatchArgs ba{};
    ba.n = nb;
    const int rows_per_tile = fused ? kMT : tiled_rows(p->din);
    int tiles = 0;
    for (int i = 0; i < nb; ++i) {
      ba.tile_start[i] = tiles;
      ba.t_tgt[i] = ttok[b0 + i];
      ba.row_base[i] = static_cast<int32_t>(row_base);
      row_base += ttok[b0 + i];
      tiles += (ttok[b0 + i] + rows_per_tile - 1) / rows_per_tile;
    }
    ba.tile_start[nb] = tiles;
    if (tiles == 0) continue;
    const char* sk = static_cast<const char*>(io.src_k) + b0 * io.src_stride[1] * esz;
    const char* sv = static_cast<const char*>(io.src_v) + b0 * io.src_stride[1] * esz;
    // paged: blocks are shared by all contexts; the table row moves instead
    const int64_t toff = paged ? 0 : b0 * io.tgt_stride[1] * esz;
    char* tk = static_cast<char*>(io.tgt_k) + toff;
    char* tv = static_cast<char*>(io.tgt_v) + toff;
    const Paging pg{paged ? io.block_table + b0 * io.max_blocks : nullptr,
                    paged ? io.block_size : 1, paged ? io.max_blocks : 0};
    if (fused) {
      FusedArgs a{};
      a.src[0] = reinterpret_cast<const bf16_t*>(sk);
      a.src[1] = reinterpret_cast<const bf16_t*>(sv);
      a.ss = ss;
      a.tgt[0] = reinterpret_cast<bf16_t*>(tk);
      a.tgt[1] = reinterpret_cast<bf16_t*>(tv);
      a.ts = ts;
      a.wp[0] = static_cast<const bf16x8*>(p->w[0]);
      a.wp[1] = static_cast<const bf16x8*>(p->w[1]);
      a.wh[0] = static_cast<const bf16x8*>(p->wh[0]);
      a.wh[1] = static_cast<const bf16x8*>(p->wh[1]);
      a.bias[0] = p->bias[0];
      a.bias[1] = p->bias[1];
      a.layer_map = p->layer_map;
      a.mix = p->mix;
      a.hs = static_cast<int32_t>(Hs);
      a.ht = static_cast<int32_t>(Ht);
      a.dt = static_cast<int32_t>(Dt);
      a.din = p->din;
      a.dout = p->dout;
      a.ds = static_cast<int32_t>(Ds);
      a.lt = static_cast<int32_t>(Lt);
      a.fs = p->fs;
      a.ft = p->ft;
      a.zsink = static_cast<const bf16_t*>(p->zsink);
      a.trash = static_cast<bf16_t*>(p->trash);
      a.row_ptr = io.row_ptr;
      a.col_idx = io.col_idx;
      a.weight = io.weight;
      a.n_tiles = (p->dout / 64 + 3) / 4;
      a.row_tiles = tiles;
      a.pg = pg;
      a.split_mask = p->split_mask;
      a.ba = ba;
      const int64_t total = int64_t(tiles) * a.n_tiles * 2 * Lt;
      if (total > INT32_MAX) return KVX_ESHAPE;
      a.total_tiles = static_cast<int32_t>(total);
      // the resident order (a row tile's chunks kept in LDS for its N tiles)
      // serves span maps; identity-aligned calls of such plans take the
      // contiguous order
      a.interleave = p->tile_order == 2 && identity ? 0 : p->tile_order;
      // persistent: one workgroup per compute unit (the kernel's LDS use
      // allows exactly one)
      const int grid = static_cast<int>(total < p->n_cu ? total : p->n_cu);
      launch_fused(identity, Ds == 128, p->precision, grid, st, a);
    } else {
      const size_t lds = tiled_lds_bytes(p->din);
      if (p->dtype == KVX_F32) {
        TiledArgs<float> a{};
        a.src[0] = reinterpret_cast<const float*>(sk);
        a.src[1] = reinterpret_cast<const float*>(sv);
        a.tgt[0] = reinterpret_cast<float*>(tk);
        a.tgt[1] = reinterpret_cast<float*>(tv);
        a.w[0] = static_cast<const float*>(p->w[0]);
        a.w[1] = static_cast<const float*>(p->w[1]);
        a.ss = ss; a.ts = ts;
        a.bias[0] = p->bias[0]; a.bias[1] = p->bias[1];
        a.layer_map = p->layer_map; a.mix = p->mix;
        a.hs = Hs; a.ds = Ds; a.ht = Ht; a.dt = Dt; a.din = p->din; a.dout = p->dout;
        a.fs = p->fs; a.ft = p->ft;
        a.row_ptr = io.row_ptr; a.col_idx = io.col_idx; a.weight = io.weight;
        a.identity = identity; a.rows = rows_per_tile; a.pg = pg; a.ba = ba;
        tiled_kernel<float><<<dim3(tiles, Lt, 2), dim3(256), lds, st>>>(a);
      } else {
        TiledArgs<bf16_t> a{};
        a.src[0] = reinterpret_cast<const bf16_t*>(sk);
        a.src[1] = reinterpret_cast<const bf16_t*>(sv);
        a.tgt[0] = reinterpret_cast<bf16_t*>(tk);
        a.tgt[1] = reinterpret_cast<bf16_t*>(tv);
        a.w[0] = static_cast<const bf16_t*>(p->w[0]);
        a.w[1] = static_cast<const bf16_t*>(p->w[1]);
        a.ss = ss; a.ts = ts;
        a.bias[0] = p->bias[0]; a.bias[1] = p->bias[1];
        a.layer_map = p->layer_map; a.mix = p->mix;
        a.hs = Hs; a.ds = Ds; a.ht = Ht; a.dt = Dt; a.din = p->din; a.dout = p->dout;
        a.fs = p->fs; a.ft = p->ft;
        a.row_ptr = io.row_ptr; a.col_idx = io.col_idx; a.weight = io.weight;
        a.identity = identity; a.rows = rows_per_tile; a.pg = pg; a.ba = ba;
        tiled_kernel<bf16_t><<<dim3(tiles, Lt, 2), dim3(256), lds, st>>>(a);
      }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e);
  }
  return KVX_OK;
}

namespace {

// Rows of the staged path's intermediates for one group of contexts: row
// tiles of 128 per context; the largest over the call's groups.
int64_t staged_rows(const Call& c) {
  int64_t best = 0;
  for (int64_t b0 = 0; b0 < c.io.batch; b0 += kMaxBatch) {
    int64_t r = 0;
    for (int64_t b = b0; b < c.io.batch && b < b0 + kMaxBatch; ++b)
      r += (c.ttok[b] + kStageRows - 1) / kStageRows * kStageRows;
    best = r > best ? r : best;
  }
  return best;
}

// Workspace bytes per target layer: Z (K and V, hi and lo planes, bf16) and
// U (K and V, fp32).
size_t staged_layer_bytes(const kvx_plan* p, int64_t rows) {
  return size_t(2) * (size_t(2) * rows * p->din * sizeof(bf16_t) + size_t(rows) * p->dout * 4);
}

kvx_status staged_plan_ok(const kvx_plan* p) {
  if (p->kernel != kFused || p->precision == KVX_PREC_F16) return KVX_EUNSUPPORTED;
  return KVX_OK;
}

}  // namespace

extern "C" kvx_status kvx_staged_workspace_bytes(const kvx_plan* p, const kvx_io* io_in,
                                                 int32_t layers, size_t* bytes) {
  if (bytes) *bytes = 0;
  if (!p || !io_in || !bytes || layers < 1) return KVX_EINVAL;
  kvx_status s = staged_plan_ok(p);
  if (s != KVX_OK) return s;
  Call call;
  s = prepare_call(p, io_in, call);
  if (s != KVX_OK || call.rows == 0) return s;
  const int32_t lg = layers < p->tgt.n_layers ? layers : p->tgt.n_layers;
  *bytes = staged_layer_bytes(p, staged_rows(call)) * lg;
  return KVX_OK;
}

extern "C" kvx_status kvx_translate_staged(const kvx_plan* p, const kvx_io* io_in, void* workspace,
                                           size_t workspace_bytes, uint32_t stages,
                                           void* stream) {
  if (!p || !io_in) return KVX_EINVAL;
  if (stages == 0 || (stages & ~uint32_t(KVX_STAGE_ALL)) != 0) return KVX_EINVAL;
  kvx_status s = staged_plan_ok(p);
  if (s != KVX_OK) return s;
  Call call;
  s = prepare_call(p, io_in, call);
  if (s != KVX_OK || call.rows == 0) return s;
  const kvx_io& io = call.io;
  if (!rows_aligned16(io, 2)) return KVX_EUNSUPPORTED;
  if (!workspace || !aligned16(workspace)) return KVX_EINVAL;
  const int64_t Lt = p->tgt.n_layers, B = io.batch;
  const int64_t rows_max = staged_rows(call);
  const size_t per_layer = staged_layer_bytes(p, rows_max);
  int64_t lg = static_cast<int64_t>(workspace_bytes / per_layer);
  if (lg < 1) return KVX_ESHAPE;
  lg = lg < Lt ? lg : Lt;
  // a subset of the stages reads or leaves intermediates in the workspace,
  // so one pass must cover every layer and context
  if (stages != KVX_STAGE_ALL && (lg < Lt || B > kMaxBatch)) return KVX_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  s = validate_call(call, (stages & KVX_STAGE_POOL) != 0, (stages & KVX_STAGE_STORE) != 0, st);
  if (s != KVX_OK) return s;
  if (injected_launch_fault()) return hip_fail(hipErrorLaunchFailure);

  StagedArgs a{};
  a.ss = Strides{io.src_stride[0], io.src_stride[1], io.src_stride[2], io.src_stride[3]};
  a.ts = Strides{io.tgt_stride[0], io.tgt_stride[1], io.tgt_stride[2], io.tgt_stride[3]};
  a.wp[0] = static_cast<const bf16x8*>(p->w[0]);
  a.wp[1] = static_cast<const bf16x8*>(p->w[1]);
  a.bias[0] = p->bias[0];
  a.bias[1] = p->bias[1];
  a.layer_map = p->layer_map;
  a.fs = p->fs;
  a.ft = p->ft;
  a.row_ptr = call.identity ? nullptr : io.row_ptr;
  a.col_idx = io.col_idx;
  a.weight = io.weight;
  a.mix = p->mix;
  a.hs = p->src.n_kv_heads;
  a.ds = p->src.head_dim;
  a.ht = p->tgt.n_kv_heads;
  a.dt = p->tgt.head_dim;
  a.din = p->din;
  a.dout = p->dout;
  // operands as the fused kernel's precision modes round them: two planes
  // for computed operands unless the plan rounds them once (BF16); an
  // identity-aligned V is exact
  const bool split = p->precision != KVX_PREC_BF16;
  a.planes[0] = split ? 2 : 1;
  a.planes[1] = split && !call.identity ? 2 : 1;
  int64_t row_base = 0;
  for (int64_t b0 = 0; b0 < B; b0 += kMaxBatch) {
    const int nb = static_cast<int>(B - b0 < kMaxBatch ? B - b0 : kMaxBatch);
    BatchArgs ba{};
    ba.n = nb;
    int tiles = 0;
    for (int i = 0; i < nb; ++i) {
      ba.tile_start[i] = tiles;
      ba.t_tgt[i] = call.ttok[b0 + i];
      ba.row_base[i] = static_cast<int32_t>(row_base);
      row_base += call.ttok[b0 + i];
      tiles += (call.ttok[b0 + i] + kStageRows - 1) / kStageRows;
    }
    ba.tile_start[nb] = tiles;
    if (tiles == 0) continue;
    a.ba = ba;
    a.tiles = tiles;
    a.rows_p = tiles * kStageRows;
    a.src[0] = static_cast<const bf16_t*>(io.src_k) + b0 * io.src_stride[1];
    a.src[1] = static_cast<const bf16_t*>(io.src_v) + b0 * io.src_stride[1];
    // paged: blocks are shared by all contexts; the table row moves instead
    const int64_t toff = call.paged ? 0 : b0 * io.tgt_stride[1];
    a.tgt[0] = static_cast<bf16_t*>(io.tgt_k) + toff;
    a.tgt[1] = static_cast<bf16_t*>(io.tgt_v) + toff;
    a.pg = Paging{call.paged ? io.block_table + b0 * io.max_blocks : nullptr,
                  call.paged ? io.block_size : 1, call.paged ? io.max_blocks : 0};
    for (int64_t l0 = 0; l0 < Lt; l0 += lg) {
      a.l0 = static_cast<int32_t>(l0);
      a.nl = static_cast<int32_t>(Lt - l0 < lg ? Lt - l0 : lg);
      a.z = static_cast<bf16_t*>(workspace);
      a.u = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                     size_t(a.nl) * 2 * 2 * a.rows_p * p->din * sizeof(bf16_t));
      if (stages & KVX_STAGE_POOL) launch_stage_pool(a, st);
      if (stages & KVX_STAGE_PROJECT) launch_stage_project(a, st);
      if (stages & KVX_STAGE_STORE) launch_stage_store(a, st);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(e);
    }
  }
  return KVX_OK;
}
