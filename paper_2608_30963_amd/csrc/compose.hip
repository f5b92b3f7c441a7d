// compose.hip -- translator variants of kvx.h (kvx_plan_create_factored):
// a low-rank translator W = U V (Section 5: low-dimensional latent adapters)
// or a fixed-weight mixture W = sum_k alpha_k W_k, b = sum_k alpha_k b_k
// (Section 2.2: a mixture of translator modules), composed on the device in
// fp32 and rounded once to the plan's dtype; the dense plan is then created
// from the composed weights.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "common.h"
#include "kvx.h"

using namespace kvx;

namespace {

constexpr int kMaxMix = 32;
constexpr int kCT = 16;  // output tile edge of the low-rank product

struct MixArgs {
  int32_t k;
  float alpha[kMaxMix];
};

// W[l] = U[l] V[l]: U [dout][r], V [r][din]; one 16 x 16 output tile per
// workgroup (256 threads), r streamed through LDS in slices of 16.
template <typename T>
__global__ void __launch_bounds__(256) compose_lowrank(const T* U, const T* V, T* W, int dout,
                                                       int din, int r) {
  __shared__ float us[kCT][kCT + 1];
  __shared__ float vs[kCT][kCT + 1];
  const int l = blockIdx.z;
  const int o0 = blockIdx.y * kCT, i0 = blockIdx.x * kCT;
  const int ty = threadIdx.x / kCT, tx = threadIdx.x % kCT;
  const T* Ul = U + static_cast<int64_t>(l) * dout * r;
  const T* Vl = V + static_cast<int64_t>(l) * r * din;
  float acc = 0.f;
  for (int k0 = 0; k0 < r; k0 += kCT) {
    const int uo = o0 + ty, uk = k0 + tx;
    us[ty][tx] = (uo < dout && uk < r) ? load_f32<T>(Ul + static_cast<int64_t>(uo) * r + uk) : 0.f;
    const int vk = k0 + ty, vi = i0 + tx;
    vs[ty][tx] = (vk < r && vi < din) ? load_f32<T>(Vl + static_cast<int64_t>(vk) * din + vi) : 0.f;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kCT; ++k) acc += us[ty][k] * vs[k][tx];
    __syncthreads();
  }
  const int o = o0 + ty, i = i0 + tx;
  if (o < dout && i < din)
    W[(static_cast<int64_t>(l) * dout + o) * din + i] = store_cvt<T>(acc);
}

// out[e] = sum_k alpha_k in[k * n + e] over n elements (fp32 accumulation).
template <typename TI, typename TO>
__global__ void __launch_bounds__(256) compose_mixture(const TI* in, TO* out, int64_t n,
                                                       MixArgs m) {
  for (int64_t e = blockIdx.x * 256LL + threadIdx.x; e < n; e += gridDim.x * 256LL) {
    float acc = 0.f;
    for (int k = 0; k < m.k; ++k) acc += m.alpha[k] * load_f32<TI>(in + k * n + e);
    out[e] = store_cvt<TO>(acc);
  }
}

}  // namespace

extern "C" kvx_status kvx_plan_create_factored(const kvx_plan_desc* d, const kvx_factors* f,
                                               kvx_plan** out) {
  if (out) *out = nullptr;
  if (!d || !f || !out || !d->layer_map) return KVX_EINVAL;
  if (d->dtype != KVX_F32 && d->dtype != KVX_BF16) return KVX_EINVAL;
  if (d->precision != KVX_PREC_BF16X2 && d->precision != KVX_PREC_BF16 &&
      d->precision != KVX_PREC_F16)
    return KVX_EINVAL;
  if (d->src.n_layers <= 0 || d->tgt.n_layers <= 0 || d->src.n_kv_heads <= 0 ||
      d->tgt.n_kv_heads <= 0 || d->src.head_dim <= 0 || d->tgt.head_dim <= 0 || d->mix < 1)
    return KVX_EINVAL;
  const int64_t lt = d->tgt.n_layers;
  const int64_t din = int64_t(d->mix) * d->src.n_kv_heads * d->src.head_dim;
  const int64_t dout = int64_t(d->tgt.n_kv_heads) * d->tgt.head_dim;
  if (din > (1 << 20) || dout > (1 << 20) || lt > 65535) return KVX_ESHAPE;
  const size_t esz = d->dtype == KVX_F32 ? 4 : 2;
  const int64_t nw = lt * dout * din;
  if (f->kind == KVX_FACTORS_LOWRANK) {
    if (f->rank < 1 || !f->u_k || !f->u_v || !f->v_k || !f->v_v) return KVX_EINVAL;
    if (f->rank > (1 << 20)) return KVX_ESHAPE;
  } else if (f->kind == KVX_FACTORS_MIXTURE) {
    if (f->n_mix < 1 || !f->alpha || !f->w_k || !f->w_v) return KVX_EINVAL;
    if (f->n_mix > kMaxMix) return KVX_EUNSUPPORTED;
    for (int k = 0; k < f->n_mix; ++k)
      if (!std::isfinite(f->alpha[k])) return KVX_EINVAL;
  } else {
    return KVX_EINVAL;
  }

  // composed W_k, W_v (plan dtype) and, for a mixture, b_k and b_v (fp32),
  // each bias composed only when its member biases are given (NULL: zero)
  const bool mix = f->kind == KVX_FACTORS_MIXTURE;
  const bool mixb[2] = {mix && f->b_k, mix && f->b_v};
  const size_t wbytes = size_t(nw) * esz;
  const size_t bbytes = size_t(lt) * dout * sizeof(float);
  void* buf = nullptr;
  hipError_t e = hipMalloc(&buf, 2 * wbytes + 2 * bbytes);
  if (e != hipSuccess) return hip_status(e);
  char* base = static_cast<char*>(buf);
  void* w[2] = {base, base + wbytes};
  float* b[2] = {mixb[0] ? reinterpret_cast<float*>(base + 2 * wbytes) : nullptr,
                 mixb[1] ? reinterpret_cast<float*>(base + 2 * wbytes + bbytes) : nullptr};
  if (f->kind == KVX_FACTORS_LOWRANK) {
    const void* U[2] = {f->u_k, f->u_v};
    const void* V[2] = {f->v_k, f->v_v};
    const dim3 grid(static_cast<unsigned>((din + kCT - 1) / kCT),
                    static_cast<unsigned>((dout + kCT - 1) / kCT), static_cast<unsigned>(lt));
    for (int kv = 0; kv < 2; ++kv) {
      if (d->dtype == KVX_F32)
        compose_lowrank<float><<<grid, dim3(256)>>>(static_cast<const float*>(U[kv]),
                                                    static_cast<const float*>(V[kv]),
                                                    static_cast<float*>(w[kv]),
                                                    static_cast<int>(dout), static_cast<int>(din),
                                                    f->rank);
      else
        compose_lowrank<bf16_t><<<grid, dim3(256)>>>(static_cast<const bf16_t*>(U[kv]),
                                                     static_cast<const bf16_t*>(V[kv]),
                                                     static_cast<bf16_t*>(w[kv]),
                                                     static_cast<int>(dout),
                                                     static_cast<int>(din), f->rank);
    }
  } else {
    MixArgs m{};
    m.k = f->n_mix;
    for (int k = 0; k < f->n_mix; ++k) m.alpha[k] = static_cast<float>(f->alpha[k]);
    const void* W[2] = {f->w_k, f->w_v};
    const unsigned blocks = static_cast<unsigned>(std::min<int64_t>((nw + 255) / 256, 65536));
    for (int kv = 0; kv < 2; ++kv) {
      if (d->dtype == KVX_F32)
        compose_mixture<float, float><<<blocks, dim3(256)>>>(
            static_cast<const float*>(W[kv]), static_cast<float*>(w[kv]), nw, m);
      else
        compose_mixture<bf16_t, bf16_t><<<blocks, dim3(256)>>>(
            static_cast<const bf16_t*>(W[kv]), static_cast<bf16_t*>(w[kv]), nw, m);
    }
    const float* B[2] = {f->b_k, f->b_v};
    const int64_t nb = lt * dout;
    const unsigned bb = static_cast<unsigned>(std::min<int64_t>((nb + 255) / 256, 65536));
    for (int kv = 0; kv < 2; ++kv)
      if (mixb[kv]) compose_mixture<float, float><<<bb, dim3(256)>>>(B[kv], b[kv], nb, m);
  }
  e = hipGetLastError();
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipFree(buf);
    return hip_status(e);
  }
  kvx_plan_desc dd = *d;
  dd.w_k = w[0];
  dd.w_v = w[1];
  if (f->kind == KVX_FACTORS_MIXTURE) {
    dd.b_k = b[0];
    dd.b_v = b[1];
  }
  const kvx_status st = kvx_plan_create(&dd, out);
  (void)hipFree(buf);
  return st;
}
