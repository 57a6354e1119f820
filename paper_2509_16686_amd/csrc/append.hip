// EG-MLA cache append on gfx950: compress new tokens into latent-cache rows.
//
// For each new token (Sec. 3.1 Eq. (1), App. C Eq. (C.10)):
//   [c | r] = W_DKV x       (W_DKV stacks W^DKV and W^KR: [d_c + d_r, hidden])
//   c       = RMSNorm(c) * kv_norm_w      (optional latent norm, eps 1e-6)
//   k^R     = RoPE(r, position)           (adjacent pairs, angle pos * theta^(-2m/d_r))
// and the row [c | k^R] plus the token id are stored at the token's slot.
// One work-group (256 threads) per token; each wave computes output features
// as coalesced dot products over the hidden dimension.
#include <hip/hip_runtime.h>

#include <cmath>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr int kAppendThreads = 256;
constexpr float kRmsEps = 1e-6f;

template <bool BF16>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(const void* __restrict__ x,
                                                                const int32_t* __restrict__ token_ids,
                                                                const int32_t* __restrict__ positions,
                                                                const int32_t* __restrict__ slots,
                                                                const void* __restrict__ w_dkv,
                                                                const void* __restrict__ kv_norm_w, float theta,
                                                                void* __restrict__ cache, int32_t* __restrict__ ids,
                                                                int64_t num_slots, int hidden, int DC, int DR) {
  extern __shared__ float smem[];  // x row [hidden], y [DC + DR], reduction [4]
  float* xs = smem;
  float* ys = xs + hidden;
  float* red = ys + DC + DR;
  const int i = blockIdx.x;
  const int64_t slot = slots[i];
  if (slot < 0 || slot >= num_slots) return;  // out-of-range destination: skipped
  const int DQ = DC + DR;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int k = tid; k < hidden; k += kAppendThreads) xs[k] = ld<BF16>(x, static_cast<int64_t>(i) * hidden + k);
  __syncthreads();
  // y = W_DKV x: one output feature per wave at a time, lanes stride the hidden dim
  for (int o = w; o < DQ; o += kAppendThreads / 64) {
    const int64_t rb = static_cast<int64_t>(o) * hidden;
    float acc = 0.f;
    for (int k = lane; k < hidden; k += 64) acc = fmaf(ld<BF16>(w_dkv, rb + k), xs[k], acc);
    acc = wave_sum(acc);
    if (lane == 0) ys[o] = acc;
  }
  __syncthreads();
  float inv_rms = 1.f;
  if (kv_norm_w) {
    if (w == 0) {
      float ss = 0.f;
      for (int c = lane; c < DC; c += 64) ss = fmaf(ys[c], ys[c], ss);
      ss = wave_sum(ss);
      if (lane == 0) red[0] = 1.f / sqrtf(ss / static_cast<float>(DC) + kRmsEps);
    }
    __syncthreads();
    inv_rms = red[0];
  }
  const int64_t rbase = slot * DQ;
  for (int c = tid; c < DC; c += kAppendThreads) {
    float v = ys[c];
    if (kv_norm_w) v = v * inv_rms * ld<BF16>(kv_norm_w, c);
    st<BF16>(cache, rbase + c, v);
  }
  // RoPE on adjacent pairs; the angle is formed in fp64 so large positions keep full accuracy
  const double pos = static_cast<double>(positions[i]);
  for (int m = tid; m < DR / 2; m += kAppendThreads) {
    const double inv_freq = pow(static_cast<double>(theta), -2.0 * m / static_cast<double>(DR));
    double sn, cs;
    sincos(pos * inv_freq, &sn, &cs);
    const float x0 = ys[DC + 2 * m], x1 = ys[DC + 2 * m + 1];
    st<BF16>(cache, rbase + DC + 2 * m, static_cast<float>(x0 * cs - x1 * sn));
    st<BF16>(cache, rbase + DC + 2 * m + 1, static_cast<float>(x0 * sn + x1 * cs));
  }
  if (tid == 0) ids[slot] = token_ids[i];
}

}  // namespace egmla

using namespace egmla;

extern "C" eg_mla_status eg_mla_append(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden, const void* x,
                                       const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                                       const void* w_dkv, const void* kv_norm_w, float rope_theta,
                                       void* latent_cache, int32_t* token_id_cache, int64_t num_slots,
                                       void* stream_) {
  eg_mla_status st = validate_append(dims, n_tokens, hidden, x, token_ids, positions, slots, w_dkv, latent_cache,
                                     token_id_cache, num_slots);
  if (st != EG_MLA_OK || n_tokens == 0) return st;
  const eg_mla_dims& d = *dims;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const float theta = rope_theta > 0.f ? rope_theta : 10000.f;
  const size_t lds = sizeof(float) * (static_cast<size_t>(hidden) + d.latent_dim + d.rope_dim + 4);
  (void)hipGetLastError();
  if (d.dtype == EG_MLA_BF16) {
    if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(append_kernel<true>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           static_cast<int>(lds)) != hipSuccess)
      return EG_MLA_ERR_HIP;
    hipLaunchKernelGGL(append_kernel<true>, dim3(n_tokens), dim3(kAppendThreads), lds, stream, x, token_ids,
                       positions, slots, w_dkv, kv_norm_w, theta, latent_cache, token_id_cache, num_slots, hidden,
                       d.latent_dim, d.rope_dim);
  } else {
    if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(append_kernel<false>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           static_cast<int>(lds)) != hipSuccess)
      return EG_MLA_ERR_HIP;
    hipLaunchKernelGGL(append_kernel<false>, dim3(n_tokens), dim3(kAppendThreads), lds, stream, x, token_ids,
                       positions, slots, w_dkv, kv_norm_w, theta, latent_cache, token_id_cache, num_slots, hidden,
                       d.latent_dim, d.rope_dim);
  }
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
