// Plain causal prefill in the explicit (non-absorbed) form, as a second,
// independent device-side implementation of App. C Eq. (C.2), (C.6),
// (C.11)-(C.13) with the latent-space gate of Sec. 3.1 Eq. (3)-(5).
//
//   kv kernel:   K[h][t] = [W_UK[h] c~_t ; k^R_t],  V[h][t] = W_UV[h] c~_t   (fp32 workspace)
//   attn kernel: out[t][h] = sum_{j<=t} softmax_j(tau q_t,h . K[h][j]) V[h][j]
// Deliberately simple: one work-group per (t, h), no tiling.
#include <hip/hip_runtime.h>

#include <cmath>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"
#include "prefill_mfma.h"
#include "prefill_explicit.h"

namespace egmla {

constexpr int kPrefillThreads = 256;

template <bool BF16>
__global__ __launch_bounds__(kPrefillThreads) void prefill_kv_kernel(const void* __restrict__ latent,
                                                                     const int32_t* __restrict__ token_ids,
                                                                     const void* __restrict__ gate,
                                                                     const void* __restrict__ w_uk,
                                                                     const void* __restrict__ w_uv,
                                                                     float* __restrict__ K, float* __restrict__ Vv,
                                                                     int T, int DH, int DV, int DC, int DR, int Vocab) {
  extern __shared__ float cg[];  // gated latent [DC]
  const int t = blockIdx.x, h = blockIdx.y;
  const int DQ = DC + DR;
  const int DK = DH + DR;
  const int id = clamp_id(token_ids[t], Vocab);
  for (int c = threadIdx.x; c < DC; c += kPrefillThreads)
    cg[c] = ld<BF16>(latent, static_cast<int64_t>(t) * DQ + c) * ld<BF16>(gate, static_cast<int64_t>(id) * DC + c);
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t kb = (static_cast<int64_t>(h) * T + t) * DK;
  const int64_t vb = (static_cast<int64_t>(h) * T + t) * DV;
  for (int o = w; o < DH + DV; o += kPrefillThreads / 64) {
    const bool is_k = o < DH;
    const int64_t rb = is_k ? (static_cast<int64_t>(h) * DH + o) * DC : (static_cast<int64_t>(h) * DV + (o - DH)) * DC;
    const void* wp = is_k ? w_uk : w_uv;
    float acc = 0.f;
    for (int c = lane; c < DC; c += 64) acc = fmaf(ld<BF16>(wp, rb + c), cg[c], acc);
    acc = wave_sum(acc);
    if (lane == 0) {
      if (is_k) K[kb + o] = acc;
      else Vv[vb + o - DH] = acc;
    }
  }
  for (int r = threadIdx.x; r < DR; r += kPrefillThreads)
    K[kb + DH + r] = ld<BF16>(latent, static_cast<int64_t>(t) * DQ + DC + r);
}

template <bool BF16>
__global__ __launch_bounds__(kPrefillThreads) void prefill_attn_kernel(const void* __restrict__ q,
                                                                       const float* __restrict__ K,
                                                                       const float* __restrict__ Vv,
                                                                       void* __restrict__ out, int T, int H, int DH,
                                                                       int DV, int DR, float scale) {
  extern __shared__ float sm[];  // q [DK], scores [T], reduction [kPrefillThreads / 64]
  const int DK = DH + DR;
  float* qs = sm;
  float* sc = qs + DK;
  float* red = sc + T;
  const int t = blockIdx.x, h = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  for (int k = tid; k < DK; k += kPrefillThreads) qs[k] = ld<BF16>(q, (static_cast<int64_t>(t) * H + h) * DK + k);
  __syncthreads();
  const int n = t + 1;  // causal: keys 0..t
  float mx = -INFINITY;
  for (int j = tid; j < n; j += kPrefillThreads) {
    const float* kr = K + (static_cast<int64_t>(h) * T + j) * DK;
    float dot = 0.f;
    for (int k = 0; k < DK; ++k) dot = fmaf(qs[k], kr[k], dot);
    dot *= scale;
    sc[j] = dot;
    mx = fmaxf(mx, dot);
  }
  mx = wave_max(mx);
  if (lane == 0) red[w] = mx;
  __syncthreads();
  mx = red[0];
  for (int i = 1; i < kPrefillThreads / 64; ++i) mx = fmaxf(mx, red[i]);
  __syncthreads();
  float sum = 0.f;
  for (int j = tid; j < n; j += kPrefillThreads) {
    const float e = expf(sc[j] - mx);
    sc[j] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  if (lane == 0) red[w] = sum;
  __syncthreads();
  sum = 0.f;
  for (int i = 0; i < kPrefillThreads / 64; ++i) sum += red[i];
  const float inv = 1.f / sum;
  for (int v = tid; v < DV; v += kPrefillThreads) {
    float acc = 0.f;
    for (int j = 0; j < n; ++j) acc = fmaf(sc[j], Vv[(static_cast<int64_t>(h) * T + j) * DV + v], acc);
    st<BF16>(out, (static_cast<int64_t>(t) * H + h) * DV + v, acc * inv);
  }
}

}  // namespace egmla

using namespace egmla;

namespace {
template <bool BF16>
eg_mla_status launch_prefill(const eg_mla_dims& d, int T, const void* q, const void* latent, const int32_t* ids,
                             const void* gate, const void* w_uk, const void* w_uv, float* K, float* Vv, void* out,
                             hipStream_t stream) {
  dim3 grid(T, d.num_heads);
  hipLaunchKernelGGL(prefill_kv_kernel<BF16>, grid, dim3(kPrefillThreads), sizeof(float) * d.latent_dim, stream,
                     latent, ids, gate, w_uk, w_uv, K, Vv, T, d.head_dim, d.v_head_dim, d.latent_dim, d.rope_dim,
                     d.vocab_size);
  if (hipGetLastError() != hipSuccess) return EG_MLA_ERR_HIP;
  const size_t lds = sizeof(float) * (static_cast<size_t>(d.head_dim + d.rope_dim) + T + kPrefillThreads / 64);
  if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(prefill_attn_kernel<BF16>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         static_cast<int>(lds)) != hipSuccess)
    return EG_MLA_ERR_HIP;
  hipLaunchKernelGGL(prefill_attn_kernel<BF16>, grid, dim3(kPrefillThreads), lds, stream, q, K, Vv, out, T,
                     d.num_heads, d.head_dim, d.v_head_dim, d.rope_dim, softmax_scale(d));
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
}  // namespace

extern "C" eg_mla_status eg_mla_prefill_ref(const eg_mla_dims* dims, int32_t seq_len, const void* q,
                                            const void* latent, const int32_t* token_ids, const void* gate_table,
                                            const void* w_uk, const void* w_uv, void* workspace,
                                            size_t workspace_bytes, void* out, void* stream_) {
  eg_mla_status st = validate_prefill(dims, seq_len, q, latent, token_ids, gate_table, w_uk, w_uv, workspace,
                                      workspace_bytes, out);
  if (st != EG_MLA_OK || seq_len == 0) return st;
  const eg_mla_dims& d = *dims;
  const size_t T = static_cast<size_t>(seq_len);
  float* K = static_cast<float*>(workspace);
  float* Vv = reinterpret_cast<float*>(static_cast<unsigned char*>(workspace) +
                                       align_up(static_cast<size_t>(d.num_heads) * T * (d.head_dim + d.rope_dim) * 4));
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  (void)hipGetLastError();
  if (d.dtype == EG_MLA_BF16)
    return launch_prefill<true>(d, seq_len, q, latent, token_ids, gate_table, w_uk, w_uv, K, Vv, out, stream);
  return launch_prefill<false>(d, seq_len, q, latent, token_ids, gate_table, w_uk, w_uv, K, Vv, out, stream);
}

extern "C" eg_mla_status eg_mla_prefill_varlen(const eg_mla_dims* dims, int32_t batch, int32_t total_tokens,
                                               const int32_t* cu_seqlens, const void* q, const void* latent,
                                               const int32_t* token_ids, const void* gate_table, const void* w_uk,
                                               const void* w_uv, void* workspace, size_t workspace_bytes, void* out,
                                               void* stream_) {
  eg_mla_status st = validate_prefill_varlen(dims, batch, total_tokens, cu_seqlens, q, latent, token_ids,
                                             gate_table, w_uk, w_uv, workspace, workspace_bytes, out);
  if (st != EG_MLA_OK || total_tokens == 0) return st;
  const eg_mla_dims& d = *dims;
  const int T = total_tokens;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  (void)hipGetLastError();
  const PrefillVarlenLayout L = prefill_varlen_layout(d, T);
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  int32_t* seq_start = reinterpret_cast<int32_t*>(ws + L.off_seq_start);
  uint16_t* qf = reinterpret_cast<uint16_t*>(ws + L.off_qf);
  uint16_t* olat = reinterpret_cast<uint16_t*>(ws + L.off_olat);

  hipLaunchKernelGGL(prefill_seqmap_kernel, dim3((T + 255) / 256), dim3(256), 0, stream, cu_seqlens, batch, T,
                     seq_start);
  if (!prefill_varlen_absorbed(d)) {
    // explicit form: K^C and V per head (fp16), then the attention per head
    uint16_t* kc = reinterpret_cast<uint16_t*>(ws + L.off_qf);
    uint16_t* vv = reinterpret_cast<uint16_t*>(ws + L.off_olat);
    // the gated latent of every token, once, as bf16 hi + lo rows
    uint16_t* ct_hi = reinterpret_cast<uint16_t*>(ws + L.off_ct);
    uint16_t* ct_lo = reinterpret_cast<uint16_t*>(ws + L.off_ct + align_up(static_cast<size_t>(T) * d.latent_dim * 2));
    const dim3 gate_grid(static_cast<unsigned>((static_cast<int64_t>(T) * (d.latent_dim / 8) + 255) / 256));
    hipLaunchKernelGGL(prefill_x_gate_kernel, gate_grid, dim3(256), 0, stream, static_cast<const uint16_t*>(latent),
                       token_ids, static_cast<const uint16_t*>(gate_table), ct_hi, ct_lo, T, d.latent_dim,
                       d.vocab_size);
    hipLaunchKernelGGL(prefill_x_proj_kernel, dim3((T + kPxTok - 1) / kPxTok, d.num_heads), dim3(256), 0, stream,
                       ct_hi, ct_lo, static_cast<const uint16_t*>(w_uk), static_cast<const uint16_t*>(w_uv), kc, vv, T,
                       d.latent_dim);
    PrefillXArgs x;
    x.q = static_cast<const uint16_t*>(q);
    x.latent = static_cast<const uint16_t*>(latent);
    x.kc = kc;
    x.vv = vv;
    x.seq_start = seq_start;
    x.out = static_cast<uint16_t*>(out);
    x.T = T;
    x.H = d.num_heads;
    x.DC = d.latent_dim;
    x.scale_log2 = softmax_scale(d) * 1.4426950408889634f;
    hipLaunchKernelGGL(prefill_x_attn_kernel, dim3(((T + kPxQTok - 1) / kPxQTok) * d.num_heads), dim3(256), 0,
                       stream, x);
    return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
  }
  // q_lat (bf16) and q^R for every token
  const int side_wgs = ((T + kPfUvTokens - 1) / kPfUvTokens + kPfSideChunks - 1) / kPfSideChunks;
  hipLaunchKernelGGL(prefill_absorb_kernel, dim3(side_wgs, d.num_heads), dim3(256), 0, stream,
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(w_uk), qf, T);
  // the gated latent of every token, once (keys and values of every head)
  uint16_t* ct = reinterpret_cast<uint16_t*>(ws + L.off_ct);
  const dim3 gate_grid(static_cast<unsigned>((static_cast<int64_t>(T) * 16 + 255) / 256));
  hipLaunchKernelGGL(prefill_gate_kernel, gate_grid, dim3(256), 0, stream, static_cast<const uint16_t*>(latent),
                     token_ids, static_cast<const uint16_t*>(gate_table), ct, T, d.vocab_size);
  PrefillArgs a;
  a.qf = qf;
  a.latent = static_cast<const uint16_t*>(latent);
  a.ct = ct;
  a.seq_start = seq_start;
  a.olat = olat;
  a.T = T;
  a.scale_log2 = softmax_scale(d) * 1.4426950408889634f;
  hipLaunchKernelGGL(prefill_attn_mfma_kernel, dim3((T + kPfTokens - 1) / kPfTokens), dim3(kPfThreads), 0, stream,
                     a);
  hipLaunchKernelGGL(prefill_uv_kernel, dim3(side_wgs, d.num_heads), dim3(256), 0, stream,
                     olat, static_cast<const uint16_t*>(w_uv), static_cast<uint16_t*>(out), T);
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
