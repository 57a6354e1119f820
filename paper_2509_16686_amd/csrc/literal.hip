// Decode with the paper-literal gate on gfx950 (Sec. 3.1 Eq. (2)-(5) as
// printed, and the model listing's order): per cached token j,
//   kv_j = W^UKV c_j           (per head h: [W_UK[h] c_j ; W_UV[h] c_j], head-major)
//   x_j  = kv_j (.) g_j        (or kv_j + g_j: the ablation), g_j = G[i_j] of width H (d_h + d_v)
//   y_j  = LN(x_j)             (over all H (d_h + d_v) dims, weight and bias; or none: the ablation)
// and per head k_j = [y_j[h, :d_h] ; k^R_j], v_j = y_j[h, d_h:],
//   out[b, h] = sum_j softmax_j(q_h . k_j / sqrt(d_h + d_r)) v_j.
// The gate sits after the up-projection and the LayerNorm spans all heads, so
// nothing can be absorbed: every step up-projects every cached token.
//
// Two kernels (bf16 storage, d_c = d_h = d_v = 128, d_r = 64, any head count):
//  1. literal_kv_kernel: for the cached rows of every sequence, x = kv (.) g
//     on v_mfma_f32_32x32x16_bf16 (A: 32 rows of W_UK[h] or W_UV[h] from LDS,
//     where one head's 256 rows are staged with coalesced loads while the
//     previous head computes; B: the row's latent, in registers), written in
//     bf16 to the workspace by cache row, with the row's mean and
//     1/sqrt(var + eps) over all dims (moments summed in fp32 from the
//     unrounded products).
//  2. literal_attn_kernel: one work-group per (sequence, head).  The
//     LayerNorm is applied while reading: a score is
//     rstd (sum_d q_d w_d x_d - mu sum_d q_d w_d) + sum_d q_d b_d + q^R . k^R,
//     and the value sum is w_v (sum_j a_j x_j - sum_j a_j mu_j) / sum_j p_j + b_v
//     with a_j = p_j rstd_j, so the normalised rows are never stored.
#include <hip/hip_runtime.h>

#include <cmath>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr int kLtDC = 128, kLtDH = 128, kLtDV = 128, kLtDR = 64;
constexpr int kLtHeadW = kLtDH + kLtDV;  // gated dims per head
constexpr float kLtLnEps = 1e-5f;        // the listing's LayerNorm default
typedef __attribute__((ext_vector_type(16))) float lt_f32x16_t;

constexpr int kLtWRow = kLtDC + 8;                  // padded LDS row of W (272 bytes: 16-lane reads hit 16 bank groups)
constexpr int kLtWLds = kLtHeadW * kLtWRow * 2;      // one head's W_UK and W_UV rows in LDS (69.6 KB)

__global__ __launch_bounds__(256, 2) void literal_kv_kernel(const uint16_t* __restrict__ cache,
                                                            const int32_t* __restrict__ ids,
                                                            const uint16_t* __restrict__ gate,
                                                            const uint16_t* __restrict__ w_uk,
                                                            const uint16_t* __restrict__ w_uv,
                                                            const int32_t* __restrict__ seq_lens,
                                                            const int32_t* __restrict__ page_table, int P,
                                                            int max_pages, int64_t num_slots, int H, int V,
                                                            int add_mode, uint16_t* __restrict__ Y,
                                                            float2* __restrict__ stats) {
  extern __shared__ __attribute__((aligned(16))) uint16_t wsh[];  // [256 rows: W_UK[h] then W_UV[h]][kLtWRow]
  const int b = blockIdx.y;
  const int L = clamp_len(seq_lens[b], P * max_pages);
  const int j0 = blockIdx.x * 128;
  if (j0 >= L) return;  // whole work-group, before any barrier
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int j = j0 + 32 * w + r32;
  const bool ok = j < L;  // positions past the sequence repeat its last token and are not stored
  const int64_t row = cache_slot(page_table, b, min(j, L - 1), P, max_pages, num_slots);
  const int id = clamp_id(ids[row], V);
  const int width = H * kLtHeadW;
  bf16x8_t cb[kLtDC / 16];  // B operand: the row's latent, dims 16 c + 8 h .. + 7
#pragma unroll
  for (int c = 0; c < kLtDC / 16; ++c)
    cb[c] = *reinterpret_cast<const bf16x8_t*>(cache + row * (kLtDC + kLtDR) + 16 * c + 8 * h);
  const uint16_t* grow = gate + static_cast<int64_t>(id) * width + 4 * h;
  uint16_t* yrow = Y + row * width + 4 * h;

  // a head's 256 weight rows (W_UK[h] then W_UV[h]) as 4096 16-byte pieces:
  // thread tid takes pieces tid + 256 i (row (tid + 256 i) / 16: 16 lanes read one 256-byte row)
  u32x4_t stage[16];
  auto fetch = [&](int head) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int p = tid + 256 * i, r = p >> 4, k8 = (p & 15) * 8;
      const uint16_t* src = (r < kLtDH ? w_uk + (static_cast<int64_t>(head) * kLtDH + r) * kLtDC
                                       : w_uv + (static_cast<int64_t>(head) * kLtDV + r - kLtDH) * kLtDC) + k8;
      stage[i] = *reinterpret_cast<const u32x4_t*>(src);
    }
  };
  auto put = [&]() {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int p = tid + 256 * i;
      *reinterpret_cast<u32x4_t*>(wsh + (p >> 4) * kLtWRow + (p & 15) * 8) = stage[i];
    }
  };
  float s1 = 0.f, s2 = 0.f;
  fetch(0);
  for (int head = 0; head < H; ++head) {
    __syncthreads();  // every wave is done with the previous head's rows
    put();
    __syncthreads();
    if (head + 1 < H) fetch(head + 1);  // travels while this head's 8 blocks compute
#pragma unroll 2
    for (int blk = 0; blk < kLtHeadW / 32; ++blk) {  // 32 outputs: LDS rows 32 blk .. + 31
      const int ob = head * (kLtHeadW / 32) + blk;
      u32x2_t gv[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) gv[q] = *reinterpret_cast<const u32x2_t*>(grow + 32 * ob + 8 * q);
      lt_f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
      const uint16_t* arow = wsh + (32 * blk + r32) * kLtWRow + 8 * h;
#pragma unroll
      for (int c = 0; c < kLtDC / 16; ++c)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8_t*>(arow + 16 * c), cb[c], acc,
                                                      0, 0, 0);
      // lane holds outputs 32 ob + 8 q + 4 h + e of its row in acc[4 q + e]
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float x[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float g = (e & 1) ? bf16_hi(gv[q][e >> 1]) : bf16_lo(gv[q][e >> 1]);
          x[e] = add_mode ? acc[4 * q + e] + g : acc[4 * q + e] * g;
          s1 += x[e];
          s2 = fmaf(x[e], x[e], s2);
        }
        if (ok)
          *reinterpret_cast<u32x2_t*>(yrow + 32 * ob + 8 * q) = u32x2_t{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
      }
    }
  }
  // lanes r32 and r32 + 32 hold the two halves of the row's outputs
  const uint32_t u1 = __float_as_uint(s1), u2 = __float_as_uint(s2);
  const auto t1 = __builtin_amdgcn_permlane32_swap(u1, u1, false, false);
  const auto t2 = __builtin_amdgcn_permlane32_swap(u2, u2, false, false);
  const float m1 = (__uint_as_float(t1[0]) + __uint_as_float(t1[1])) / static_cast<float>(width);
  const float m2 = (__uint_as_float(t2[0]) + __uint_as_float(t2[1])) / static_cast<float>(width);
  if (ok && h == 0) stats[row] = make_float2(m1, 1.0f / sqrtf(fmaxf(m2 - m1 * m1, 0.f) + kLtLnEps));
}

__global__ __launch_bounds__(256) void literal_attn_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ cache,
                                                           const uint16_t* __restrict__ Y,
                                                           const float2* __restrict__ stats,
                                                           const uint16_t* __restrict__ ln_w,
                                                           const uint16_t* __restrict__ ln_b, int use_ln,
                                                           const int32_t* __restrict__ seq_lens,
                                                           const int32_t* __restrict__ page_table, int P,
                                                           int max_pages, int64_t num_slots, int H, float scale,
                                                           uint16_t* __restrict__ out) {
  extern __shared__ float sm[];  // qa[128] qb-sum, qr[64], wv[128], bv[128], red[16], acc[4][128], p[L]
  float* qa = sm;             // q_d w_d (key part)
  float* qr = qa + kLtDH;     // q^R
  float* wv = qr + kLtDR;     // value-part LayerNorm weight
  float* bv = wv + kLtDV;     // value-part LayerNorm bias
  float* red = bv + kLtDV;    // reductions
  float* part = red + 16;     // [4][128] partial value sums
  float* pj = part + 4 * kLtDV;  // a_j = p_j rstd_j
  const int hh = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int L = clamp_len(seq_lens[b], P * max_pages);
  uint16_t* orow = out + (static_cast<int64_t>(b) * H + hh) * kLtDV;
  if (L == 0) {
    if (tid < kLtDV) orow[tid] = 0;
    return;
  }
  const int width = H * kLtHeadW;
  const int64_t kbase = static_cast<int64_t>(hh) * kLtHeadW;
  const uint16_t* qrow = q + (static_cast<int64_t>(b) * H + hh) * (kLtDH + kLtDR);
  // key-part LayerNorm folded into the query: qa = q w, and sum_d q_d b_d, sum_d q_d w_d
  float qb = 0.f, qw = 0.f;
  if (tid < kLtDH) {
    const float qd = bf16_to_f32(qrow[tid]);
    const float wd = use_ln ? bf16_to_f32(ln_w[kbase + tid]) : 1.f;
    const float bd = use_ln ? bf16_to_f32(ln_b[kbase + tid]) : 0.f;
    qa[tid] = qd * wd;
    qb = qd * bd;
    qw = qd * wd;
  } else if (tid < kLtDH + kLtDR) {
    qr[tid - kLtDH] = bf16_to_f32(qrow[tid]);
  }
  if (tid < kLtDV) {
    wv[tid] = use_ln ? bf16_to_f32(ln_w[kbase + kLtDH + tid]) : 1.f;
    bv[tid] = use_ln ? bf16_to_f32(ln_b[kbase + kLtDH + tid]) : 0.f;
  }
  qb = wave_sum(qb);
  qw = wave_sum(qw);
  if (lane == 0) {
    red[w] = qb;
    red[4 + w] = qw;
  }
  __syncthreads();
  const float sum_qb = red[0] + red[1] + red[2] + red[3];
  const float sum_qw = red[4] + red[5] + red[6] + red[7];
  __syncthreads();

  // scores: one token per thread
  float mx = -INFINITY;
  for (int j = tid; j < L; j += 256) {
    const int64_t row = cache_slot(page_table, b, j, P, max_pages, num_slots);
    const float2 st = use_ln ? stats[row] : make_float2(0.f, 1.f);
    const uint16_t* yk = Y + row * width + kbase;
    float dot = 0.f;
#pragma unroll 4
    for (int c = 0; c < kLtDH / 8; ++c) {
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(yk + 8 * c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        dot = fmaf(qa[8 * c + 2 * e], bf16_lo(v[e]), dot);
        dot = fmaf(qa[8 * c + 2 * e + 1], bf16_hi(v[e]), dot);
      }
    }
    const uint16_t* kr = cache + row * (kLtDC + kLtDR) + kLtDC;
    float rdot = 0.f;
#pragma unroll
    for (int c = 0; c < kLtDR / 8; ++c) {
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(kr + 8 * c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        rdot = fmaf(qr[8 * c + 2 * e], bf16_lo(v[e]), rdot);
        rdot = fmaf(qr[8 * c + 2 * e + 1], bf16_hi(v[e]), rdot);
      }
    }
    const float s = scale * (st.y * (dot - st.x * sum_qw) + sum_qb + rdot);
    pj[j] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max(mx);
  if (lane == 0) red[w] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float psum = 0.f, amu = 0.f;
  for (int j = tid; j < L; j += 256) {
    const int64_t row = cache_slot(page_table, b, j, P, max_pages, num_slots);
    const float2 st = use_ln ? stats[row] : make_float2(0.f, 1.f);
    const float p = expf(pj[j] - mx);
    psum += p;
    pj[j] = p * st.y;
    amu = fmaf(p * st.y, st.x, amu);
  }
  psum = wave_sum(psum);
  amu = wave_sum(amu);
  if (lane == 0) {
    red[w] = psum;
    red[4 + w] = amu;
  }
  __syncthreads();
  psum = red[0] + red[1] + red[2] + red[3];
  amu = red[4] + red[5] + red[6] + red[7];

  // values: wave w takes tokens j = w, w + 4, ...; lane takes dims 2 lane, 2 lane + 1
  float v0 = 0.f, v1 = 0.f;
  for (int j = w; j < L; j += 4) {
    const int64_t row = cache_slot(page_table, b, j, P, max_pages, num_slots);
    const uint32_t v = *reinterpret_cast<const uint32_t*>(Y + row * width + kbase + kLtDH + 2 * lane);
    const float a = pj[j];
    v0 = fmaf(a, bf16_lo(v), v0);
    v1 = fmaf(a, bf16_hi(v), v1);
  }
  part[w * kLtDV + 2 * lane] = v0;
  part[w * kLtDV + 2 * lane + 1] = v1;
  __syncthreads();
  if (tid < kLtDV) {
    const float s = part[tid] + part[kLtDV + tid] + part[2 * kLtDV + tid] + part[3 * kLtDV + tid];
    orow[tid] = f32_to_bf16(wv[tid] * (s - amu) / psum + bv[tid]);
  }
}

}  // namespace egmla

using namespace egmla;

extern "C" size_t eg_mla_decode_literal_workspace_size(const eg_mla_dims* dims, int64_t num_slots) {
  if (check_dims(dims) != EG_MLA_OK || num_slots < 0) return 0;
  return literal_workspace_bytes(*dims, num_slots);
}

extern "C" eg_mla_status eg_mla_decode_literal(const eg_mla_dims* dims, int32_t batch, const void* q,
                                               const void* latent_cache, const int32_t* token_id_cache,
                                               const void* gate_full, const void* w_uk, const void* w_uv,
                                               const void* ln_weight, const void* ln_bias, uint32_t flags,
                                               const int32_t* seq_lens, const int32_t* page_table,
                                               int32_t max_pages_per_seq, int64_t num_slots, void* workspace,
                                               size_t workspace_bytes, void* out, void* stream_) {
  eg_mla_status st = validate_literal(dims, batch, q, latent_cache, token_id_cache, gate_full, w_uk, w_uv, ln_weight,
                                      ln_bias, flags, seq_lens, page_table, max_pages_per_seq, num_slots, workspace,
                                      workspace_bytes, out);
  if (st != EG_MLA_OK || batch == 0) return st;
  const eg_mla_dims& d = *dims;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  (void)hipGetLastError();
  const int P = d.page_size, cap = P * max_pages_per_seq;
  uint16_t* Y = static_cast<uint16_t*>(workspace);
  float2* stats = reinterpret_cast<float2*>(static_cast<unsigned char*>(workspace) + literal_stats_offset(d, num_slots));
  const bool use_ln = (flags & EG_MLA_LITERAL_NO_LN) == 0;
  const int add = (flags & EG_MLA_LITERAL_ADD) != 0;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(literal_kv_kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                          kLtWLds) != hipSuccess)
    return EG_MLA_ERR_HIP;
  hipLaunchKernelGGL(literal_kv_kernel, dim3((cap + 127) / 128, batch), dim3(256), kLtWLds, stream,
                     static_cast<const uint16_t*>(latent_cache), token_id_cache, static_cast<const uint16_t*>(gate_full),
                     static_cast<const uint16_t*>(w_uk), static_cast<const uint16_t*>(w_uv), seq_lens, page_table, P,
                     max_pages_per_seq, num_slots, d.num_heads, d.vocab_size, add, Y, stats);
  const size_t lds = sizeof(float) * (static_cast<size_t>(kLtDH + kLtDR + 2 * kLtDV + 16 + 4 * kLtDV) + cap);
  if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(literal_attn_kernel),
                                         hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)) != hipSuccess)
    return EG_MLA_ERR_HIP;
  hipLaunchKernelGGL(literal_attn_kernel, dim3(d.num_heads, batch), dim3(256), lds, stream,
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(latent_cache), Y, stats,
                     static_cast<const uint16_t*>(ln_weight), static_cast<const uint16_t*>(ln_bias),
                     use_ln ? 1 : 0, seq_lens, page_table, P, max_pages_per_seq, num_slots, d.num_heads,
                     softmax_scale(d), static_cast<uint16_t*>(out));
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
