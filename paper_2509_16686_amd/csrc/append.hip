// EG-MLA cache append on gfx950: compress new tokens into latent-cache rows.
//
// For each new token (Sec. 3.1 Eq. (1), App. C Eq. (C.10)):
//   [c | r] = W_DKV x       (W_DKV stacks W^DKV and W^KR: [d_c + d_r, hidden])
//   c       = RMSNorm(c) * kv_norm_w      (optional latent norm, eps 1e-6)
//   k^R     = RoPE(r, position)           (adjacent pairs, angle pos * theta^(-2m/d_r))
// and the row [c | k^R] plus the token id are stored at the token's slot.
// General shapes: one work-group (256 threads) per token; each wave computes
// output features as coalesced dot products over the hidden dimension.  The
// d_c 128 / d_r 64 bf16 layer takes the MFMA kernel below.
#include <hip/hip_runtime.h>

#include <algorithm>
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

// ---------------------------------------------------------------------------
// MFMA append for bf16 storage with d_c = 128, d_r = 64 and hidden a multiple
// of 128: Y^T[o][t] = sum_k W_DKV[o][k] x[t][k] on v_mfma_f32_32x32x16_bf16,
// both operands straight from global (A: output row o = lane % 32, 8
// consecutive k; B: token t = lane % 32, the same k), so the accumulator holds
// 32 outputs x 32 tokens with each token's values in lanes t and t + 32.
// Work-group y = 0 takes the 128 latent outputs (the RMSNorm needs all of a
// token's latent), y = 1 the 64 RoPE outputs (a rotation pair, outputs 2m and
// 2m + 1, sits in one lane).  KSPLIT (few tokens): the 4 waves share 32 tokens
// and split the hidden dimension, partial sums meet in LDS and wave 0 finishes;
// otherwise each wave takes its own 32 tokens over the whole hidden dimension.
// Every load is in bounds: token rows past n repeat the last token and are not
// stored.
// ---------------------------------------------------------------------------
constexpr int kAppMfmaDC = 128, kAppMfmaDR = 64;
typedef __attribute__((ext_vector_type(16))) float app_f32x16_t;

template <int NOB, bool KSPLIT, bool LATENT>
__device__ __forceinline__ void append_mfma_part(const uint16_t* __restrict__ x, const int32_t* __restrict__ token_ids,
                                                 const int32_t* __restrict__ positions,
                                                 const int32_t* __restrict__ slots,
                                                 const uint16_t* __restrict__ w_dkv,
                                                 const uint16_t* __restrict__ kv_norm_w, float theta,
                                                 uint16_t* __restrict__ cache, int32_t* __restrict__ ids,
                                                 int64_t num_slots, int n, int hidden, float* red,
                                                 const double* freq) {
  constexpr int DQ = kAppMfmaDC + kAppMfmaDR;
  constexpr int O0 = LATENT ? 0 : kAppMfmaDC;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int tok = blockIdx.x * (KSPLIT ? 32 : 128) + (KSPLIT ? 0 : 32 * w) + r32;
  const int tc = min(tok, n - 1);
  const int kspan = KSPLIT ? hidden / 4 : hidden;
  const int k_lo = KSPLIT ? w * kspan : 0;
  const uint16_t* xb = x + static_cast<int64_t>(tc) * hidden + k_lo + 8 * h;
  const uint16_t* wb = w_dkv + static_cast<int64_t>(O0 + r32) * hidden + k_lo + 8 * h;
  // the epilogue's inputs travel while the products run: destination slot,
  // token id or position, and with few tokens (KSPLIT: registers to spare)
  // the norm weights of this lane's 4 x NOB groups of 4 outputs
  const int64_t slot_pre = slots[tc];
  const int32_t aux_pre = LATENT ? token_ids[tc] : positions[tc];
  constexpr bool kNormEarly = LATENT && KSPLIT;
  u32x2_t nw_pre[LATENT ? NOB * 4 : 1];
  auto load_norm = [&]() {
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        nw_pre[4 * ob + q] = kv_norm_w ? *reinterpret_cast<const u32x2_t*>(kv_norm_w + 32 * ob + 8 * q + 4 * h)
                                       : u32x2_t{0u, 0u};
  };
  if constexpr (kNormEarly) load_norm();
  app_f32x16_t acc[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[ob][r] = 0.f;
  // batches of 4 chunks of 16: the next batch's loads are in flight while
  // this batch's products run (kspan is a multiple of 128: an even count)
  bf16x8_t bv[2][4], av[2][4][NOB];
  auto load = [&](int buf, int k0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      bv[buf][c] = *reinterpret_cast<const bf16x8_t*>(xb + k0 + 16 * c);
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
        av[buf][c][ob] = *reinterpret_cast<const bf16x8_t*>(wb + static_cast<int64_t>(32 * ob) * hidden + k0 + 16 * c);
    }
  };
  auto products = [&](int buf) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
        acc[ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[buf][c][ob], bv[buf][c], acc[ob], 0, 0, 0);
  };
  load(0, 0);
  for (int k0 = 0; k0 < kspan; k0 += 128) {
    load(1, k0 + 64);
    __builtin_amdgcn_sched_barrier(0);
    products(0);
    if (k0 + 128 < kspan) load(0, k0 + 128);
    __builtin_amdgcn_sched_barrier(0);
    products(1);
  }
  if constexpr (KSPLIT) {
    // partial sums of waves 1..3 to LDS ([wave][ob][r][lane]), wave 0 adds them in order
    if (w > 0) {
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(((w - 1) * NOB + ob) * 16 + r) * 64 + lane] = acc[ob][r];
    }
    __syncthreads();
    if (w > 0) return;
#pragma unroll
    for (int v = 0; v < 3; ++v)
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[ob][r] += red[((v * NOB + ob) * 16 + r) * 64 + lane];
  }
  if (tok >= n) return;
  const int64_t slot = slot_pre;
  const bool store = slot >= 0 && slot < num_slots;  // out-of-range destination: skipped
  uint16_t* row = cache + (store ? slot : 0) * DQ + O0 + 4 * h;
  // lane holds outputs O0 + 32 ob + 8 q + 4 h + (0..3) of token tok in acc[ob][4 q + (0..3)]
  if constexpr (LATENT) {
    if constexpr (!kNormEarly) load_norm();
    float inv_rms = 1.f;
    if (kv_norm_w) {
      float ss = 0.f;
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int r = 0; r < 16; ++r) ss = fmaf(acc[ob][r], acc[ob][r], ss);
      const uint32_t u = __float_as_uint(ss);
      const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
      ss = __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
      inv_rms = 1.f / sqrtf(ss / static_cast<float>(kAppMfmaDC) + kRmsEps);
    }
    if (store) {
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[e] = acc[ob][4 * q + e];
            if (kv_norm_w) {
              const uint32_t wpair = nw_pre[4 * ob + q][e >> 1];
              v[e] = v[e] * inv_rms * ((e & 1) ? bf16_hi(wpair) : bf16_lo(wpair));
            }
          }
          *reinterpret_cast<u32x2_t*>(row + 32 * ob + 8 * q) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        }
      if (h == 0) ids[slot] = aux_pre;
    }
  } else {
    if (store) {
      // the angle pos * theta^(-2m/d_r) and its reduction to [-pi, pi] are
      // formed in fp64 (frequencies from the work-group's table), so that
      // large positions keep full accuracy; the sine and cosine of the reduced
      // angle are fp32 (error ~1e-7, far below the bf16 result)
      const double pos = static_cast<double>(aux_pre);
      constexpr double kTwoPi = 6.283185307179586476925286766559;
#pragma unroll
      for (int ob = 0; ob < NOB; ++ob)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
#pragma unroll
          for (int pr = 0; pr < 2; ++pr) {
            const int m = (32 * ob + 8 * q + 4 * h + 2 * pr) / 2;  // pair index within the RoPE key
            const double ang = pos * freq[m];
            const double turns = rint(ang * (1.0 / kTwoPi));
            const float red_ang = static_cast<float>(fma(-turns, kTwoPi, ang));
            float sn, cs;
            sincosf(red_ang, &sn, &cs);
            const float x0 = acc[ob][4 * q + 2 * pr], x1 = acc[ob][4 * q + 2 * pr + 1];
            v[2 * pr] = x0 * cs - x1 * sn;
            v[2 * pr + 1] = x0 * sn + x1 * cs;
          }
          *reinterpret_cast<u32x2_t*>(row + 32 * ob + 8 * q) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
        }
    }
  }
}

template <bool KSPLIT>
__global__ __launch_bounds__(256) void append_mfma_kernel(const uint16_t* __restrict__ x,
                                                          const int32_t* __restrict__ token_ids,
                                                          const int32_t* __restrict__ positions,
                                                          const int32_t* __restrict__ slots,
                                                          const uint16_t* __restrict__ w_dkv,
                                                          const uint16_t* __restrict__ kv_norm_w, float theta,
                                                          uint16_t* __restrict__ cache, int32_t* __restrict__ ids,
                                                          int64_t num_slots, int n, int hidden) {
  __shared__ float red[KSPLIT ? 3 * 4 * 16 * 64 : 1];
  __shared__ double freq[kAppMfmaDR / 2];  // theta^(-2m/d_r), m = 0 .. d_r/2 - 1
  if (threadIdx.x < kAppMfmaDR / 2)
    freq[threadIdx.x] = pow(static_cast<double>(theta), -2.0 * threadIdx.x / static_cast<double>(kAppMfmaDR));
  __syncthreads();
  if (blockIdx.y == 0)
    append_mfma_part<4, KSPLIT, true>(x, token_ids, positions, slots, w_dkv, kv_norm_w, theta, cache, ids, num_slots,
                                      n, hidden, red, freq);
  else
    append_mfma_part<2, KSPLIT, false>(x, token_ids, positions, slots, w_dkv, kv_norm_w, theta, cache, ids,
                                       num_slots, n, hidden, red, freq);
}

// ---------------------------------------------------------------------------
// Split append (eg_mla_append_ws) for the bf16 layers with d_r = 64 and
// d_c = 128 or 512: the hidden dimension is cut into nks slices (a multiple of
// 256 wide each) so that a few tokens' call spreads W_DKV over many
// work-groups instead of streaming it through a few; many tokens take one
// slice, and the second pass then only applies the norm and the rotation.
//  Pass 1: work-group (ks, tg, ob) forms the partial sums of outputs
//    32 ob .. + 31 (the latent first, then the RoPE key) of 32 NTG tokens
//    (NTG = 1, or 2 above 32 tokens) over slice ks: wave w takes a quarter of
//    the slice, 4 chunks of 16 k at a time with the next 4 in flight, on
//    v_mfma_f32_32x32x16_bf16 (A: W_DKV row o = lane % 32, 8 consecutive k;
//    B: the token row, the same k; one A serves NTG token blocks); the 4
//    waves' sums are added in LDS in wave order and stored as fp32
//    part[ks][t][o].
//  Pass 2: a wave per token (d_c 128; d_c 512 with few slices, 4 latent
//    pairs per lane) or a work-group per token (d_c 512 with many slices, a
//    pair per thread) adds the slices' sums in slice order (lane l: latent
//    pairs l + T i, and for l < d_r / 2 the RoPE pair l), applies the latent
//    RMSNorm and the rotation, and writes the row and the id.
// Every load is in bounds: token rows past n repeat the last token and are not
// stored.
// ---------------------------------------------------------------------------
constexpr int kAppSliceUnit = 256;    // slice widths are multiples of this
#ifndef EGMLA_APPEND_TARGET_GROUPS
#define EGMLA_APPEND_TARGET_GROUPS 512
#endif
constexpr int kAppTargetGroups = EGMLA_APPEND_TARGET_GROUPS;  // pass-1 work-groups the slice count aims for
#ifndef EGMLA_APPEND_GEMM_TARGET
#define EGMLA_APPEND_GEMM_TARGET 128
#endif
constexpr int kAppGemmTarget = EGMLA_APPEND_GEMM_TARGET;   // the same for the tiled product (measured)
#ifndef EGMLA_APPEND_GEMM_MIN
#define EGMLA_APPEND_GEMM_MIN (256 * 576)
#endif
constexpr int64_t kAppGemmMin = EGMLA_APPEND_GEMM_MIN;  // outputs (tokens x (d_c + d_r)) from which the tiled product pays
constexpr int kAppFinishWaveSlices = 4;  // d_c 512: pass 2 takes a wave per token up to this many slices
constexpr int kAppSplitMax128 = 2048;   // d_c 128: largest call taken by the split passes (measured crossover)
constexpr int kAppSplitMax512 = 1 << 20;  // d_c 512: every call (the one-pass kernel is the general one)

template <int DQ, int NTG>
__global__ __launch_bounds__(256) void append_slice_kernel(const uint16_t* __restrict__ x,
                                                           const uint16_t* __restrict__ w_dkv,
                                                           float* __restrict__ part, int n, int hidden, int slice) {
  __shared__ float red[3 * NTG * 16 * 64];
  const int ks = blockIdx.x, tg = blockIdx.y, ob = blockIdx.z;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int kw = slice / 4;  // a multiple of 64
  const int64_t k0 = static_cast<int64_t>(slice) * ks + kw * w + 8 * h;
  const uint16_t* xb[NTG];
#pragma unroll
  for (int g = 0; g < NTG; ++g)
    xb[g] = x + static_cast<int64_t>(min(32 * (NTG * tg + g) + r32, n - 1)) * hidden + k0;
  const uint16_t* wb = w_dkv + static_cast<int64_t>(32 * ob + r32) * hidden + k0;
  bf16x8_t av[2][4], bv[2][NTG][4];
  auto load = [&](int buf, int k) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      av[buf][c] = *reinterpret_cast<const bf16x8_t*>(wb + k + 16 * c);
#pragma unroll
      for (int g = 0; g < NTG; ++g) bv[buf][g][c] = *reinterpret_cast<const bf16x8_t*>(xb[g] + k + 16 * c);
    }
  };
  app_f32x16_t acc[NTG];
#pragma unroll
  for (int g = 0; g < NTG; ++g)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[g][r] = 0.f;
  auto products = [&](int buf) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
      for (int g = 0; g < NTG; ++g)
        acc[g] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[buf][c], bv[buf][g][c], acc[g], 0, 0, 0);
  };
  load(0, 0);
  for (int k = 0; k < kw; k += 128) {
    const bool second = k + 64 < kw;
    if (second) load(1, k + 64);
    __builtin_amdgcn_sched_barrier(0);
    products(0);
    if (k + 128 < kw) load(0, k + 128);
    __builtin_amdgcn_sched_barrier(0);
    if (second) products(1);
  }
  if (w > 0) {
#pragma unroll
    for (int g = 0; g < NTG; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) red[(((w - 1) * NTG + g) * 16 + r) * 64 + lane] = acc[g][r];
  }
  __syncthreads();
  if (w > 0) return;
#pragma unroll
  for (int v = 0; v < 3; ++v)
#pragma unroll
    for (int g = 0; g < NTG; ++g)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[g][r] += red[((v * NTG + g) * 16 + r) * 64 + lane];
  // lane holds outputs 32 ob + 8 q + 4 h + (0..3) of token 32 (NTG tg + g) + r32 in acc[g][4 q + (0..3)]
#pragma unroll
  for (int g = 0; g < NTG; ++g) {
    const int tok = 32 * (NTG * tg + g) + r32;
    if (tok >= n) break;
    float* dst = part + (static_cast<int64_t>(ks) * n + tok) * DQ + 32 * ob + 4 * h;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(dst + 8 * q) =
          make_float4(acc[g][4 * q], acc[g][4 * q + 1], acc[g][4 * q + 2], acc[g][4 * q + 3]);
  }
}

// Pass 1 for many tokens: the same partial sums from an LDS-tiled product.
// Work-group (ks, tt, ot) takes tokens 128 tt .. + 127 and outputs
// 192 ot .. + 191 over slice ks, in steps of 32 k: each step's 128 token rows
// and 192 W_DKV rows (64 B each) are staged in LDS (row stride 80 B, so that
// the operand reads of 16 rows by 16 lanes hit 64 distinct banks), double
// buffered, with the global loads two steps ahead in registers.  Wave
// (wt, wo) = (w % 2, w / 2) forms tokens 64 wt .. + 63 x outputs 96 wo .. + 95
// as 2 x 3 tiles of v_mfma_f32_32x32x16_bf16 (A: W_DKV rows, B: token rows).
constexpr int kGemmTok = 128, kGemmOut = 192, kGemmK = 32, kGemmStride = kGemmK + 8;
constexpr int kGemmRows = kGemmTok + kGemmOut;
constexpr int kGemmLoads = kGemmRows * (kGemmK / 8) / 256;  // 16-byte copies per thread and step
static_assert(kGemmRows * (kGemmK / 8) % 256 == 0, "whole copies per thread");

template <int DQ>
__global__ __launch_bounds__(256, 2) void append_gemm_kernel(const uint16_t* __restrict__ x,
                                                            const uint16_t* __restrict__ w_dkv,
                                                            float* __restrict__ part, int n, int hidden, int slice) {
  __shared__ __attribute__((aligned(16))) uint16_t stage[2][kGemmRows * kGemmStride];
  const int ks = blockIdx.x, tt = blockIdx.y, ot = blockIdx.z;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int wt = w & 1, wo = w >> 1;
  const int64_t kb = static_cast<int64_t>(slice) * ks;
  // copy j = tid + 256 i: row j / 4 (token rows first, then W_DKV rows), 16 bytes at 8 (j % 4)
  const uint16_t* src[kGemmLoads];
  int dst[kGemmLoads];
#pragma unroll
  for (int i = 0; i < kGemmLoads; ++i) {
    const int j = tid + 256 * i, row = j >> 2, c = j & 3;
    src[i] = row < kGemmTok ? x + static_cast<int64_t>(min(kGemmTok * tt + row, n - 1)) * hidden + kb + 8 * c
                            : w_dkv + static_cast<int64_t>(kGemmOut * ot + row - kGemmTok) * hidden + kb + 8 * c;
    dst[i] = row * kGemmStride + 8 * c;
  }
  bf16x8_t g[2][kGemmLoads];
  auto fetch = [&](int set, int step) {
#pragma unroll
    for (int i = 0; i < kGemmLoads; ++i)
      g[set][i] = *reinterpret_cast<const bf16x8_t*>(src[i] + static_cast<int64_t>(kGemmK) * step);
  };
  auto put = [&](int buf, int set) {
#pragma unroll
    for (int i = 0; i < kGemmLoads; ++i) *reinterpret_cast<bf16x8_t*>(&stage[buf][dst[i]]) = g[set][i];
  };
  app_f32x16_t acc[2][3];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int ob = 0; ob < 3; ++ob)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[tb][ob][r] = 0.f;
  const int brow = (64 * wt + r32) * kGemmStride + 8 * h;
  const int arow = (kGemmTok + 96 * wo + r32) * kGemmStride + 8 * h;
  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < kGemmK / 16; ++kk) {
      bf16x8_t bv[2], av[3];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
        bv[tb] = *reinterpret_cast<const bf16x8_t*>(&stage[buf][brow + 32 * tb * kGemmStride + 16 * kk]);
#pragma unroll
      for (int ob = 0; ob < 3; ++ob)
        av[ob] = *reinterpret_cast<const bf16x8_t*>(&stage[buf][arow + 32 * ob * kGemmStride + 16 * kk]);
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int ob = 0; ob < 3; ++ob)
          acc[tb][ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[ob], bv[tb], acc[tb][ob], 0, 0, 0);
    }
  };
  // step s computes from buffer s % 2; the data of step s + 1 (register set
  // (s + 1) % 2) is written to the other buffer after it, and step s + 3 is
  // fetched into the freed set.  The loop has no branch (the step count is
  // even: slices are multiples of 256 wide; past the last step the last one is
  // fetched and written again, to a buffer nothing reads), so that each write
  // to LDS waits only for its own set's loads while the newer set stays in
  // flight.
  const int steps = slice / kGemmK;
  fetch(0, 0);
  fetch(1, 1);
  put(0, 0);
  fetch(0, min(2, steps - 1));
  __syncthreads();
  for (int s0 = 0; s0 < steps; s0 += 2) {
    compute(0);
    put(1, 1);
    fetch(1, min(s0 + 3, steps - 1));
    __syncthreads();
    compute(1);
    put(0, 0);
    fetch(0, min(s0 + 4, steps - 1));
    __syncthreads();
  }
  // lane holds outputs (96 wo + 32 ob) + 8 q + 4 h + (0..3) of token 64 wt + 32 tb + r32 in acc[tb][ob][4 q + (0..3)]
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int tok = kGemmTok * tt + 64 * wt + 32 * tb + r32;
    if (tok >= n) break;
    float* row = part + (static_cast<int64_t>(ks) * n + tok) * DQ + kGemmOut * ot + 96 * wo + 4 * h;
#pragma unroll
    for (int ob = 0; ob < 3; ++ob)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(row + 32 * ob + 8 * q) =
            make_float4(acc[tb][ob][4 * q], acc[tb][ob][4 * q + 1], acc[tb][ob][4 * q + 2], acc[tb][ob][4 * q + 3]);
  }
}

template <int DC, int DR, int TPT>
__global__ __launch_bounds__(256) void append_finish_kernel(const float* __restrict__ part, int nks,
                                                            const int32_t* __restrict__ token_ids,
                                                            const int32_t* __restrict__ positions,
                                                            const int32_t* __restrict__ slots,
                                                            const uint16_t* __restrict__ kv_norm_w, float theta,
                                                            uint16_t* __restrict__ cache, int32_t* __restrict__ ids,
                                                            int64_t num_slots, int n) {
  // TPT threads per token, each with NPL latent pairs (l + TPT i) and, for
  // l < d_r / 2, the RoPE pair l
  constexpr int DQ = DC + DR, TPB = 256 / TPT, WPT = TPT / 64, NPL = DC / 2 / TPT;
  static_assert(TPT % 64 == 0 && 256 % TPT == 0 && DC % (2 * TPT) == 0 && DR / 2 <= TPT, "token groups");
  __shared__ float red[WPT];
  const int tid = threadIdx.x, l = tid % TPT, lane = tid & 63;
  const int t = TPB * blockIdx.x + tid / TPT;
  if (t >= n) return;  // uniform over a token's threads
  // every load of the token is issued before the first use (none depends on
  // another): its slot, id, position, norm weights and the slices' sums
  const int64_t slot = slots[t];
  const int32_t tok_id = token_ids[t];
  const int32_t pos = positions[t];
  const bool rope = l < DR / 2;
  uint32_t wpair[NPL];
#pragma unroll
  for (int i = 0; i < NPL; ++i)
    wpair[i] = kv_norm_w ? *reinterpret_cast<const uint32_t*>(kv_norm_w + 2 * (l + TPT * i)) : 0u;
  // the slices' sums are loaded kBatch at a time (one round trip for up to
  // kBatch slices: this pass is bound by the latency of its loads), then added
  // in slice order
  constexpr int kBatch = 32 / NPL;
  float2 c[NPL], r = make_float2(0.f, 0.f);
#pragma unroll
  for (int i = 0; i < NPL; ++i) c[i] = make_float2(0.f, 0.f);
  for (int k0 = 0; k0 < nks; k0 += kBatch) {
    float2 av[kBatch][NPL], bv[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (k0 + u < nks) {
        const float* row = part + (static_cast<int64_t>(k0 + u) * n + t) * DQ;
#pragma unroll
        for (int i = 0; i < NPL; ++i) av[u][i] = *reinterpret_cast<const float2*>(row + 2 * (l + TPT * i));
        bv[u] = rope ? *reinterpret_cast<const float2*>(row + DC + 2 * l) : make_float2(0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (k0 + u < nks) {
#pragma unroll
        for (int i = 0; i < NPL; ++i) {
          c[i].x += av[u][i].x;
          c[i].y += av[u][i].y;
        }
        r.x += bv[u].x;
        r.y += bv[u].y;
      }
    }
  }
  // uniform over a token's threads (the whole work-group when a token takes
  // several waves, so the barrier below is reached by all or none)
  if (slot < 0 || slot >= num_slots) return;  // out-of-range destination: skipped
  uint16_t* dst = cache + slot * DQ;
  if (kv_norm_w) {
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NPL; ++i) ss += c[i].x * c[i].x + c[i].y * c[i].y;
    ss = wave_sum(ss);
    if constexpr (WPT > 1) {
      if (lane == 0) red[tid >> 6] = ss;
      __syncthreads();
      ss = red[0];
#pragma unroll
      for (int v = 1; v < WPT; ++v) ss += red[v];
    }
    const float inv_rms = 1.f / sqrtf(ss / static_cast<float>(DC) + kRmsEps);
#pragma unroll
    for (int i = 0; i < NPL; ++i) {
      c[i].x = c[i].x * inv_rms * bf16_lo(wpair[i]);
      c[i].y = c[i].y * inv_rms * bf16_hi(wpair[i]);
    }
  }
#pragma unroll
  for (int i = 0; i < NPL; ++i)
    *reinterpret_cast<uint32_t*>(dst + 2 * (l + TPT * i)) = pack_bf16x2(c[i].x, c[i].y);
  if (rope) {
    // the angle pos * theta^(-2m/d_r) and its reduction to [-pi, pi] in fp64,
    // the sine and cosine of the reduced angle in fp32 (as the one-pass kernel)
    constexpr double kTwoPi = 6.283185307179586476925286766559;
    const double ang = static_cast<double>(pos) * pow(static_cast<double>(theta), -2.0 * l / static_cast<double>(DR));
    const double turns = rint(ang * (1.0 / kTwoPi));
    const float red_ang = static_cast<float>(fma(-turns, kTwoPi, ang));
    float sn, cs;
    sincosf(red_ang, &sn, &cs);
    *reinterpret_cast<uint32_t*>(dst + DC + 2 * l) = pack_bf16x2(r.x * cs - r.y * sn, r.x * sn + r.y * cs);
  }
  if (l == 0) ids[slot] = tok_id;
}

bool append_split_shape(const eg_mla_dims& d, int32_t n_tokens, int32_t hidden) {
  if (d.dtype != EG_MLA_BF16 || d.rope_dim != 64 || hidden % kAppSliceUnit != 0 || n_tokens < 1) return false;
  if (d.latent_dim == 128) return n_tokens <= kAppSplitMax128;
  if (d.latent_dim == 512) return n_tokens <= kAppSplitMax512;
  return false;
}

// Pass 1 takes the LDS-tiled product from kAppGemmMin outputs on (256 tokens
// at d_c 512, 768 at d_c 128: below, its 128 x 192 tiles are too few).
bool append_split_gemm(const eg_mla_dims& d, int32_t n_tokens) {
  return static_cast<int64_t>(n_tokens) * (d.latent_dim + d.rope_dim) >= kAppGemmMin;
}

// Tokens per pass-1 work-group: 32, or 64 above 32 tokens (W_DKV is then
// read half as often), or 128 in the tiled product.
int append_split_tokens(const eg_mla_dims& d, int32_t n_tokens) {
  return append_split_gemm(d, n_tokens) ? kGemmTok : n_tokens <= 32 ? 32 : 64;
}

// Slice count: the fewest (a divisor of hidden / 256) that still give the
// first pass its target number of work-groups, else the most.
int append_split_slices(const eg_mla_dims& d, int32_t n_tokens, int32_t hidden) {
  const int64_t units = hidden / kAppSliceUnit;
  const int per = append_split_tokens(d, n_tokens);
  const bool gemm = append_split_gemm(d, n_tokens);
  const int64_t groups = static_cast<int64_t>((n_tokens + per - 1) / per) *
                         ((d.latent_dim + d.rope_dim) / (gemm ? kGemmOut : 32));
  const int64_t target = gemm ? kAppGemmTarget : kAppTargetGroups;
  for (int64_t s = 1; s < units; ++s)
    if (units % s == 0 && s * groups >= target) return static_cast<int>(s);
  return static_cast<int>(units);
}

size_t append_split_bytes(const eg_mla_dims& d, int32_t n_tokens, int32_t hidden) {
  return static_cast<size_t>(append_split_slices(d, n_tokens, hidden)) * static_cast<size_t>(n_tokens) *
         static_cast<size_t>(d.latent_dim + d.rope_dim) * 4;
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
  const bool aligned = reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(w_dkv) % 16 == 0 &&
                       reinterpret_cast<uintptr_t>(latent_cache) % 8 == 0 &&
                       reinterpret_cast<uintptr_t>(kv_norm_w) % 8 == 0;  // null passes
  if (d.dtype == EG_MLA_BF16 && d.latent_dim == kAppMfmaDC && d.rope_dim == kAppMfmaDR && hidden % 512 == 0 &&
      aligned) {
    // few tokens: split the hidden dimension over the 4 waves of a 32-token work-group
    const bool ksplit = n_tokens <= 8192;
    const int per = ksplit ? 32 : 128;
    const dim3 grid((n_tokens + per - 1) / per, 2);
    const uint16_t* xb = static_cast<const uint16_t*>(x);
    const uint16_t* wb = static_cast<const uint16_t*>(w_dkv);
    const uint16_t* nw = static_cast<const uint16_t*>(kv_norm_w);
    uint16_t* cb = static_cast<uint16_t*>(latent_cache);
    if (ksplit)
      hipLaunchKernelGGL(append_mfma_kernel<true>, grid, dim3(256), 0, stream, xb, token_ids, positions, slots, wb, nw,
                         theta, cb, token_id_cache, num_slots, n_tokens, hidden);
    else
      hipLaunchKernelGGL(append_mfma_kernel<false>, grid, dim3(256), 0, stream, xb, token_ids, positions, slots, wb,
                         nw, theta, cb, token_id_cache, num_slots, n_tokens, hidden);
  } else if (d.dtype == EG_MLA_BF16) {
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

extern "C" size_t eg_mla_append_workspace_size(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden) {
  if (check_dims(dims) != EG_MLA_OK || n_tokens < 0 || hidden < 1) return 0;
  if (!append_split_shape(*dims, n_tokens, hidden)) return kAlign;
  return std::max<size_t>(align_up(append_split_bytes(*dims, n_tokens, hidden)), kAlign);
}

extern "C" eg_mla_status eg_mla_append_ws(const eg_mla_dims* dims, int32_t n_tokens, int32_t hidden, const void* x,
                                          const int32_t* token_ids, const int32_t* positions, const int32_t* slots,
                                          const void* w_dkv, const void* kv_norm_w, float rope_theta,
                                          void* latent_cache, int32_t* token_id_cache, int64_t num_slots,
                                          void* workspace, size_t workspace_bytes, void* stream_) {
  eg_mla_status st = validate_append(dims, n_tokens, hidden, x, token_ids, positions, slots, w_dkv, latent_cache,
                                     token_id_cache, num_slots);
  if (st != EG_MLA_OK || n_tokens == 0) return st;
  const eg_mla_dims& d = *dims;
  const bool aligned = reinterpret_cast<uintptr_t>(x) % 16 == 0 && reinterpret_cast<uintptr_t>(w_dkv) % 16 == 0 &&
                       reinterpret_cast<uintptr_t>(latent_cache) % 4 == 0 &&
                       reinterpret_cast<uintptr_t>(kv_norm_w) % 4 == 0;  // null passes
  if (!append_split_shape(d, n_tokens, hidden) || !aligned)
    return eg_mla_append(dims, n_tokens, hidden, x, token_ids, positions, slots, w_dkv, kv_norm_w, rope_theta,
                         latent_cache, token_id_cache, num_slots, stream_);
  if (!workspace || workspace_bytes < append_split_bytes(d, n_tokens, hidden) ||
      reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
    return EG_MLA_ERR_WORKSPACE;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const float theta = rope_theta > 0.f ? rope_theta : 10000.f;
  (void)hipGetLastError();
  const int nks = append_split_slices(d, n_tokens, hidden);
  const int slice = hidden / nks;
  float* part = static_cast<float*>(workspace);
  const uint16_t* xb = static_cast<const uint16_t*>(x);
  const uint16_t* wb = static_cast<const uint16_t*>(w_dkv);
  const uint16_t* nw = static_cast<const uint16_t*>(kv_norm_w);
  uint16_t* cb = static_cast<uint16_t*>(latent_cache);
  const int per = append_split_tokens(d, n_tokens);
  const bool gemm = append_split_gemm(d, n_tokens);
  const dim3 grid1(nks, (n_tokens + per - 1) / per, (d.latent_dim + d.rope_dim) / (gemm ? kGemmOut : 32));
  auto pass1 = [&](auto kernel) {
    hipLaunchKernelGGL(kernel, grid1, dim3(256), 0, stream, xb, wb, part, n_tokens, hidden, slice);
  };
  if (d.latent_dim == 128) {
    if (gemm) pass1(append_gemm_kernel<192>);
    else if (per == 32) pass1(append_slice_kernel<192, 1>);
    else pass1(append_slice_kernel<192, 2>);
    hipLaunchKernelGGL((append_finish_kernel<128, 64, 64>), dim3((n_tokens + 3) / 4), dim3(256), 0, stream, part,
                       nks, token_ids, positions, slots, nw, theta, cb, token_id_cache, num_slots, n_tokens);
  } else {
    if (gemm) pass1(append_gemm_kernel<576>);
    else if (per == 32) pass1(append_slice_kernel<576, 1>);
    else pass1(append_slice_kernel<576, 2>);
    // pass 2: a wave per token when the slices are few (4 tokens per
    // work-group), a work-group per token (one pair per thread) when many
    if (nks <= kAppFinishWaveSlices)
      hipLaunchKernelGGL((append_finish_kernel<512, 64, 64>), dim3((n_tokens + 3) / 4), dim3(256), 0, stream, part,
                         nks, token_ids, positions, slots, nw, theta, cb, token_id_cache, num_slots, n_tokens);
    else
      hipLaunchKernelGGL((append_finish_kernel<512, 64, 256>), dim3(n_tokens), dim3(256), 0, stream, part, nks,
                         token_ids, positions, slots, nw, theta, cb, token_id_cache, num_slots, n_tokens);
  }
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
