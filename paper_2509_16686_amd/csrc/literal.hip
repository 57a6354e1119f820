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
// The LayerNorm is linear once a token's moments are known, so neither the
// gated rows nor the normalised ones are ever stored:
//   score  = tau (rstd (sum_d q_d w_d (x_d - K) - (mu - K) sum_d q_d w_d) + sum_d q_d b_d + q^R . k^R)
//   out    = w_v (sum_j a_j (x_j - mu_j)) / sum_j p_j + b_v,   a_j = p_j rstd_j.
// K is a per-token pivot (the token's first gated value): the moments and
// the key dots are sums of x - K, which stay of the size of the spread of x
// even when |mu| is many times sigma (no cancellation in m2 - m1^2), and the
// value pass centres each x on its token's mean before weighting it.
// Two kernels (bf16 storage, d_c = d_h = d_v = 128, d_r = 64):
//  1. literal_tile_kernel: one work-group per (sequence, 128 cached tokens),
//     4 waves of 32 tokens, split-K style.  Pass 1 walks the heads: one head's
//     W_UK and W_UV rows are staged in LDS (coalesced, the next head's rows
//     travel in registers meanwhile) and x = kv (.) g comes out of
//     v_mfma_f32_32x32x16_bf16 with a token's outputs in its own lanes, so the
//     token's moments and its key dots with q w are lane-local sums.  Then the
//     scores, the tile's max per head and a_j.  Pass 2 walks the heads again
//     for the value part with the operands swapped (a lane holds one value dim
//     for 16 tokens), its gate tile staged in LDS by whole 256-byte rows and
//     read back with ds_read_b64_tr_b16, so sum_j a_j x_j is 16 FMAs per lane
//     and one exchange between the lane halves.  Emits per (tile, head)
//     o = sum_j a_j (x_j - mu_j), the max and sum_j p_j.
//  2. literal_merge_kernel: one work-group per (sequence, head) rescales the
//     tiles' partials to a common max and applies the value part's affine.
// HBM traffic per cached token: its gate row once, plus the value half again
// in pass 2 (1.5 H (d_h + d_v) x 2 bytes), its cache row and id.

#include <hip/hip_runtime.h>

#include <cmath>
#include <type_traits>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr int kLtDC = 128, kLtDH = 128, kLtDV = 128, kLtDR = 64;
constexpr int kLtHeadW = kLtDH + kLtDV;  // gated dims per head
constexpr float kLtLnEps = 1e-5f;        // the listing's LayerNorm default
typedef __attribute__((ext_vector_type(16))) float lt_f32x16_t;

constexpr int kLtWRow = kLtDC + 8;  // padded LDS row of W (272 bytes: 16-lane reads hit 16 bank groups)
// LDS region R: pass 1 holds a head's 256 weight rows; pass 2 the head's 128
// W_UV rows and then four 8 KB value-gate tiles (32 tokens x 128 dims each)
constexpr int kLtRegion = kLtHeadW * kLtWRow * 2;
constexpr int kLtTileOff = kLtDV * kLtWRow;  // element offset of the gate tiles in R
static_assert(kLtTileOff * 2 + 4 * 32 * kLtDV * 2 <= kLtRegion, "pass-2 LDS layout");

// 16 bytes at a wave-uniform base plus a 32-bit lane offset (global_load with
// an SGPR base: one VGPR of address per lane however many pieces share it)
__device__ __forceinline__ u32x4_t ld_lane16(const uint16_t* base, uint32_t byte_off) {
  return *reinterpret_cast<const u32x4_t*>(reinterpret_cast<const unsigned char*>(base) + byte_off);
}

__device__ __forceinline__ float lane_half_sum(float v) {
  // lanes l and l + 32 exchange and add (both end with the sum)
  const uint32_t u = __float_as_uint(v);
  const auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

template <bool LN, bool ADD>
__global__ __launch_bounds__(256, 2) void literal_tile_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ cache, const int32_t* __restrict__ ids,
    const uint16_t* __restrict__ gate, const uint16_t* __restrict__ w_uk, const uint16_t* __restrict__ w_uv,
    const uint16_t* __restrict__ ln_w, const uint16_t* __restrict__ ln_b, const int32_t* __restrict__ seq_lens,
    const int32_t* __restrict__ page_table, int P, int max_pages, int64_t num_slots, int H, int V,
    float scale_log2, float* __restrict__ part) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lt_lds[];
  uint16_t* wsh = reinterpret_cast<uint16_t*>(lt_lds);        // region R
  float* kd = reinterpret_cast<float*>(lt_lds + kLtRegion);    // [4 waves][H][32 tokens]: key dot, score, a_j
  float* ob = kd + 4 * H * 32;                                 // [4][d_v] pass-2 sums; pass 1: q w of the head
  float* sqw = ob + 4 * kLtDV;                                 // [H] sum_d q_d w_d
  float* sqb = sqw + H;                                        // [H] sum_d q_d b_d
  float* wr = sqb + H;                                         // [2][4][H] per-wave max, sum p
  float* mus = wr + 12 * H;                                    // [4 waves][32 tokens] token means
  // at least one head (the host checks): every head loop runs, so no load is
  // left pending on a zero-trip path into the loops after it
  __builtin_assume(H >= 1);
  const int b = blockIdx.y, tile = blockIdx.x;
  const int L = clamp_len(seq_lens[b], P * max_pages);
  const int j0 = tile * 128;
  if (j0 >= L) return;  // whole work-group, before any barrier
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, t = lane & 31, hf = lane >> 5;
  const int j = j0 + 32 * w + t;
  const bool ok = j < L;  // positions past the sequence repeat its last token and get p = 0
  const int64_t row = cache_slot(page_table, b, min(j, L - 1), P, max_pages, num_slots);
  const int id = clamp_id(ids[row], V);
  const int width = H * kLtHeadW;
  const uint16_t* qb = q + static_cast<int64_t>(b) * H * (kLtDH + kLtDR);
  float* pb = part + (static_cast<int64_t>(b) * gridDim.x + tile) * H * (kLtDV + 4);
  bf16x8_t cb[kLtDC / 16];  // the token's latent, dims 16 c + 8 hf .. + 7 (an MFMA operand in both passes)
#pragma unroll
  for (int c = 0; c < kLtDC / 16; ++c)
    cb[c] = *reinterpret_cast<const bf16x8_t*>(cache + row * (kLtDC + kLtDR) + 16 * c + 8 * hf);

  // ---- pass 1: moments, key dots --------------------------------------------
  // LDS rows 0..127 (K half) hold W_UK[h], rows 128..255 (V half) W_UV[h].  The
  // K half is refilled with the next head's rows at the barrier after the key
  // blocks, the V half at the barrier that starts the next head, so each half
  // travels in registers (32 VGPRs) while the other half is read.
  constexpr int NB = LN ? 8 : 4;  // 32-output blocks per head: key and value part, or the key part only
  // weight pieces: thread tid takes rows tid / 16 + 16 i, 16-byte chunk tid % 16;
  // the base of piece i is wave-uniform, the lane's byte offset is the same for all
  const uint32_t woff = ((tid >> 4) * kLtDC + (tid & 15) * 8) * 2;
  u32x4_t ws[8];
  auto fetch_half = [&](const uint16_t* wmat, int head) {
#pragma unroll
    for (int i = 0; i < 8; ++i) ws[i] = ld_lane16(wmat + (static_cast<int64_t>(head) * kLtDH + 16 * i) * kLtDC, woff);
  };
  auto put_half = [&](int half) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = tid + 256 * i;
      *reinterpret_cast<u32x4_t*>(wsh + (half * kLtDH + (p >> 4)) * kLtWRow + (p & 15) * 8) = ws[i];
    }
  };
  uint32_t qn = 0, wn = 0;  // q and the LayerNorm weight at dim tid % 128 of the next head
  auto fetch_qa = [&](int head) {
    qn = qb[head * (kLtDH + kLtDR) + (tid & 127)];
    wn = LN ? ln_w[head * kLtHeadW + (tid & 127)] : 0x3f80u;  // bf16 1.0 without a LayerNorm
  };
  auto put_qa = [&]() {
    if (tid < kLtDH) ob[tid] = bf16_to_f32(static_cast<uint16_t>(qn)) * bf16_to_f32(static_cast<uint16_t>(wn));
  };
  const uint16_t* grow = gate + static_cast<int64_t>(id) * width + 4 * hf;
  u32x2_t gv[4][4];  // gate words of the block 4 ahead (ring slot = block % 4)
  auto fetch_g = [&](int head, int blk) {
#pragma unroll
    for (int qq = 0; qq < 4; ++qq)
      gv[blk & 3][qq] = *reinterpret_cast<const u32x2_t*>(grow + head * kLtHeadW + 32 * blk + 8 * qq);
  };
  // issue order as in the loop (the V half's rows older than the 16 gate loads),
  // so the waits at the loop head stay partial on entry too
  fetch_half(w_uk, 0);
  fetch_qa(0);
  put_half(0);
  put_qa();
  if (LN) fetch_half(w_uv, 0);
  __builtin_amdgcn_sched_barrier(0);  // keep that order
#pragma unroll
  for (int blk = 0; blk < 4; ++blk) fetch_g(0, blk);
  __builtin_amdgcn_sched_barrier(0);
  if (LN) {
    // sum_d q_d w_d and sum_d q_d b_d of every head (a wave covers 64 dims of one head)
    for (int i = tid; i < H * kLtDH; i += 256) {
      const int hh = i >> 7, d = i & 127;
      const float qd = bf16_to_f32(qb[hh * (kLtDH + kLtDR) + d]);
      const float pw = wave_sum(qd * bf16_to_f32(ln_w[hh * kLtHeadW + d]));
      const float pbias = wave_sum(qd * bf16_to_f32(ln_b[hh * kLtHeadW + d]));
      if (lane == 0) {
        kd[2 * (i >> 6)] = pw;
        kd[2 * (i >> 6) + 1] = pbias;
      }
    }
    __syncthreads();
    for (int hh = tid; hh < H; hh += 256) {
      sqw[hh] = kd[4 * hh] + kd[4 * hh + 2];
      sqb[hh] = kd[4 * hh + 1] + kd[4 * hh + 3];
    }
  }
  // moments of the token's x - K (K: the pivot) and the key dots sum q w (x - K)
  float s1 = 0.f, s2 = 0.f, K = 0.f;
  auto block = [&](int head, int blk, float& kdp) {
    lt_f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
    const uint16_t* arow = wsh + (32 * blk + t) * kLtWRow + 8 * hf;
#pragma unroll
    for (int c = 0; c < kLtDC / 16; ++c)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(*reinterpret_cast<const bf16x8_t*>(arow + 16 * c), cb[c], acc, 0,
                                                    0, 0);
    // lane holds outputs 32 blk + 8 qq + 4 hf + e of its token in acc[4 qq + e]
    if (LN && blk == 0) {
      // pivot: the token's first gated value (output 0 of head 0, in the lane
      // half hf = 0), the same in both halves; set on the first head only
      const uint32_t gw = gv[0][0][0];
      const float x0 = ADD ? acc[0] + bf16_lo(gw) : acc[0] * bf16_lo(gw);
      const uint32_t u = __float_as_uint(x0);
      const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
      K = head == 0 ? __uint_as_float(sw[0]) : K;
    }
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      float4 qa = make_float4(0.f, 0.f, 0.f, 0.f);
      if (blk < 4) qa = *reinterpret_cast<const float4*>(ob + 32 * blk + 8 * qq + 4 * hf);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const uint32_t gw = gv[blk & 3][qq][e >> 1];
        const float g = (e & 1) ? bf16_hi(gw) : bf16_lo(gw);
        const float x = (ADD ? acc[4 * qq + e] + g : acc[4 * qq + e] * g) - K;  // K = 0 without a LayerNorm
        if (LN) {
          s1 += x;
          s2 = fmaf(x, x, s2);
        }
        if (blk < 4) kdp = fmaf((&qa.x)[e], x, kdp);
      }
    }
    const int nxt = min(head + 1, H - 1);
    if (blk + 4 < NB)
      fetch_g(head, blk + 4);
    else
      fetch_g(nxt, blk + 4 - NB);
    __builtin_amdgcn_sched_barrier(0);  // one block's operands and accumulator live at a time
  };
  for (int head = 0; head < H; ++head) {
    // the next head's operands (the last head fetches itself again: no branch in the loop)
    const int nxt = min(head + 1, H - 1);
    __syncthreads();  // K half and q w of this head visible; the V half is free
    if (LN) put_half(1);
    fetch_half(w_uk, nxt);
    fetch_qa(nxt);
    float kdp = 0.f;
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) block(head, blk, kdp);
    const float kdf = lane_half_sum(kdp);
    if (hf == 0) kd[(w * H + head) * 32 + t] = kdf;
    __syncthreads();  // every wave is done with the K half (and q w); the V half is visible
    put_half(0);
    put_qa();
    if (LN) {
      fetch_half(w_uv, nxt);
#pragma unroll
      for (int blk = 4; blk < NB; ++blk) block(head, blk, kdp);
    }
  }

  // ---- scores, the tile's softmax statistics ---------------------------------
  // pass 2's first operands travel while the scores are formed
  // W_UV rows (8 pieces per thread, one head ahead) and the wave's value-gate
  // tile (8 pieces per lane) of the next two heads: ga for even heads, gb for odd
  u32x4_t vs[8], ga[8], gb[8];
  int idk[8];            // ids of tokens 4 k + lane / 16 of this wave
#pragma unroll
  for (int k = 0; k < 8; ++k) idk[k] = __shfl(id, 4 * k + (lane >> 4), 64);
  uint32_t goff[8];  // byte offsets of those tokens' gate rows (the gate table is below 4 GB)
#pragma unroll
  for (int k = 0; k < 8; ++k) goff[k] = (static_cast<uint32_t>(idk[k]) * width + (lane & 15) * 8) * 2;
  auto fetch_v = [&](int head) {
#pragma unroll
    for (int i = 0; i < 8; ++i) vs[i] = ld_lane16(w_uv + (static_cast<int64_t>(head) * kLtDV + 16 * i) * kLtDC, woff);
  };
  auto fetch_gt = [&](u32x4_t (&g)[8], int head) {
#pragma unroll
    for (int k = 0; k < 8; ++k) g[k] = ld_lane16(gate + head * kLtHeadW + kLtDH, goff[k]);
  };
  fetch_v(0);
  fetch_gt(ga, 0);
  fetch_gt(gb, min(1, H - 1));
  u32x4_t kr[2];  // q^R . k^R: lane half hf takes RoPE dims 32 hf .. + 31
  kr[0] = *reinterpret_cast<const u32x4_t*>(cache + row * (kLtDC + kLtDR) + kLtDC + 32 * hf);
  kr[1] = *reinterpret_cast<const u32x4_t*>(cache + row * (kLtDC + kLtDR) + kLtDC + 32 * hf + 8);
  u32x4_t kr2[2];
  kr2[0] = *reinterpret_cast<const u32x4_t*>(cache + row * (kLtDC + kLtDR) + kLtDC + 32 * hf + 16);
  kr2[1] = *reinterpret_cast<const u32x4_t*>(cache + row * (kLtDC + kLtDR) + kLtDC + 32 * hf + 24);
  __syncthreads();  // region R is free
  float* qrs = reinterpret_cast<float*>(lt_lds);  // [H][d_r]
  for (int i = tid; i < H * kLtDR; i += 256) qrs[i] = bf16_to_f32(qb[(i >> 6) * (kLtDH + kLtDR) + kLtDH + (i & 63)]);
  float mu = 0.f, dmu = 0.f, rstd = 1.f;  // mean, mean - K, 1 / sigma
  if (LN) {
    // moments about the pivot: m1 = mean(x - K) is of the size of sigma or a
    // few sigma, so m2 - m1^2 keeps its precision
    const float m1 = lane_half_sum(s1) / static_cast<float>(width);
    const float m2 = lane_half_sum(s2) / static_cast<float>(width);
    dmu = m1;
    mu = K + m1;
    rstd = 1.0f / sqrtf(fmaxf(m2 - m1 * m1, 0.f) + kLtLnEps);
    if (hf == 0) mus[w * 32 + t] = mu;
  }
  __syncthreads();
  for (int head = 0; head < H; ++head) {
    const float* qr = qrs + head * kLtDR + 32 * hf;
    float rp = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const u32x4_t v = c < 2 ? kr[c] : kr2[c - 2];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        rp = fmaf(qr[8 * c + 2 * e], bf16_lo(v[e]), rp);
        rp = fmaf(qr[8 * c + 2 * e + 1], bf16_hi(v[e]), rp);
      }
    }
    const float rd = lane_half_sum(rp);
    float* kp = kd + (w * H + head) * 32 + t;
    const float dot = *kp;
    const float base = LN ? rstd * (dot - dmu * sqw[head]) + sqb[head] : dot;
    const float s = ok ? scale_log2 * (base + rd) : -INFINITY;
    const float wm = wave_max(s);
    if (hf == 0) *kp = s;
    if (lane == 0) wr[w * H + head] = wm;
  }
  __syncthreads();
  for (int head = 0; head < H; ++head) {
    const float m = fmaxf(fmaxf(wr[head], wr[H + head]), fmaxf(wr[2 * H + head], wr[3 * H + head]));
    float* kp = kd + (w * H + head) * 32 + t;
    const float p = exp2f(*kp - m);  // 0 past the sequence
    const float a = p * rstd;
    // both lane halves hold the same token: half of the wave sum is exact
    const float sp = 0.5f * wave_sum(p);
    __builtin_amdgcn_wave_barrier();
    if (hf == 0) *kp = a;
    if (lane == 0) wr[(4 + w) * H + head] = sp;
  }
  __syncthreads();
  for (int hh = tid; hh < H; hh += 256) {
    float* rec = pb + hh * (kLtDV + 4) + kLtDV;
    rec[0] = fmaxf(fmaxf(wr[hh], wr[H + hh]), fmaxf(wr[2 * H + hh], wr[3 * H + hh]));
    rec[1] = (wr[4 * H + hh] + wr[5 * H + hh]) + (wr[6 * H + hh] + wr[7 * H + hh]);
  }

  // ---- pass 2: sum_j a_j x_j of the value part ---------------------------------
  uint16_t* gt = wsh + kLtTileOff + w * (32 * kLtDV);  // this wave's tile: [token][d_v], 32-byte groups swizzled
  const int r16 = lane & 15, G1 = (lane >> 4) & 1;
  auto flush = [&](int head) {  // the four waves' sums of a finished head
    if (tid < kLtDV)
      pb[head * (kLtDV + 4) + tid] = (ob[tid] + ob[kLtDV + tid]) + (ob[2 * kLtDV + tid] + ob[3 * kLtDV + tid]);
  };
  auto stage = [&](const u32x4_t (&g)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int p = tid + 256 * i;
      *reinterpret_cast<u32x4_t*>(wsh + (p >> 4) * kLtWRow + (p & 15) * 8) = vs[i];
    }
    // piece (token 4 k + lane / 16, 16-byte chunk c8 = lane % 16): 32-byte group c8 / 2 of a row
    // lands in group (c8 / 2) ^ (token % 4), so a transposed read of 4 rows hits 4 bank ranges
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int tok = 4 * k + (lane >> 4), c8 = lane & 15;
      *reinterpret_cast<u32x4_t*>(gt + tok * kLtDV + 16 * ((c8 >> 1) ^ (tok & 3)) + 8 * (c8 & 1)) = g[k];
    }
  };
  auto values = [&](int head) {
    // a_j and mu_j of tokens 8 qq + 4 hf + i (the rows of this lane's accumulator registers)
    float4 av[4], mv[4];
#pragma unroll
    for (int qq = 0; qq < 4; ++qq) {
      av[qq] = *reinterpret_cast<const float4*>(kd + (w * H + head) * 32 + 8 * qq + 4 * hf);
      mv[qq] = LN ? *reinterpret_cast<const float4*>(mus + w * 32 + 8 * qq + 4 * hf) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int blk = 0; blk < kLtDV / 32; ++blk) {
      lt_f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
      const uint16_t* brow = wsh + (32 * blk + t) * kLtWRow + 8 * hf;
#pragma unroll
      for (int c = 0; c < kLtDC / 16; ++c)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cb[c], *reinterpret_cast<const bf16x8_t*>(brow + 16 * c), acc,
                                                      0, 0, 0);
      // acc[4 qq + i]: token 8 qq + 4 hf + i, value dim 32 blk + t
      float o = 0.f;
#pragma unroll
      for (int qq = 0; qq < 4; ++qq) {
        const int tr = 8 * qq + 4 * hf + (r16 >> 2);  // the row this lane addresses
        const uint16_t* gp = gt + tr * kLtDV + 16 * ((2 * blk + G1) ^ (r16 >> 2)) + 4 * (r16 & 3);
        const s16x4_t g4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)gp);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float g = bf16_to_f32(static_cast<uint16_t>(g4[i]));
          const float x = (ADD ? acc[4 * qq + i] + g : acc[4 * qq + i] * g) - (&mv[qq].x)[i];  // x - mu_j
          o = fmaf((&av[qq].x)[i], x, o);
        }
      }
      o = lane_half_sum(o);
      if (hf == 0) ob[w * kLtDV + 32 * blk + t] = o;
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // heads in pairs, so the two gate-tile register sets keep fixed names; each
  // set is refilled two heads ahead, the W_UV rows one head ahead
  // (whole pairs in the loop and an odd last head after it, so the loop's back
  // edge follows the odd head and the waits at its top stay partial)
  int head = 0;
  for (; head + 1 < H; head += 2) {
    __syncthreads();  // R and ob are free (previous head computed, its sums read)
    if (head > 0) flush(head - 1);
    stage(ga);
    __syncthreads();
    fetch_v(head + 1);
    fetch_gt(ga, min(head + 2, H - 1));
    values(head);
    __syncthreads();
    flush(head);
    stage(gb);
    __syncthreads();
    fetch_v(min(head + 2, H - 1));
    fetch_gt(gb, min(head + 3, H - 1));
    values(head + 1);
  }
  if (head < H) {  // the last of an odd head count: its operands are in vs and ga
    __syncthreads();
    if (head > 0) flush(head - 1);
    stage(ga);
    __syncthreads();
    values(head);
  }
  __syncthreads();
  flush(H - 1);
}

// out[b, h, v] from the tiles' partials: rescale to the common max, then the
// value part's LayerNorm affine (identity without the LayerNorm).
__global__ __launch_bounds__(128) void literal_merge_kernel(const float* __restrict__ part,
                                                            const uint16_t* __restrict__ ln_w,
                                                            const uint16_t* __restrict__ ln_b, int use_ln,
                                                            const int32_t* __restrict__ seq_lens, int cap, int tiles,
                                                            int H, uint16_t* __restrict__ out) {
  const int hh = blockIdx.x, b = blockIdx.y, v = threadIdx.x;
  const int L = clamp_len(seq_lens[b], cap);
  const int nt = (L + 127) / 128;
  uint16_t* orow = out + (static_cast<int64_t>(b) * H + hh) * kLtDV;
  if (nt == 0) {
    orow[v] = 0;
    return;
  }
  const int64_t stride = static_cast<int64_t>(H) * (kLtDV + 4);
  const float* pp = part + static_cast<int64_t>(b) * tiles * stride + hh * (kLtDV + 4);
  // 8 tiles' loads at a time (independent, so one round trip per 8 tiles)
  float m = -INFINITY;
  for (int i0 = 0; i0 < nt; i0 += 8) {
    float mk[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) mk[k] = i0 + k < nt ? pp[(i0 + k) * stride + kLtDV] : -INFINITY;
#pragma unroll
    for (int k = 0; k < 8; ++k) m = fmaxf(m, mk[k]);
  }
  float o = 0.f, l = 0.f;
  for (int i0 = 0; i0 < nt; i0 += 8) {
    float ok_[8], mk[8], lk[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float* rec = pp + min(i0 + k, nt - 1) * stride;
      ok_[k] = rec[v];
      mk[k] = i0 + k < nt ? rec[kLtDV] : -INFINITY;  // a missing tile weighs 0
      lk[k] = rec[kLtDV + 1];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const float e = exp2f(mk[k] - m);
      o = fmaf(e, ok_[k], o);
      l = fmaf(e, lk[k], l);
    }
  }
  const float wv = use_ln ? bf16_to_f32(ln_w[hh * kLtHeadW + kLtDH + v]) : 1.f;
  const float bv = use_ln ? bf16_to_f32(ln_b[hh * kLtHeadW + kLtDH + v]) : 0.f;
  orow[v] = f32_to_bf16(wv * o / l + bv);  // o: sum of a_j (x_j - mu_j), already centred
}

// ---------------------------------------------------------------------------
// Other shapes (any d_c, d_h, d_v, d_r and head count that fit the LDS, bf16 or
// fp32 storage): the same arithmetic as the tile kernel (the LayerNorm applied
// through each token's moments about a pivot, its first gated value; scores in
// the log2 domain; per 128-token tile and head the record (o, max, sum) that
// the merge combines) in plain fp32 VALU code.  One work-group of 4 waves per
// (sequence, 128-token tile) walks the tile in groups of 8 tokens: their
// latents go to LDS; in pass A wave w takes heads w, w + 4, ..., its lanes a
// head's up-projected outputs 64 at a time, each lane one W row against the 8
// latents (broadcast LDS reads, so a row is read once per 8 tokens), forming
// the tokens' moments and the heads' key dots; then an online softmax per head
// (state in LDS); pass B the value sums the same way.  Not tuned: it serves
// the layers the tile kernel does not take.
// ---------------------------------------------------------------------------
constexpr int kLgTok = 8;  // tokens per group

struct LiteralGenericArgs {
  const void* q;
  const void* cache;
  const int32_t* ids;
  const void* gate;
  const void* w_uk;
  const void* w_uv;
  const void* ln_w;
  const void* ln_b;
  const int32_t* seq_lens;
  const int32_t* page_table;
  int P, max_pages;
  int64_t num_slots;
  int H, DH, DV, DC, DR, V;
  float scale_log2;
  float* part;
};

template <bool BF16, bool LN, bool ADD>
__global__ __launch_bounds__(256) void literal_generic_tile_kernel(LiteralGenericArgs a) {
  extern __shared__ float lg[];
  const int H = a.H, DH = a.DH, DV = a.DV, DC = a.DC, DR = a.DR, HW = DH + DV;
  float* cs = lg;                      // [8][d_c] the group's latents
  float* kdot = cs + kLgTok * DC;      // [8][H] key dots sum q w (x - K)
  float* pst = kdot + kLgTok * H;      // [8][H] weights of the value sums (p, or p rstd)
  float* mom = pst + kLgTok * H;       // [4 waves][8][2] moment sums
  float* tokf = mom + 4 * kLgTok * 2;  // [3][8] pivot K, mean - K, rstd
  float* sq = tokf + 3 * kLgTok;       // [2][H] sum q w, sum q b (key dims)
  float* hst = sq + 2 * H;             // [3][H] running max, sum, this group's rescale
  float* ob = hst + 3 * H;             // [H][d_v] value sums
  const int b = blockIdx.y, tile = blockIdx.x;
  const int L = clamp_len(a.seq_lens[b], a.P * a.max_pages);
  const int j0 = tile * 128;
  if (j0 >= L) return;  // whole work-group, before any barrier
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int nj = min(128, L - j0);
  const int64_t qb = static_cast<int64_t>(b) * H * (DH + DR);
  const int64_t grow_len = static_cast<int64_t>(H) * HW;
  for (int h = w; h < H; h += 4) {
    float sw = 0.f, sb = 0.f;
    if (LN) {
      for (int d = lane; d < DH; d += 64) {
        const float qd = ld<BF16>(a.q, qb + static_cast<int64_t>(h) * (DH + DR) + d);
        sw = fmaf(qd, ld<BF16>(a.ln_w, static_cast<int64_t>(h) * HW + d), sw);
        sb = fmaf(qd, ld<BF16>(a.ln_b, static_cast<int64_t>(h) * HW + d), sb);
      }
    }
    sw = wave_sum(sw);
    sb = wave_sum(sb);
    if (lane == 0) {
      sq[h] = sw;
      sq[H + h] = sb;
      hst[h] = -INFINITY;
      hst[H + h] = 0.f;
    }
  }
  for (int i = tid; i < H * DV; i += 256) ob[i] = 0.f;
  __syncthreads();
  for (int g0 = 0; g0 < nj; g0 += kLgTok) {
    // the group's tokens (past the tile's end the last token again, weight 0)
    int64_t rowk[kLgTok];
    int idk[kLgTok];
#pragma unroll
    for (int k = 0; k < kLgTok; ++k) {
      rowk[k] = cache_slot(a.page_table, b, j0 + min(g0 + k, nj - 1), a.P, a.max_pages, a.num_slots);
      idk[k] = clamp_id(a.ids[rowk[k]], a.V);
    }
    for (int i = tid; i < kLgTok * DC; i += 256) cs[i] = ld<BF16>(a.cache, rowk[i / DC] * (DC + DR) + i % DC);
    __syncthreads();
    if (tid < kLgTok) {
      // pivot: the token's first gated value (output 0 of head 0); none without a LayerNorm
      float x = 0.f;
      for (int c = 0; c < DC; ++c) x = fmaf(ld<BF16>(a.w_uk, c), cs[tid * DC + c], x);
      const float gg = ld<BF16>(a.gate, static_cast<int64_t>(idk[tid]) * grow_len);
      tokf[tid] = LN ? (ADD ? x + gg : x * gg) : 0.f;
    }
    __syncthreads();
    float piv[kLgTok];
#pragma unroll
    for (int k = 0; k < kLgTok; ++k) piv[k] = tokf[k];
    // ---- pass A: moments about the pivot, key dots ----
    float s1[kLgTok], s2[kLgTok];
#pragma unroll
    for (int k = 0; k < kLgTok; ++k) s1[k] = s2[k] = 0.f;
    for (int h = w; h < H; h += 4) {
      float kd[kLgTok];
#pragma unroll
      for (int k = 0; k < kLgTok; ++k) kd[k] = 0.f;
      for (int e = lane; e < HW; e += 64) {
        const bool isk = e < DH;
        const void* wm = isk ? a.w_uk : a.w_uv;
        const int64_t wrow = (static_cast<int64_t>(h) * (isk ? DH : DV) + (isk ? e : e - DH)) * DC;
        float x[kLgTok];
#pragma unroll
        for (int k = 0; k < kLgTok; ++k) x[k] = 0.f;
        for (int c = 0; c < DC; ++c) {
          const float wc = ld<BF16>(wm, wrow + c);
#pragma unroll
          for (int k = 0; k < kLgTok; ++k) x[k] = fmaf(wc, cs[k * DC + c], x[k]);
        }
        const float qw = isk ? ld<BF16>(a.q, qb + static_cast<int64_t>(h) * (DH + DR) + e) *
                                   (LN ? ld<BF16>(a.ln_w, static_cast<int64_t>(h) * HW + e) : 1.f)
                             : 0.f;
#pragma unroll
        for (int k = 0; k < kLgTok; ++k) {
          const float gg = ld<BF16>(a.gate, static_cast<int64_t>(idk[k]) * grow_len + static_cast<int64_t>(h) * HW + e);
          const float y = (ADD ? x[k] + gg : x[k] * gg) - piv[k];
          s1[k] += y;
          s2[k] = fmaf(y, y, s2[k]);
          kd[k] = fmaf(qw, y, kd[k]);
        }
      }
#pragma unroll
      for (int k = 0; k < kLgTok; ++k) {
        const float t = wave_sum(kd[k]);
        if (lane == 0) kdot[k * H + h] = t;
      }
    }
#pragma unroll
    for (int k = 0; k < kLgTok; ++k) {
      const float t1 = wave_sum(s1[k]), t2 = wave_sum(s2[k]);
      if (lane == 0) {
        mom[(w * kLgTok + k) * 2] = t1;
        mom[(w * kLgTok + k) * 2 + 1] = t2;
      }
    }
    __syncthreads();
    if (tid < kLgTok) {
      const float n = static_cast<float>(grow_len);
      float t1 = 0.f, t2 = 0.f;
      for (int v = 0; v < 4; ++v) {
        t1 += mom[(v * kLgTok + tid) * 2];
        t2 += mom[(v * kLgTok + tid) * 2 + 1];
      }
      const float m1 = t1 / n, m2 = t2 / n;
      tokf[kLgTok + tid] = LN ? m1 : 0.f;  // mean - K
      tokf[2 * kLgTok + tid] = LN ? 1.0f / sqrtf(fmaxf(m2 - m1 * m1, 0.f) + kLtLnEps) : 1.f;
    }
    __syncthreads();
    // ---- scores and the online softmax of each head ----
    for (int h = tid; h < H; h += 256) {
      float sc[kLgTok], mx = -INFINITY;
#pragma unroll
      for (int k = 0; k < kLgTok; ++k) {
        const float base = LN ? tokf[2 * kLgTok + k] * (kdot[k * H + h] - tokf[kLgTok + k] * sq[h]) + sq[H + h]
                              : kdot[k * H + h];
        float rd = 0.f;
        for (int r = 0; r < DR; ++r)
          rd = fmaf(ld<BF16>(a.q, qb + static_cast<int64_t>(h) * (DH + DR) + DH + r),
                    ld<BF16>(a.cache, rowk[k] * (DC + DR) + DC + r), rd);
        sc[k] = g0 + k < nj ? a.scale_log2 * (base + rd) : -INFINITY;
        mx = fmaxf(mx, sc[k]);
      }
      const float m_new = fmaxf(hst[h], mx);  // finite: token g0 is in the tile
      const float alpha = exp2f(hst[h] - m_new);
      float l = hst[H + h] * alpha;
#pragma unroll
      for (int k = 0; k < kLgTok; ++k) {
        const float p = exp2f(sc[k] - m_new);
        l += p;
        pst[k * H + h] = LN ? p * tokf[2 * kLgTok + k] : p;
      }
      hst[h] = m_new;
      hst[H + h] = l;
      hst[2 * H + h] = alpha;
    }
    __syncthreads();
    // ---- pass B: value sums (centred on each token's mean with a LayerNorm) ----
    for (int h = w; h < H; h += 4) {
      const float alpha = hst[2 * H + h];
      for (int e = lane; e < DV; e += 64) {
        const int64_t wrow = (static_cast<int64_t>(h) * DV + e) * DC;
        float x[kLgTok];
#pragma unroll
        for (int k = 0; k < kLgTok; ++k) x[k] = 0.f;
        for (int c = 0; c < DC; ++c) {
          const float wc = ld<BF16>(a.w_uv, wrow + c);
#pragma unroll
          for (int k = 0; k < kLgTok; ++k) x[k] = fmaf(wc, cs[k * DC + c], x[k]);
        }
        float acc = ob[h * DV + e] * alpha;
#pragma unroll
        for (int k = 0; k < kLgTok; ++k) {
          const float gg =
              ld<BF16>(a.gate, static_cast<int64_t>(idk[k]) * grow_len + static_cast<int64_t>(h) * HW + DH + e);
          const float xg = ADD ? x[k] + gg : x[k] * gg;
          acc = fmaf(pst[k * H + h], LN ? xg - (piv[k] + tokf[kLgTok + k]) : xg, acc);
        }
        ob[h * DV + e] = acc;
      }
    }
    __syncthreads();  // the next group overwrites the latents and the weights
  }
  // the tile's records: o, the maximum, the sum (as the tile kernel's)
  float* pb = a.part + (static_cast<int64_t>(b) * gridDim.x + tile) * H * (DV + 4);
  for (int i = tid; i < H * DV; i += 256) pb[static_cast<int64_t>(i / DV) * (DV + 4) + i % DV] = ob[i];
  for (int h = tid; h < H; h += 256) {
    pb[static_cast<int64_t>(h) * (DV + 4) + DV] = hst[h];
    pb[static_cast<int64_t>(h) * (DV + 4) + DV + 1] = hst[H + h];
  }
}

// The merge for the generic tile kernel's records (any d_v, bf16 or fp32 output).
template <bool BF16>
__global__ __launch_bounds__(256) void literal_generic_merge_kernel(const float* __restrict__ part,
                                                                    const void* __restrict__ ln_w,
                                                                    const void* __restrict__ ln_b, int use_ln,
                                                                    const int32_t* __restrict__ seq_lens, int cap,
                                                                    int tiles, int H, int DH, int DV,
                                                                    void* __restrict__ out) {
  const int hh = blockIdx.x, b = blockIdx.y;
  const int L = clamp_len(seq_lens[b], cap);
  const int nt = (L + 127) / 128;
  const int64_t obase = (static_cast<int64_t>(b) * H + hh) * DV;
  if (nt == 0) {
    for (int v = threadIdx.x; v < DV; v += 256) st<BF16>(out, obase + v, 0.f);
    return;
  }
  const int64_t stride = static_cast<int64_t>(H) * (DV + 4);
  const float* pp = part + static_cast<int64_t>(b) * tiles * stride + static_cast<int64_t>(hh) * (DV + 4);
  float m = -INFINITY;
  for (int i = 0; i < nt; ++i) m = fmaxf(m, pp[i * stride + DV]);
  for (int v = threadIdx.x; v < DV; v += 256) {
    float o = 0.f, l = 0.f;
    for (int i = 0; i < nt; ++i) {
      const float e = exp2f(pp[i * stride + DV] - m);
      o = fmaf(e, pp[i * stride + v], o);
      l = fmaf(e, pp[i * stride + DV + 1], l);
    }
    const int64_t c = static_cast<int64_t>(hh) * (DH + DV) + DH + v;
    const float wv = use_ln ? ld<BF16>(ln_w, c) : 1.f;
    const float bv = use_ln ? ld<BF16>(ln_b, c) : 0.f;
    st<BF16>(out, obase + v, wv * o / l + bv);
  }
}

}  // namespace egmla

using namespace egmla;

extern "C" size_t eg_mla_decode_literal_workspace_size(const eg_mla_dims* dims, int32_t batch,
                                                       int32_t max_pages_per_seq) {
  if (check_dims(dims) != EG_MLA_OK || batch < 0 || max_pages_per_seq < 0) return 0;
  return literal_workspace_bytes(*dims, batch, max_pages_per_seq);
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
  const int P = d.page_size, cap = P * max_pages_per_seq, tiles = (cap + 127) / 128, H = d.num_heads;
  float* part = static_cast<float*>(workspace);
  const bool use_ln = (flags & EG_MLA_LITERAL_NO_LN) == 0;
  const bool add = (flags & EG_MLA_LITERAL_ADD) != 0;
  const float scale_log2 = softmax_scale(d) * 1.4426950408889634f;
  if (!literal_tile_shape(d)) {
    LiteralGenericArgs g;
    g.q = q;
    g.cache = latent_cache;
    g.ids = token_id_cache;
    g.gate = gate_full;
    g.w_uk = w_uk;
    g.w_uv = w_uv;
    g.ln_w = ln_weight;
    g.ln_b = ln_bias;
    g.seq_lens = seq_lens;
    g.page_table = page_table;
    g.P = P;
    g.max_pages = max_pages_per_seq;
    g.num_slots = num_slots;
    g.H = H;
    g.DH = d.head_dim;
    g.DV = d.v_head_dim;
    g.DC = d.latent_dim;
    g.DR = d.rope_dim;
    g.V = d.vocab_size;
    g.scale_log2 = scale_log2;
    g.part = part;
    const bool bf = d.dtype == EG_MLA_BF16;
    auto pick = [&](auto b16) {
      constexpr bool BF = decltype(b16)::value;
      return use_ln ? (add ? literal_generic_tile_kernel<BF, true, true> : literal_generic_tile_kernel<BF, true, false>)
                    : (add ? literal_generic_tile_kernel<BF, false, true>
                           : literal_generic_tile_kernel<BF, false, false>);
    };
    const auto gk = bf ? pick(std::true_type{}) : pick(std::false_type{});
    const int glds = static_cast<int>(literal_generic_lds_bytes(d));
    if (glds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(gk),
                                            hipFuncAttributeMaxDynamicSharedMemorySize, glds) != hipSuccess)
      return EG_MLA_ERR_HIP;
    hipLaunchKernelGGL(gk, dim3(tiles, batch), dim3(256), glds, stream, g);
    const auto mk = bf ? literal_generic_merge_kernel<true> : literal_generic_merge_kernel<false>;
    hipLaunchKernelGGL(mk, dim3(H, batch), dim3(256), 0, stream, part, ln_weight, ln_bias, use_ln ? 1 : 0, seq_lens,
                       cap, tiles, H, d.head_dim, d.v_head_dim, out);
    return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
  }
  const auto kern = use_ln ? (add ? literal_tile_kernel<true, true> : literal_tile_kernel<true, false>)
                           : (add ? literal_tile_kernel<false, true> : literal_tile_kernel<false, false>);
  const int lds = static_cast<int>(literal_lds_bytes(H));
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, lds) !=
      hipSuccess)
    return EG_MLA_ERR_HIP;
  hipLaunchKernelGGL(kern, dim3(tiles, batch), dim3(256), lds, stream, static_cast<const uint16_t*>(q),
                     static_cast<const uint16_t*>(latent_cache), token_id_cache, static_cast<const uint16_t*>(gate_full),
                     static_cast<const uint16_t*>(w_uk), static_cast<const uint16_t*>(w_uv),
                     static_cast<const uint16_t*>(ln_weight), static_cast<const uint16_t*>(ln_bias), seq_lens,
                     page_table, P, max_pages_per_seq, num_slots, H, d.vocab_size, scale_log2, part);
  hipLaunchKernelGGL(literal_merge_kernel, dim3(H, batch), dim3(kLtDV), 0, stream, part,
                     static_cast<const uint16_t*>(ln_weight), static_cast<const uint16_t*>(ln_bias), use_ln ? 1 : 0,
                     seq_lens, cap, tiles, H, static_cast<uint16_t*>(out));
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
