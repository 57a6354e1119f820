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
  const auto kern = use_ln ? (add ? literal_tile_kernel<true, true> : literal_tile_kernel<true, false>)
                           : (add ? literal_tile_kernel<false, true> : literal_tile_kernel<false, false>);
  const int lds = static_cast<int>(literal_lds_bytes(H));
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, lds) !=
      hipSuccess)
    return EG_MLA_ERR_HIP;
  const float scale_log2 = softmax_scale(d) * 1.4426950408889634f;
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
