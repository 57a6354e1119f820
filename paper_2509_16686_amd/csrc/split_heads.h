// Head-split MFMA split kernel of EG-MLA decode for many heads and a wide
// latent (bf16 storage, 128 heads per work-group, d_c = 512, d_r = 64).
// Included by decode.hip after SplitArgs.
//
// One work-group of 8 waves per (sequence, split, block of 128 heads); wave w
// owns heads 16w .. 16w + 15.  The split's tokens are taken 16 at a time (a
// tile).  For a tile, the whole work-group
//   * loads the rows and gate rows into registers (each thread: 2 x 16 bytes
//     of latent, the matching 2 x 16 bytes of gate, and 16 bytes of the RoPE
//     key for the first 128 threads), one tile ahead of its use;
//   * gates in fp32 (exact products, one bf16 rounding) and stores the gated
//     tile, with its RoPE keys, row-major in one of two LDS buffers (one
//     barrier per tile);
// then every wave, for its own 16 heads,
//   * computes S^T[token][head] on v_mfma_f32_16x16x32_bf16: A operand from
//     the LDS tile (lane: token lane%16, 8 consecutive dims), B operand the
//     absorbed query, rounded to bf16 and kept in registers (the query rounding
//     adds a relative error of 2^-9 per element, of the same size as the gated
//     latent's own rounding);
//   * runs the online softmax on the accumulator layout (lane: one head, 4
//     tokens), rescaling only when a head's maximum grows by more than 2^8;
//   * accumulates O^T[dim][head] += C~^T x P^T for all d_c dims, the A operand
//     read with ds_read_b64_tr_b16 (16-lane transpose) and P already in the B
//     operand layout of v_mfma_f32_16x16x16_bf16.
// The waves' heads are disjoint, so each writes its own part of the split's
// partial result; nothing is merged inside the work-group.
#pragma once

namespace egmla {

template <int DC, int DR>
struct HsplitCfg {
  static constexpr int NW = 8;                   // waves = head groups of 16
  static constexpr int NT = NW * 64;             // threads
  static constexpr int NC = DC / 32;             // 32-dim latent chunks (score MFMA steps)
  static constexpr int NR = DR / 32;             // 32-dim RoPE chunks
  static constexpr int NB = DC / 16;             // 16-dim blocks of the value product
  static constexpr int TS = DC + DR + 8;         // bf16 elements per LDS tile row (16 bytes of padding)
  static constexpr int LAT16 = DC / 8;           // 16-byte latent (and gate) pieces per token
  static constexpr int ROPE16 = DR / 8;          // 16-byte RoPE pieces per token
  static constexpr int LPASS = 16 * LAT16 / NT;  // latent pieces per thread per tile
  static constexpr int LDS_TOK = kMaxSplitTokensDevice * 8;
  static constexpr int LDS_TILE = 2 * 16 * TS * 2;
  static constexpr int LDS_BYTES = LDS_TOK + LDS_TILE;
  static_assert(16 * LAT16 % NT == 0 && 16 * ROPE16 <= NT, "tile load distribution");
  static_assert(DC % 32 == 0 && DR % 32 == 0, "chunking");
};

template <int DC, int DR>
__global__ __launch_bounds__((HsplitCfg<DC, DR>::NT)) void split_heads_kernel(SplitArgs a) {
  using Cfg = HsplitCfg<DC, DR>;
  constexpr int NW = Cfg::NW, NT = Cfg::NT, NC = Cfg::NC, NR = Cfg::NR, NB = Cfg::NB, TS = Cfg::TS;
  constexpr int LPASS = Cfg::LPASS, LAT16 = Cfg::LAT16, ROPE16 = Cfg::ROPE16;
  constexpr int DQ = DC + DR;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Cfg::LDS_BYTES];
  int* tok_slot = reinterpret_cast<int*>(lds);
  int* tok_id = tok_slot + kMaxSplitTokensDevice;
  uint16_t* tiles = reinterpret_cast<uint16_t*>(lds + Cfg::LDS_TOK);  // [2][16][TS]

  const int item = xcd_logical_block(blockIdx.x, gridDim.x);
  const int hb = item % a.groups;  // block of 128 heads
  const int s = (item / a.groups) % a.s_max;
  const int b = item / (a.groups * a.s_max);
  const int t0 = s * a.split;
  const int L = clamp_len(a.seq_lens[b], a.cap);
  if (t0 >= L) return;  // empty split (uniform over the work-group)
  const int n = min(t0 + a.split, L) - t0;
  const int ntiles = (n + 15) / 16;

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int head0 = hb * (NW * 16) + w * 16;  // this wave's first head

  // ---- slots and ids of the split into LDS; this wave's query chunks ----
  for (int j = tid; j < n; j += NT) {
    const int sl = static_cast<int>(cache_slot(a.page_table, b, t0 + j, a.P, a.max_pages, a.num_slots));
    tok_slot[j] = sl;
    tok_id[j] = clamp_id(a.ids[sl], a.V);
  }
  bf16x8_t qb[NC + NR];  // B operand: head r16, dims 32 c + 8 g .. + 7 (latent chunks, then RoPE)
  {
    const float* qrow = a.qfull + (static_cast<int64_t>(b) * a.H + head0 + r16) * DQ + g * 8;
#pragma unroll
    for (int c = 0; c < NC + NR; ++c) {
      const float4 x0 = *reinterpret_cast<const float4*>(qrow + c * 32);
      const float4 x1 = *reinterpret_cast<const float4*>(qrow + c * 32 + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) qb[c][e] = static_cast<__bf16>(x[e]);  // RoPE part: stored bf16, exact
    }
  }
  __syncthreads();

  // ---- tile loads: thread tid takes latent/gate piece tid + NT p of the tile
  // (token piece / LAT16, 16-byte column piece % LAT16) and, for tid < 16 *
  // ROPE16, RoPE piece tid.  Tokens past the split repeat its last token. ----
  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate);
  u32x4_t lat[LPASS], gat[LPASS], rop;
  auto issue = [&](int t) {
#pragma unroll
    for (int p = 0; p < LPASS; ++p) {
      const int piece = tid + NT * p;
      const int j = min(t * 16 + piece / LAT16, n - 1);
      const int col = (piece % LAT16) * 8;
      lat[p] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(cache + static_cast<int64_t>(tok_slot[j]) * DQ + col));
      gat[p] = *reinterpret_cast<const u32x4_t*>(gate + static_cast<int64_t>(tok_id[j]) * DC + col);
    }
    {
      const int piece = min(tid, 16 * ROPE16 - 1);
      const int j = min(t * 16 + piece / ROPE16, n - 1);
      rop = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(
          cache + static_cast<int64_t>(tok_slot[j]) * DQ + DC + (piece % ROPE16) * 8));
    }
  };
  // gated tile t (in registers) -> LDS buffer t & 1
  auto stage = [&](int t) {
    uint16_t* tile = tiles + (t & 1) * 16 * TS;
#pragma unroll
    for (int p = 0; p < LPASS; ++p) {
      const int piece = tid + NT * p;
      *reinterpret_cast<u32x4_t*>(tile + (piece / LAT16) * TS + (piece % LAT16) * 8) = gate_chunk(lat[p], gat[p]);
    }
    if (tid < 16 * ROPE16) *reinterpret_cast<u32x4_t*>(tile + (tid / ROPE16) * TS + DC + (tid % ROPE16) * 8) = rop;
  };

  f32x4_t o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // reference maximum of head r16 (log2 domain), identical across g
  float l_run = 0.f;        // this lane's share of the sum relative to m_run

  issue(0);
  for (int t = 0; t < ntiles; ++t) {
    stage(t);          // waits for tile t's loads
    issue(t + 1);      // registers free again: next tile (past the end: repeats, unused)
    __syncthreads();   // tile t visible; every wave is past tile t - 1
    const uint16_t* tile = tiles + (t & 1) * 16 * TS;
    const int nt = n - t * 16;  // valid tokens of the tile (1..16)

    // S^T[token 4g + q][head r16]
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC + NR; ++c) {
      const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(tile + r16 * TS + c * 32 + g * 8);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qb[c], acc, 0, 0, 0);
    }
    // online softmax over the tile's 16 tokens
    float x[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = acc[q] * a.scale_log2;
    if (nt < 16) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (4 * g + q >= nt) x[q] = -INFINITY;
    }
    const float mt = max_over_row_groups(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
    const float m_new = fmaxf(m_run, mt);  // finite: the tile has a valid token
    const bool grow = m_new > m_run + kLazyRescale;
    if (__builtin_amdgcn_ballot_w64(grow)) {
      const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
      m_run = grow ? m_new : m_run;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NB; ++db) o[db] *= alpha;
    }
    float p[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      p[q] = __builtin_amdgcn_exp2f(x[q] - m_run);
      l_run += p[q];
    }
    const s16x4_t pb = __builtin_bit_cast(s16x4_t, u32x2_t{pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])});
    // O^T[dim][head] += C~^T[dim][token] x P^T[token][head]: lane r16 of group
    // g reads dims 16 db + 4 (r16 % 4) .. + 3 of token 4g + r16 / 4; the
    // transposed read hands it dim 16 db + r16 of tokens 4g .. 4g + 3.
    uint16_t* tread = const_cast<uint16_t*>(tile) + (4 * g + (r16 >> 2)) * TS + 4 * (r16 & 3);
#pragma unroll
    for (int db = 0; db < NB; ++db) {
      const s16x4_t at =
          __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(tread + db * 16));
      o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(at, pb, o[db], 0, 0, 0);
    }
  }

  // ---- this wave's heads of the split's partial result ----
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t pbase = (static_cast<int64_t>(b) * a.s_max + s) * a.H + head0;
  // lane holds O^T[dim = 16 db + 4g + q][head r16]
#pragma unroll
  for (int db = 0; db < NB; ++db)
    __builtin_nontemporal_store(o[db], reinterpret_cast<f32x4_t*>(a.part_o + (pbase + r16) * DC + db * 16 + 4 * g));
  if (g == 0) {
    __builtin_nontemporal_store(m_run, a.part_ml + (pbase + r16) * 2 + 0);
    __builtin_nontemporal_store(l_run, a.part_ml + (pbase + r16) * 2 + 1);
  }
}

}  // namespace egmla
