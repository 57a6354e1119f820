// MFMA absorption and combine kernels of EG-MLA decode (bf16 storage).
// Included by decode.hip.  Both are short, latency-bound kernels, so each
// issues all of its global loads in one batch before using any of them.
#pragma once

namespace egmla {

// ---------------------------------------------------------------------------
// Absorption on MFMA: qfull[b, h, c] = sum_k q^C[b, h, k] W_UK[h, k, c] for
// BLOCKS (1..4) blocks of 16 sequences x COLS (32 or 128) latent columns per
// work-group (grid H x ceil(B / (16 blocks)) x ceil(DC/COLS), 256 threads),
// plus the q^R copy.  More blocks per work-group read W_UK fewer times; fewer
// blocks and narrower column slices spread a small batch over more compute
// units.
// W_UK[h][:, c-block] is read once per work-group with 16-byte row loads and
// stored row-major in LDS; the B operand (8 consecutive k of one column) is
// two ds_read_b64_tr_b16, whose 16-lane transpose hands lane n the column n
// of 4 consecutive rows, and serves every sequence block.  The A operands (8
// consecutive k of one query row) come straight from global.  Every load is
// issued before the first use.  bf16 x bf16 products are exact in fp32 and
// accumulate in fp32.
// ---------------------------------------------------------------------------
constexpr int kAbsRows = 16;    // sequences per MFMA row block
constexpr int kAbsBlocks = 4;   // row blocks per work-group, at most
constexpr int kAbsCols = 128;     // latent columns per work-group, at most
constexpr int kAbsColsNarrow = 32;
// Below this many work-groups the absorption takes the narrow column slices.
constexpr int kAbsMinWorkGroups = 128;

// HALF: instead of fp32 rows [B, H, DC + DR], write 16-bit rows [B, H, DC + DR]
// = [q_lat in fp16 (one rounding) | q^R in bf16 (copied)], the operands of the
// wide kernel's fp16 latent product and exact bf16 RoPE product; the grid then
// has one more column of work-groups (blockIdx.x == H), the first of which
// computes the wide kernel's balanced schedule from the lengths (sa).
template <int DH, int BLOCKS, int COLS, bool HALF = false>
__global__ __launch_bounds__(256) void absorb_mfma_kernel(const uint16_t* __restrict__ q,
                                                          const uint16_t* __restrict__ w_uk,
                                                          float* __restrict__ qfull, int B, int H, int DC, int DR,
                                                          WideSchedArgs sa) {
  static_assert(BLOCKS >= 1 && BLOCKS <= kAbsBlocks, "row blocks per work-group");
  if constexpr (HALF) {
    // the extra column of work-groups: the head-split kernel's schedule
    if (blockIdx.x == H) {
      if (blockIdx.y == 0 && blockIdx.z == 0) wide_schedule<256>(sa, B);
      return;
    }
  }
  static_assert(COLS % 16 == 0 && COLS <= 128, "latent columns per work-group");
  constexpr int RS = COLS + 8;  // padded LDS row (bf16 elements)
  constexpr int NK = DH / 32;
  __shared__ __attribute__((aligned(16))) uint16_t wrm[DH * RS];  // [k][c], row-major
  constexpr int ROWS = kAbsRows * BLOCKS;  // sequences of this work-group
  const int h = blockIdx.x;
  const int b0 = blockIdx.y * ROWS;
  const int c0 = blockIdx.z * COLS;
  const int nc = min(COLS, DC - c0);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int DQin = DH + DR, DQ = DC + DR;

  // (1) issue every load: this thread's W rows (16 B = 8 columns each), its A
  // operand chunks for every row block, and its RoPE query values
  constexpr int kRowsPerPass = 256 / (COLS / 8);  // e.g. 16 rows of 128 columns per pass
  constexpr int kPasses = (DH + kRowsPerPass - 1) / kRowsPerPass;
  const int cc = (tid % (COLS / 8)) * 8;  // first of this thread's 8 columns
  u32x4_t wv[kPasses];
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const int k = p * kRowsPerPass + tid / (COLS / 8);
    const int kk = min(k, DH - 1);
    const int c = min(c0 + cc, DC - 8);
    wv[p] = *reinterpret_cast<const u32x4_t*>(w_uk + (static_cast<int64_t>(h) * DH + kk) * DC + c);
  }
  u32x4_t qa[BLOCKS][NK];
#pragma unroll
  for (int rb = 0; rb < BLOCKS; ++rb) {
    const int bq = min(b0 + rb * kAbsRows + r16, B - 1);
#pragma unroll
    for (int ks = 0; ks < NK; ++ks)
      qa[rb][ks] = *reinterpret_cast<const u32x4_t*>(q + (static_cast<int64_t>(bq) * H + h) * DQin + ks * 32 + g * 8);
  }
  // RoPE part of the query rows (copied as fp32): when d_r is a multiple of 4
  // and at most 64, thread t loads 4 consecutive values of row t / (d_r / 4)
  // of each row block (8-byte loads, rows clamped so the loads are
  // unconditional); other shapes copy element by element after the product.
  const bool rope_vec = blockIdx.z == 0 && DR > 0 && DR % 4 == 0 && DR <= 64;
  const int rq_row = rope_vec ? tid / (DR / 4) : 0;  // row within a block
  const int rq_col = rope_vec ? 4 * (tid % (DR / 4)) : 0;
  uint2 rq[BLOCKS];
#pragma unroll
  for (int rb = 0; rb < BLOCKS; ++rb) {
    const int rb_b = min(b0 + rb * kAbsRows + min(rq_row, kAbsRows - 1), B - 1);
    rq[rb] = rope_vec ? *reinterpret_cast<const uint2*>(q + (static_cast<int64_t>(rb_b) * H + h) * DQin + DH + rq_col)
                      : make_uint2(0u, 0u);
  }
  // (2) W rows into LDS as loaded (columns past DC hold unused values)
#pragma unroll
  for (int p = 0; p < kPasses; ++p) {
    const int k = p * kRowsPerPass + tid / (COLS / 8);
    if (k < DH) *reinterpret_cast<u32x4_t*>(wrm + k * RS + cc) = wv[p];
  }
  __syncthreads();
  // (3) wave w computes column tiles w, w+4 (16 columns each) of every row
  // block.  For rows k0 .. k0 + 3 of the tile, lane r16 of group g reads
  // columns 4 (r16 % 4) .. + 3 of row k0 + r16 / 4; the transposed read hands
  // lane r16 column r16 of the 4 rows.
  for (int nt = w; nt * 16 < nc; nt += 4) {
    f32x4_t acc[BLOCKS];
#pragma unroll
    for (int rb = 0; rb < BLOCKS; ++rb) acc[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < NK; ++ks) {
      uint16_t* t0 = wrm + (ks * 32 + 8 * g + (r16 >> 2)) * RS + nt * 16 + 4 * (r16 & 3);
      const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)t0);
      const s16x4_t hi =
          __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(t0 + 4 * RS));
      const u32x2_t l2 = __builtin_bit_cast(u32x2_t, lo), h2 = __builtin_bit_cast(u32x2_t, hi);
      const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, u32x4_t{l2[0], l2[1], h2[0], h2[1]});
#pragma unroll
      for (int rb = 0; rb < BLOCKS; ++rb)
        acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, qa[rb][ks]), bv, acc[rb], 0, 0, 0);
    }
    // lane holds D[b = 4g + r][c = nt*16 + r16] of each row block
    const int c = c0 + nt * 16 + r16;
#pragma unroll
    for (int rb = 0; rb < BLOCKS; ++rb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int b = b0 + rb * kAbsRows + 4 * g + r;
        if (b < B && c < DC) {
          if constexpr (HALF) {
            reinterpret_cast<_Float16*>(qfull)[(static_cast<int64_t>(b) * H + h) * DQ + c] =
                static_cast<_Float16>(acc[rb][r]);
          } else {
            qfull[(static_cast<int64_t>(b) * H + h) * DQ + c] = acc[rb][r];
          }
        }
      }
    }
  }
  if (rope_vec) {
#pragma unroll
    for (int rb = 0; rb < BLOCKS; ++rb) {
      const int b = b0 + rb * kAbsRows + rq_row;
      if (rq_row < kAbsRows && b < B) {
        if constexpr (HALF)
          *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(qfull) + (static_cast<int64_t>(b) * H + h) * DQ + DC +
                                    rq_col) = rq[rb];
        else
          *reinterpret_cast<float4*>(qfull + (static_cast<int64_t>(b) * H + h) * DQ + DC + rq_col) =
              make_float4(bf16_lo(rq[rb].x), bf16_hi(rq[rb].x), bf16_lo(rq[rb].y), bf16_hi(rq[rb].y));
      }
    }
  } else if (blockIdx.z == 0) {
    for (int i = tid; i < ROWS * DR; i += 256) {
      const int bb = i / DR, r = i % DR;
      if (b0 + bb < B) {
        const uint16_t v = q[(static_cast<int64_t>(b0 + bb) * H + h) * DQin + DH + r];
        if constexpr (HALF)
          reinterpret_cast<uint16_t*>(qfull)[(static_cast<int64_t>(b0 + bb) * H + h) * DQ + DC + r] = v;
        else
          qfull[(static_cast<int64_t>(b0 + bb) * H + h) * DQ + DC + r] = bf16_to_f32(v);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Combine on MFMA: grid (H, ceil(B / spw)), 1024 threads (16 waves), one head
// and up to spw <= 16 sequences per work-group (fewer for small batches, so
// that the grid still spreads over the chip).
//  1. Waves 0 .. nvt-1 issue the W_UV rows of their 16-row output tile (first
//     for d_c <= 128; after step 3 for wider latents, to stay in registers).
//  2. The partials of each sequence (`slices` per context split; a partial
//     of an id slice without tokens has maximum -inf and is skipped) are
//     merged online in fp32: with n sequences in the group, each gets
//     wps = 16 / pow2ceil(n) waves, and wave p of a sequence merges its
//     partials p, p + wps, ... in batches of 4, 8 or 16 (at most 8 for
//     d_c > 128) (maxima, sums and partial outputs loaded together) into LDS.
//  3. All threads merge each sequence's wps parts into its latent row o / l,
//     split once into bf16 hi + lo in LDS.
//  4. out^T[v][b] = W_UV[h][v][:] . o[b][:] on v_mfma_f32_16x16x32_bf16, the
//     16 sequences being the 16 columns of the B operand, a product each for
//     hi and lo, so the up-projection adds only W_UV's own rounding.
// ---------------------------------------------------------------------------
constexpr int kCombSeq = 16;
constexpr int kCombWaves = 16;
// merged rows as bf16 hi + lo ([2][kCombSeq][DC + 8]), then the waves' partial merges and their (m, l)
constexpr size_t combine_lds_bytes(int DC) {
  return 2 * sizeof(uint16_t) * kCombSeq * (DC + 8) + sizeof(float) * (kCombWaves * DC + 2 * kCombWaves);
}

// Latent dim held in accumulator j of a combine lane: with an even number of
// dims per lane, lane l holds the adjacent pairs 128 i + 2 l + {0, 1} (8-byte
// loads); otherwise dims l + 64 j.
template <int DC>
__device__ __forceinline__ int comb_dim(int lane, int j) {
  constexpr int PER = DC / 64;
  if constexpr (PER % 2 == 0) return 128 * (j >> 1) + 2 * lane + (j & 1);
  else return lane + 64 * j;
}

// One batch of SB splits of the online merge: the splits first + stride * t
// for t = s0 .. s0 + SB - 1 (t clamped to ns - 1, counted while t < ns).
// Their maxima, sums and partial outputs load together.
template <int DC, int SB>
__device__ __forceinline__ void merge_batch(const float* __restrict__ part_ml, const float* __restrict__ part_o,
                                            int64_t base, int H, int first, int stride, int s0, int ns, int lane,
                                            float& M, float& Ls, float (&acc)[DC / 64]) {
  constexpr int PER = DC / 64;
  float pv[SB][PER];
  float2 ml[SB];
#pragma unroll
  for (int u = 0; u < SB; ++u) {
    const int64_t row = base + static_cast<int64_t>(first + stride * min(s0 + u, ns - 1)) * H;
    ml[u] = *reinterpret_cast<const float2*>(part_ml + row * 2);
    if constexpr (PER % 2 == 0) {
#pragma unroll
      for (int i = 0; i < PER / 2; ++i) {
        const float2 v = *reinterpret_cast<const float2*>(part_o + row * DC + 128 * i + 2 * lane);
        pv[u][2 * i] = v.x;
        pv[u][2 * i + 1] = v.y;
      }
    } else {
#pragma unroll
      for (int j = 0; j < PER; ++j) pv[u][j] = part_o[row * DC + lane + 64 * j];
    }
  }
  float mb = -INFINITY;
#pragma unroll
  for (int u = 0; u < SB; ++u) mb = fmaxf(mb, ml[u].x);  // repeated last split: no effect on the max
  const float Mn = fmaxf(M, mb);
  // a partial without tokens has maximum -inf; while every partial so far is
  // one, nothing is accumulated (and exp2(-inf - -inf) is never formed)
  const bool live = Mn > -INFINITY;
  const float sc = live ? __builtin_amdgcn_exp2f(M - Mn) : 1.f;  // 0 for the first live batch (exp2(-inf))
  Ls *= sc;
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] *= sc;
#pragma unroll
  for (int u = 0; u < SB; ++u) {
    const float e = s0 + u < ns && live ? __builtin_amdgcn_exp2f(ml[u].x - Mn) : 0.f;
    Ls += ml[u].y * e;
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] = fmaf(e, pv[u][j], acc[j]);
  }
  M = Mn;
}

template <int DC, int DV>
__global__ __launch_bounds__(kCombWaves * 64) void combine_mfma_kernel(const float* __restrict__ part_ml,
                                                                       const float* __restrict__ part_o,
                                                                       const uint16_t* __restrict__ w_uv,
                                                                       const int32_t* __restrict__ seq_lens,
                                                                       uint16_t* __restrict__ out, int B, int H,
                                                                       int cap, int split, int s_max, int slices,
                                                                       const int2* __restrict__ seq_rows, int spw) {
  constexpr int OS = DC + 8;     // bf16 elements per merged row in LDS
  constexpr int PER = DC / 64;  // latent columns per lane
  constexpr int NKC = DC / 32;
  constexpr int nvt = (DV + 15) / 16;
  static_assert(nvt <= kCombWaves, "one output tile per wave");
  extern __shared__ __attribute__((aligned(16))) float comb_lds[];  // combine_lds_bytes(DC) bytes
  uint16_t* o_s = reinterpret_cast<uint16_t*>(comb_lds);           // [2][kCombSeq][OS]: merged rows, hi then lo
  float* o_part = comb_lds + kCombSeq * OS;                         // [kCombWaves][DC]: each wave's partial merge
  float* m_part = o_part + kCombWaves * DC;                         // [kCombWaves]
  float* l_part = m_part + kCombWaves;                              // [kCombWaves]
  const int h = blockIdx.x;
  const int b0 = blockIdx.y * spw;  // spw <= kCombSeq sequences per work-group
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nseq = min(spw, B - b0);
  int np2 = 1;
  while (np2 < nseq) np2 <<= 1;
  const int wps = kCombWaves / np2;  // waves per sequence (power of two)

  // (1) W_UV rows of this wave's output tile, issued first for narrow
  // latents; for wide ones (NKC x 16 bytes per lane) after the merge, which
  // then has the registers to itself.
  constexpr bool kEarlyW = DC <= 128;
  constexpr int kSBMax = DC <= 128 ? 16 : 8;  // splits per merge batch, at most
  u32x4_t wa[NKC];
  const int vt = w;
  auto load_w = [&]() {
    if (vt < nvt) {
      const int v = min(vt * 16 + r16, DV - 1);
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc)
        wa[kc] = *reinterpret_cast<const u32x4_t*>(w_uv + (static_cast<int64_t>(h) * DV + v) * DC + kc * 32 + g * 8);
    }
  };
  if constexpr (kEarlyW) load_w();

  // (2) this wave's part of its sequence's splits
  const int k = w / wps, part = w % wps;
  const int b = b0 + k;
  const int L = (k < nseq) ? clamp_len(seq_lens[b], cap) : 0;
  // partials of sequence b: `slices` per split (a split below the sequence's
  // length holds a token, though one of its id slices may hold none), or the
  // rows seq_rows[b] lists (balanced schedule)
  const int ns_all = L <= 0 ? 0 : seq_rows ? seq_rows[b].y : min((L + split - 1) / split, s_max) * slices;
  const int ns = ns_all > part ? (ns_all - part + wps - 1) / wps : 0;  // this part's partials
  float M = -INFINITY, Ls = 0.f;
  float acc[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) acc[j] = 0.f;
  if (ns > 0) {
    const int64_t row0 = seq_rows ? seq_rows[b].x : static_cast<int64_t>(b) * s_max * slices;
    const int64_t base = row0 * H + h;  // + partial * H
    if (ns <= 4) {
      merge_batch<DC, 4>(part_ml, part_o, base, H, part, wps, 0, ns, lane, M, Ls, acc);
    } else if (ns <= 8) {
      merge_batch<DC, 8>(part_ml, part_o, base, H, part, wps, 0, ns, lane, M, Ls, acc);
    } else {
      for (int s0 = 0; s0 < ns; s0 += kSBMax)
        merge_batch<DC, kSBMax>(part_ml, part_o, base, H, part, wps, s0, ns, lane, M, Ls, acc);
    }
  }
#pragma unroll
  for (int j = 0; j < PER; ++j) o_part[w * DC + comb_dim<DC>(lane, j)] = acc[j];
  if (lane == 0) {
    m_part[w] = M;
    l_part[w] = Ls;
  }
  __syncthreads();

  // (3) merge the parts of each sequence into its row o / l (rows past the
  // group's sequences, and empty sequences, are zero)
  for (int i = tid; i < kCombSeq * DC; i += kCombWaves * 64) {
    const int kk = i / DC, c = i - kk * DC;
    float v = 0.f;
    if (kk < nseq) {
      float Mx = -INFINITY;
      for (int p = 0; p < wps; ++p) Mx = fmaxf(Mx, m_part[kk * wps + p]);
      if (Mx > -INFINITY) {
        float num = 0.f, den = 0.f;
        for (int p = 0; p < wps; ++p) {
          const float e = __builtin_amdgcn_exp2f(m_part[kk * wps + p] - Mx);  // empty part: exp2(-inf) = 0
          num = fmaf(e, o_part[(kk * wps + p) * DC + c], num);
          den = fmaf(e, l_part[kk * wps + p], den);
        }
        v = num / den;
      }
    }
    const __bf16 hi = static_cast<__bf16>(v);
    o_s[kk * OS + c] = __builtin_bit_cast(uint16_t, hi);
    o_s[(kCombSeq + kk) * OS + c] = __builtin_bit_cast(uint16_t, static_cast<__bf16>(v - static_cast<float>(hi)));
  }
  __syncthreads();

  // (4) out^T[vt*16 + 4g + r][b0 + r16] for this wave's tile
  if constexpr (!kEarlyW) load_w();
  if (vt < nvt) {
    f32x4_t o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const int row = r16 * OS + kc * 32 + g * 8;
      const bf16x8_t hi = *reinterpret_cast<const bf16x8_t*>(o_s + row);
      const bf16x8_t lo = *reinterpret_cast<const bf16x8_t*>(o_s + kCombSeq * OS + row);
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, wa[kc]);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, hi, o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, lo, o, 0, 0, 0);
    }
    const int bb = b0 + r16;
    if (r16 < nseq) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = vt * 16 + 4 * g + r;
        if (vv < DV) out[(static_cast<int64_t>(bb) * H + h) * DV + vv] = f32_to_bf16(o[r]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Merge of the head-split kernel's partial rows (d_c 512, d_v 128): grid
// (H, ceil(B / 32)), 512 threads (8 waves), one head and up to 32 sequences
// per work-group.  Each partial row is O / l in fp16 with (m, l) in fp32, and
// seq_rows[b] = (first row, number of rows) lists sequence b's rows.
//  1. Wave w loads the row lists of sequences w + 8 k (k = 0 .. 3) of the
//     group, then the first 4 rows of each (lane l: latent dims 8 l .. 8 l + 7,
//     one 16-byte load per row), then the W_UV rows of output tile w (rows
//     16 w .. 16 w + 15, all 512 latent columns).  Loads complete in issue
//     order, so the merge waits for the rows only while W_UV is on its way.
//  2. Each sequence's rows are merged online in fp32 with weights e l,
//     e = exp2(m - M) (loads past a sequence's rows re-read its last row and
//     enter with weight 0; rows past the fourth are loaded as the merge
//     reaches them).  The merged row o / l goes to LDS split once into bf16
//     hi + lo (zero for an empty sequence), the B operands of every tile.
//  3. out^T[v][b] = W_UV[h][v][:] . o[b][:] for tile w and both blocks of 16
//     sequences on v_mfma_f32_16x16x32_bf16, a product each for hi and lo, so
//     the up-projection adds only W_UV's own rounding.
// ---------------------------------------------------------------------------
constexpr int kCombWideSeq = 32;
constexpr int kCombWideWaves = 8;
constexpr int kCombWideOS = 512 + 8;  // LDS row of a merged sequence (bf16 elements; 16-byte rotation per row)
constexpr size_t combine_wide_lds_bytes() { return 2 * sizeof(uint16_t) * kCombWideSeq * kCombWideOS; }

__global__ __launch_bounds__(kCombWideWaves * 64) void combine_wide_kernel(const float* __restrict__ part_ml,
                                                                          const uint16_t* __restrict__ part_o,
                                                                          const uint16_t* __restrict__ w_uv,
                                                                          const int2* __restrict__ seq_rows,
                                                                          uint16_t* __restrict__ out, int B, int H) {
  constexpr int DC = 512, DV = 128, NKC = DC / 32, OS = kCombWideOS;
  constexpr int SPW = kCombWideSeq / kCombWideWaves;  // sequences per wave
  static_assert(DV / 16 == kCombWideWaves && SPW % 2 == 0, "one output tile per wave; sequences in pairs");
  // merged rows o / l as bf16 hi + lo: [2][kCombWideSeq][OS]
  extern __shared__ __attribute__((aligned(16))) uint16_t cw_lds[];
  const int h = blockIdx.x;
  const int b0 = blockIdx.y * kCombWideSeq;
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  // (1) the row lists of this wave's sequences, then the first 4 rows of
  // each (lane l: latent dims 8 l .. 8 l + 7), then W_UV rows 16 w + r16
  // (columns 32 kc + 8 g .. + 7): loads complete in issue order, so the merge
  // waits for the rows only and W_UV arrives while it runs
  int2 sr[SPW];
#pragma unroll
  for (int k = 0; k < SPW; ++k) {
    const int b = b0 + w + kCombWideWaves * k;  // uniform over the wave
    sr[k] = b < B ? seq_rows[b] : make_int2(0, 0);
  }
  const int coff = 8 * lane;
  float2 ml[SPW][4];
  u32x4_t pv[SPW][4];
  // rows s0 .. s0 + 3 of sequence k (rows past its list repeat its last row)
  auto load_rows = [&](int k, int s0, float2 (&m4)[4], u32x4_t (&p4)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t row = static_cast<int64_t>(sr[k].x + min(s0 + u, sr[k].y - 1)) * H + h;
      m4[u] = *reinterpret_cast<const float2*>(part_ml + row * 2);
      p4[u] = *reinterpret_cast<const u32x4_t*>(part_o + row * DC + coff);
    }
  };
#pragma unroll
  for (int k = 0; k < SPW; ++k)
    if (sr[k].y > 0) load_rows(k, 0, ml[k], pv[k]);
  u32x4_t wa[NKC];
  {
    const uint16_t* wrow = w_uv + (static_cast<int64_t>(h) * DV + 16 * w + r16) * DC + 8 * g;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) wa[kc] = *reinterpret_cast<const u32x4_t*>(wrow + 32 * kc);
  }

  // (2) online merge of each sequence's rows in fp32, weights e l with
  // e = exp2(m - M) (rows past the list: weight 0), into LDS as o / l
  auto fold = [&](int n, int s0, const float2 (&m4)[4], const u32x4_t (&p4)[4], float& M, float& Ls,
                  float (&acc)[8]) {
    float mb = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u) mb = fmaxf(mb, s0 + u < n ? m4[u].x : -INFINITY);
    const float Mn = fmaxf(M, mb);
    // nothing is accumulated while every row so far has maximum -inf
    const bool live = Mn > -INFINITY;
    const float sc = live ? __builtin_amdgcn_exp2f(M - Mn) : 1.f;  // 0 for the first live batch
    Ls *= sc;
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] *= sc;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float e = s0 + u < n && live ? __builtin_amdgcn_exp2f(m4[u].x - Mn) : 0.f;
      Ls = fmaf(m4[u].y, e, Ls);
      const float wgt = e * m4[u].y;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t v = p4[u][j];
        acc[2 * j] = fmaf(wgt, static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(v & 0xffffu))),
                          acc[2 * j]);
        acc[2 * j + 1] =
            fmaf(wgt, static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(v >> 16))), acc[2 * j + 1]);
      }
    }
    M = Mn;
  };
#pragma unroll
  for (int k = 0; k < SPW; ++k) {
    const int n = sr[k].y;
    float M = -INFINITY, Ls = 0.f;
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    if (n > 0) {
      fold(n, 0, ml[k], pv[k], M, Ls, acc);
      for (int s0 = 4; s0 < n; s0 += 4) {  // sequences over more than 4 token ranges
        float2 m4[4];
        u32x4_t p4[4];
        load_rows(k, s0, m4, p4);
        fold(n, s0, m4, p4, M, Ls, acc);
      }
    }
    const float inv = Ls > 0.f ? 1.f / Ls : 0.f;  // a sequence with tokens has Ls >= 1
    bf16x8_t hi, lo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x = acc[e] * inv;
      hi[e] = static_cast<__bf16>(x);
      lo[e] = static_cast<__bf16>(x - static_cast<float>(hi[e]));
    }
    const int row = (w + kCombWideWaves * k) * OS + coff;
    *reinterpret_cast<bf16x8_t*>(cw_lds + row) = hi;
    *reinterpret_cast<bf16x8_t*>(cw_lds + kCombWideSeq * OS + row) = lo;
  }
  __syncthreads();

  // (3) out^T[16 w + 4 g + r][b0 + 16 bb + r16]
#pragma unroll
  for (int bb = 0; bb < kCombWideSeq / 16; ++bb) {
    f32x4_t o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      const int row = (16 * bb + r16) * OS + 32 * kc + 8 * g;
      const bf16x8_t hi = *reinterpret_cast<const bf16x8_t*>(cw_lds + row);
      const bf16x8_t lo = *reinterpret_cast<const bf16x8_t*>(cw_lds + kCombWideSeq * OS + row);
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, wa[kc]);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, hi, o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, lo, o, 0, 0, 0);
    }
    const int b = b0 + 16 * bb + r16;
    if (b < B) {
      uint16_t* orow = out + (static_cast<int64_t>(b) * H + h) * DV + 16 * w + 4 * g;
#pragma unroll
      for (int r = 0; r < 4; ++r) orow[r] = f32_to_bf16(o[r]);
    }
  }
}

// ---------------------------------------------------------------------------
// Merge on MFMA with small work-groups: grid (H, ceil(B / 4)), 256 threads,
// one head and up to 4 sequences per work-group.  For batches whose partials
// fit one merge batch per sequence, many small work-groups finish sooner than
// 16-wave ones.  Wave w merges sequence b0 + w (every partial of it: `slices`
// per context split) online in fp32 and writes its row o / l to LDS; then
// out^T[v][b] = W_UV[h][v][:] . o[b][:] on v_mfma_f32_16x16x32_bf16, wave w
// taking output tiles w, w + 4, ... of 16 rows, the merged rows as the B
// operand's first 4 columns (split once into bf16 hi + lo as they go to LDS,
// a product each).  The W_UV rows are loaded first;
// `wait(b)` is called by each wave before it loads the partials of its
// sequence (nothing to wait for in a kernel of its own).
// ---------------------------------------------------------------------------
constexpr int kComb4Seq = 4;

template <int DC, int DV, typename Wait>
__device__ __forceinline__ void combine4_block(const float* __restrict__ part_ml, const float* __restrict__ part_o,
                                               const uint16_t* __restrict__ w_uv,
                                               const int32_t* __restrict__ seq_lens, uint16_t* __restrict__ out,
                                               int B, int H, int cap, int split, int s_max, int slices, int h,
                                               int b0, uint16_t* o_s, Wait wait) {
  constexpr int OS = DC + 8;  // bf16 elements: o / l hi in rows 0 .. 3, lo in rows 4 .. 7
  constexpr int PER = DC / 64;
  constexpr int NKC = DC / 32;
  constexpr int nvt = (DV + 15) / 16;
  constexpr int TPW = (nvt + 3) / 4;  // output tiles per wave
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nseq = min(kComb4Seq, B - b0);

  // (1) this wave's W_UV rows
  u32x4_t wa[TPW][NKC];
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int vt = w + 4 * t;
    const int v = min(vt * 16 + r16, DV - 1);
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      wa[t][kc] = *reinterpret_cast<const u32x4_t*>(w_uv + (static_cast<int64_t>(h) * DV + v) * DC + kc * 32 + g * 8);
  }
  // (2) wave w merges sequence b0 + w
  {
    const int b = b0 + w;
    const int L = w < nseq ? clamp_len(seq_lens[b], cap) : 0;
    const int ns = L > 0 ? min((L + split - 1) / split, s_max) * slices : 0;
    float M = -INFINITY, Ls = 0.f;
    float acc[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) acc[j] = 0.f;
    if (w < nseq) wait(b);
    if (ns > 0) {
      const int64_t base = static_cast<int64_t>(b) * s_max * slices * H + h;
      if (ns <= 8) {
        merge_batch<DC, 8>(part_ml, part_o, base, H, 0, 1, 0, ns, lane, M, Ls, acc);
      } else {
        for (int s0 = 0; s0 < ns; s0 += 16)
          merge_batch<DC, 16>(part_ml, part_o, base, H, 0, 1, s0, ns, lane, M, Ls, acc);
      }
    }
    const float inv = Ls > 0.f ? 1.f / Ls : 0.f;  // a sequence with tokens has Ls >= 1
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const float x = acc[j] * inv;
      const __bf16 hi = static_cast<__bf16>(x);
      o_s[w * OS + comb_dim<DC>(lane, j)] = __builtin_bit_cast(uint16_t, hi);
      o_s[(kComb4Seq + w) * OS + comb_dim<DC>(lane, j)] =
          __builtin_bit_cast(uint16_t, static_cast<__bf16>(x - static_cast<float>(hi)));
    }
  }
  __syncthreads();
  // (3) out^T[vt*16 + 4g + r][b0 + r16] for this wave's tiles
#pragma unroll
  for (int t = 0; t < TPW; ++t) {
    const int vt = w + 4 * t;
    if (vt >= nvt) continue;
    f32x4_t o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      u32x4_t hv = {0u, 0u, 0u, 0u}, lv = {0u, 0u, 0u, 0u};
      if (r16 < kComb4Seq) {
        hv = *reinterpret_cast<const u32x4_t*>(o_s + r16 * OS + kc * 32 + g * 8);
        lv = *reinterpret_cast<const u32x4_t*>(o_s + (kComb4Seq + r16) * OS + kc * 32 + g * 8);
      }
      const bf16x8_t hi = __builtin_bit_cast(bf16x8_t, hv), lo = __builtin_bit_cast(bf16x8_t, lv);
      const bf16x8_t av = __builtin_bit_cast(bf16x8_t, wa[t][kc]);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, hi, o, 0, 0, 0);
      o = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, lo, o, 0, 0, 0);
    }
    if (r16 < nseq) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int vv = vt * 16 + 4 * g + r;
        if (vv < DV) out[(static_cast<int64_t>(b0 + r16) * H + h) * DV + vv] = f32_to_bf16(o[r]);
      }
    }
  }
}
template <int DC, int DV>
__global__ __launch_bounds__(256) void combine4_kernel(const float* __restrict__ part_ml, const float* __restrict__ part_o,
                                                       const uint16_t* __restrict__ w_uv, const int32_t* __restrict__ seq_lens,
                                                       uint16_t* __restrict__ out, int B, int H, int cap, int split,
                                                       int s_max, int slices) {
  __shared__ __attribute__((aligned(16))) uint16_t o_s[2 * kComb4Seq * (DC + 8)];
  combine4_block<DC, DV>(part_ml, part_o, w_uv, seq_lens, out, B, H, cap, split, s_max, slices, blockIdx.x,
                         blockIdx.y * kComb4Seq, o_s, [](int) {});
}

}  // namespace egmla
