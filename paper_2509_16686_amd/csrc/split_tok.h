// Token-split MFMA split kernel of EG-MLA decode (bf16 storage, 16 heads per
// work-group, latent dim <= 128).  Included by decode.hip after SplitArgs.
//
// One work-group of NWT waves per (sequence, split, head group of 16).  The
// split's tokens form 16-token units; unit u belongs to wave u % NWT, so the
// waves of a work-group stream neighbouring rows at the same time.  A wave
// owns whole rows and all 16 heads of its units, so scores, softmax and the
// value product need nothing from other waves; the waves merge their
// (max, sum, output) once, at the end.  For a unit the wave
//   * loads each token's latent, RoPE key and gate rows straight into the
//     layout of the MFMA A operand (lane: token lane%16, 16 bytes = 8
//     consecutive dims of a 32-dim chunk), and gates in fp32 (exact product),
//     rounding the gated latent to bf16 once;
//   * computes S^T[token][head] with v_mfma_f32_16x16x32_bf16; the fp32
//     absorbed query enters as bf16 hi + lo (two products), so a score
//     carries only the rounding of the gated latent, and the RoPE part (bf16
//     query times bf16 key) is exact;
//   * runs the online softmax on the accumulator layout (lane: one head, 4
//     tokens), rescaling its accumulators only when a head's maximum grows by
//     more than 2^8, so the probabilities stay below 2^8 and the rescale is
//     rare; the probabilities are exactly the B operand of the value product;
//   * stores the gated unit row-major in its own LDS tile and reads each
//     16-dim block back with ds_read_b64_tr_b16, whose 16-lane transpose
//     yields exactly the A operand of v_mfma_f32_16x16x16_bf16 (lane: dim
//     lane%16, tokens 4*(lane/16)..+3), and accumulates
//     O^T[dim][head] += C~^T x P^T.
// Every global load of a unit depends only on LDS and is issued D units ahead
// of its use, unconditionally (indexes past the split repeat its last token),
// so the compiler's wait counters track each unit and D units stay in flight.
#pragma once

namespace egmla {

template <int DC, int DR, int NWT>
struct TsplitCfg {
  static constexpr int NC = DC / 32;  // 32-dim latent chunks
  static constexpr int NR = DR / 32;  // 32-dim RoPE chunks
  static constexpr int NB = DC / 16;  // 16-dim blocks of the value product
  static constexpr int TS = DC + 8;   // bf16 elements per row of a wave's unit tile (16 bytes of padding)
  static constexpr int LDS_TOK = kMaxSplitTokensDevice * 8;  // slot + id of every token of the split
  static constexpr int LDS_TILE = NWT * 16 * TS * 2;         // each wave's gated unit, row-major
  static constexpr int LDS_MERGE = NWT * NB * 64 * 16;       // every wave's output accumulators (aliases the above)
  static constexpr int LDS_MAIN = LDS_TOK + LDS_TILE > LDS_MERGE ? LDS_TOK + LDS_TILE : LDS_MERGE;
  static constexpr int LDS_STAT = NWT * 16 * 4 * 2;          // every wave's max and sum per head
  static constexpr int LDS_BYTES = LDS_MAIN + LDS_STAT;
  static_assert(DC % 32 == 0 && DR % 32 == 0 && DC <= 128, "token-split shapes");
};

// One unit's operands (16 tokens, this lane's 16 bytes of every chunk).
template <int NC, int NR>
struct UnitRegs {
  u32x4_t lat[NC];
  u32x4_t gat[NC];
  u32x4_t rop[NR > 0 ? NR : 1];
};

// Largest growth (log2 units) of a head's maximum absorbed without rescaling.
constexpr float kLazyRescale = 8.0f;

template <int DC, int DR, int NWT, int D>
__global__ __launch_bounds__(NWT * 64, 2) void split_tok_kernel(SplitArgs a) {
  using Cfg = TsplitCfg<DC, DR, NWT>;
  constexpr int NC = Cfg::NC, NR = Cfg::NR, NB = Cfg::NB;
  constexpr int DQ = DC + DR;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Cfg::LDS_BYTES];
  int* tok_slot = reinterpret_cast<int*>(lds);
  int* tok_id = tok_slot + kMaxSplitTokensDevice;
  uint16_t* tile_all = reinterpret_cast<uint16_t*>(lds + Cfg::LDS_TOK);  // [NWT][16][TS]
  f32x4_t* obuf = reinterpret_cast<f32x4_t*>(lds);                        // [NWT][NB][64], after the units
  float* mbuf = reinterpret_cast<float*>(lds + Cfg::LDS_MAIN);            // [NWT][16]
  float* lbuf = mbuf + NWT * 16;                                          // [NWT][16]

  const int item = xcd_logical_block(blockIdx.x, gridDim.x);
  const int hg = item % a.groups;
  const int s = (item / a.groups) % a.s_max;
  const int b = item / (a.groups * a.s_max);
  const int t0 = s * a.split;
  const int L = clamp_len(a.seq_lens[b], a.cap);
  if (t0 >= L) return;  // empty split (uniform over the work-group)
  const int n = min(t0 + a.split, L) - t0;
  const int nunits = (n + 15) / 16;  // every unit below nunits holds a valid token

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);     // wave-uniform
  const int nu = nunits > w ? (nunits - w + NWT - 1) / NWT : 0;  // this wave's units

  // ---- slots and ids of the split; query chunks; 0/1 selection operands ----
  for (int j = tid; j < n; j += NWT * 64) {
    const int sl = static_cast<int>(cache_slot(a.page_table, b, t0 + j, a.P, a.max_pages, a.num_slots));
    tok_slot[j] = sl;
    tok_id[j] = clamp_id(a.ids[sl], a.V);
  }
  bf16x8_t qh[NC], ql[NC];
  bf16x8_t qr[NR > 0 ? NR : 1];
  {
    const float* qrow = a.qfull + (static_cast<int64_t>(b) * a.H + hg * 16 + r16) * DQ + g * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const float4 x0 = *reinterpret_cast<const float4*>(qrow + c * 32);
      const float4 x1 = *reinterpret_cast<const float4*>(qrow + c * 32 + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        qh[c][e] = static_cast<__bf16>(x[e]);
        ql[c][e] = static_cast<__bf16>(x[e] - static_cast<float>(qh[c][e]));
      }
    }
#pragma unroll
    for (int rc = 0; rc < NR; ++rc) {
      const float4 x0 = *reinterpret_cast<const float4*>(qrow + DC + rc * 32);
      const float4 x1 = *reinterpret_cast<const float4*>(qrow + DC + rc * 32 + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) qr[rc][e] = static_cast<__bf16>(x[e]);  // q^R is a stored bf16 value: exact
    }
  }
  __syncthreads();

  f32x4_t o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // reference maximum of head r16 (log2 domain), identical across g
  float l_run = 0.f;        // this lane's share of the sum relative to m_run

  if (nu > 0) {
    const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache) + g * 8;
    const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate) + g * 8;
    // Loads of this wave's unit i; every address comes from LDS.
    auto issue = [&](UnitRegs<NC, NR>& r, int i) {
      const int j = min((w + i * NWT) * 16 + r16, n - 1);  // past the split: repeat its last token (masked)
      const int sl = tok_slot[j];
      const int id = tok_id[j];
      const uint16_t* row = cache + static_cast<int64_t>(sl) * DQ;
      const uint16_t* grow = gate + static_cast<int64_t>(id) * DC;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        r.lat[c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(row + c * 32));
        r.gat[c] = *reinterpret_cast<const u32x4_t*>(grow + c * 32);
      }
#pragma unroll
      for (int rc = 0; rc < NR; ++rc)
        r.rop[rc] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(row + DC + rc * 32));
    };

    // Loads return in issue order, so unit i is issued before unit i + 1.
    UnitRegs<NC, NR> ring[D];
#pragma unroll
    for (int k = 0; k < D; ++k) {
      issue(ring[k], k);
      __builtin_amdgcn_sched_barrier(0);
    }

    uint16_t* tile = tile_all + w * 16 * Cfg::TS;  // this wave's [16 tokens][TS]
    uint16_t* tread = tile + (4 * g + (r16 >> 2)) * Cfg::TS + 4 * (r16 & 3);
    // Unit i of this wave (operands in r); refill: issue unit i + D into r.
    auto process = [&](UnitRegs<NC, NR>& r, int i, bool refill) {
      const int nt = n - (w + i * NWT) * 16;  // valid tokens of the unit (1..16)

      // gate the latent: exact fp32 products, rounded once to bf16; stage the
      // gated unit in this wave's tile for the transposed reads
      bf16x8_t av[NC];
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const u32x4_t hv = gate_chunk(r.lat[c], r.gat[c]);
        av[c] = __builtin_bit_cast(bf16x8_t, hv);
        *reinterpret_cast<u32x4_t*>(tile + r16 * Cfg::TS + c * 32 + g * 8) = hv;
      }
      // S^T[token 4g + q][head r16]
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[c], qh[c], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[c], ql[c], acc, 0, 0, 0);
      }
#pragma unroll
      for (int rc = 0; rc < NR; ++rc)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r.rop[rc]), qr[rc], acc, 0, 0, 0);
      // this unit's registers are free: issue unit i + D into them
      if (refill) issue(r, i + D);

      // online softmax over the unit's 16 tokens
      float x[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = acc[q] * a.scale_log2;
      if (nt < 16) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (4 * g + q >= nt) x[q] = -INFINITY;
      }
      const float mt = max_over_row_groups(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
      const float m_new = fmaxf(m_run, mt);  // finite: the unit has a valid token
      const bool grow = m_new > m_run + kLazyRescale;  // false while both are -inf
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;  // exp2(-inf) = 0
        m_run = grow ? m_new : m_run;
        l_run *= alpha;
#pragma unroll
        for (int db = 0; db < NB; ++db) o[db] *= alpha;
      }
      float p[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        p[q] = __builtin_amdgcn_exp2f(x[q] - m_run);  // masked: exp2(-inf) = 0
        l_run += p[q];
      }
      const uint32_t pb01 = pack_bf16x2(p[0], p[1]);
      const uint32_t pb23 = pack_bf16x2(p[2], p[3]);
      const s16x4_t pb = __builtin_bit_cast(s16x4_t, u32x2_t{pb01, pb23});

      // O^T[dim][head] += C~^T[dim][token] x P^T[token][head], 16 dims at a
      // time.  Lane r16 of group g reads dims 16 db + 4 (r16 % 4) .. + 3 of
      // token 4g + r16 / 4; the transposed read hands lane r16 of group g the
      // dim 16 db + r16 of tokens 4g .. 4g + 3.
      wave_lds_sync();
#pragma unroll
      for (int db = 0; db < NB; ++db) {
        const s16x4_t at =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(tread + db * 16));
        o[db] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(at, pb, o[db], 0, 0, 0);
      }
    };

    // Full groups of D units (ring slot u holds units u, u + D, ...), then the
    // remaining nu % D units straight-line.  The loop has one exit, and on
    // every path to its exit the same D units are in flight in the same
    // order, so the compiler's wait counters stay exact; an early exit from
    // inside the loop would make every wait in it conservative.
    const int nfull = nu / D;
    for (int i0 = 0; i0 < nfull * D; i0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        // Keep units in source order: hoisting a later unit's products above
        // this point would make the wave wait for that unit's loads too.
        __builtin_amdgcn_sched_barrier(0);
        process(ring[u], i0 + u, true);
      }
    }
#pragma unroll
    for (int u = 0; u < D - 1; ++u) {
      __builtin_amdgcn_sched_barrier(0);
      if (nfull * D + u < nu) process(ring[u], nfull * D + u, false);
    }
  }

  // ---- merge the waves' partial results; write the split's partial result ----
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t pbase = (static_cast<int64_t>(b) * a.s_max + s) * a.H + hg * 16;
  if (g == 0) mbuf[w * 16 + r16] = m_run;
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < NWT; ++v) M = fmaxf(M, mbuf[v * 16 + r16]);  // finite: the split has a token
  const float sc = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - M);
#pragma unroll
  for (int db = 0; db < NB; ++db) obuf[(w * NB + db) * 64 + lane] = o[db] * sc;
  if (g == 0) lbuf[w * 16 + r16] = l_run * sc;
  __syncthreads();
  // lane holds O^T[dim = 16 db + 4g + q][head r16]
  for (int db = w; db < NB; db += NWT) {
    f32x4_t sum = obuf[db * 64 + lane];
#pragma unroll
    for (int v = 1; v < NWT; ++v) sum += obuf[(v * NB + db) * 64 + lane];
    __builtin_nontemporal_store(sum, reinterpret_cast<f32x4_t*>(a.part_o + (pbase + r16) * DC + db * 16 + 4 * g));
  }
  if (w == 0 && g == 0) {
    float Ls = 0.f;
#pragma unroll
    for (int v = 0; v < NWT; ++v) Ls += lbuf[v * 16 + r16];
    __builtin_nontemporal_store(M, a.part_ml + (pbase + r16) * 2 + 0);
    __builtin_nontemporal_store(Ls, a.part_ml + (pbase + r16) * 2 + 1);
  }
}

}  // namespace egmla
