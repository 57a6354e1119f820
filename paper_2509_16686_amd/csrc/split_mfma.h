// MFMA split kernel of EG-MLA decode (bf16 storage, 16 heads per work-group).
// Included by decode.hip after SplitArgs.
//
// One work-group per (sequence, split, head group of 16).  Its NW waves split
// the row's dimensions, not its tokens: wave w owns CPW 32-dim chunks of the
// latent (and at most one 32-dim chunk of the RoPE key), and every wave sees
// every 32-token tile of the split.  For a tile, wave w
//   * loads its chunks of each token's row straight into the layout of the
//     MFMA A operand (lane: token lane%16 of a 16-token half, 16 bytes = 8
//     consecutive dims), the matching 16 bytes of the token's gate row, and
//     gates in fp32 (exact product), rounding the gated latent to fp16 once;
//   * computes its partial scores S^T[token][head] over its dims with
//     v_mfma_f32_16x16x32_f16, the fp32 absorbed query rounded once to fp16
//     (11-bit significands: rows dominated by a few keys stay within the
//     element-wise bound; magnitudes must stay below 65504), and the RoPE
//     part with v_mfma_f32_16x16x32_bf16 (bf16 x bf16: exact);
//   * adds the partial scores of all waves through LDS (double-buffered, one
//     barrier per tile), so every wave holds the full scores;
//   * runs the online softmax on the accumulator layout (lane: one head, 4
//     tokens per half); the probabilities are exactly the B operand of the
//     value product, so P never leaves registers;
//   * accumulates O^T[dim][head] += C~^T x P^T (fp16) for its own dims,
//     reading the transposed gated latent it wrote to its own LDS region.
// The waves' dims are disjoint and their softmax statistics identical, so
// each writes its part of the split's partial result directly.
//
// Load scheduling.  All work-groups start together and the whole launch
// streams through HBM at once, so memory queues stay deep and a load issued
// late waits for the bytes queued ahead of it; loads also return in issue
// order per wave.  So (1) the token ids and cache rows of the whole split
// are resolved once at the start into LDS, (2) the query chunks are loaded
// into registers at the start, and (3) in the tile loop every global load
// depends only on LDS, and is issued kDepth tiles ahead of its use.
#pragma once

namespace egmla {

template <int DC, int DR>
struct DsplitCfg {
  static constexpr int NLC = DC / 32;                  // latent chunks
  static constexpr int NRC = DR / 32;                  // RoPE chunks
  static constexpr int CPW = DC == 128 ? 1 : 2;        // latent chunks per wave
  static constexpr int NW = NLC / CPW;                 // waves per work-group
  static constexpr int RPW = NRC > 0 ? 1 : 0;          // RoPE chunk slots per wave (waves < NRC own theirs)
  static constexpr int NDB = CPW * 2;                  // 16-dim blocks of the value product per wave
  static constexpr int kDepth = DC == 128 ? 4 : 3;     // tiles in flight per wave
  static constexpr int CT_STRIDE = 40;                 // 32 token slots + 8 pad (16-bit elements)
  static constexpr int LDS_CT = NW * CPW * 32 * CT_STRIDE * 2;
  static constexpr int LDS_SC = 2 * NW * 64 * 8 * 4;   // partial scores, double-buffered
  static constexpr int LDS_TOK = kMaxSplitTokensDevice * 8;  // slot + id of every token of the split
  static constexpr int LDS_BYTES = LDS_CT + LDS_SC + LDS_TOK;
  static_assert(NLC % CPW == 0 && NRC <= NW, "chunk distribution");
};

// Position of token t (0..31) of a tile in a transposed LDS row: the 8
// k-slots of lane group g hold tokens 4g..4g+3 of each 16-token half.
__device__ __forceinline__ int ct_pos(int half, int t16) { return (t16 >> 2) * 8 + half * 4 + (t16 & 3); }

// One tile of this wave's operands, per 16-token half.
template <int CPW, int RPW>
struct TileRegs {
  u32x4_t lat[2][CPW];
  u32x4_t gat[2][CPW];
  u32x4_t rop[2][RPW > 0 ? RPW : 1];
};

template <int DC, int DR>
__global__ __launch_bounds__((DsplitCfg<DC, DR>::NW * 64)) void split_mfma_kernel(SplitArgs a) {
  using Cfg = DsplitCfg<DC, DR>;
  constexpr int NW = Cfg::NW, CPW = Cfg::CPW, RPW = Cfg::RPW, NDB = Cfg::NDB, D = Cfg::kDepth;
  constexpr int DQ = DC + DR;
  constexpr int CTS = Cfg::CT_STRIDE;
  __shared__ __attribute__((aligned(16))) unsigned char lds[Cfg::LDS_BYTES];
  uint16_t* ct_all = reinterpret_cast<uint16_t*>(lds);
  float* sbuf = reinterpret_cast<float*>(lds + Cfg::LDS_CT);          // [2][NW][64][8]
  int* tok_slot = reinterpret_cast<int*>(lds + Cfg::LDS_CT + Cfg::LDS_SC);
  int* tok_id = tok_slot + kMaxSplitTokensDevice;

  const int item = xcd_logical_block(blockIdx.x, gridDim.x);
  const int hg = item % a.groups;
  const int s = (item / a.groups) % a.s_max;
  const int b = item / (a.groups * a.s_max);
  const int t0 = s * a.split;
  const int L = clamp_len(a.seq_lens[b], a.cap);
  if (t0 >= L) return;  // empty split (uniform over the work-group)
  const int t1 = min(t0 + a.split, L);
  const int n = t1 - t0;
  const int ntiles = (n + kTile - 1) / kTile;

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const bool has_rope = RPW > 0 && w < Cfg::NRC;
  // RoPE chunk this wave loads: its own, else a duplicate of another wave's
  // (against a zero query), so the loads never depend on a branch.
  const int rope_chunk = Cfg::NRC > 0 ? w % (Cfg::NRC > 0 ? Cfg::NRC : 1) : 0;

  // ---- (1) resolve slots and ids of the split; (2) query chunks of this wave ----
  for (int j = tid; j < n; j += NW * 64) {
    const int sl = static_cast<int>(cache_slot(a.page_table, b, t0 + j, a.P, a.max_pages, a.num_slots));
    tok_slot[j] = sl;
    tok_id[j] = clamp_id(a.ids[sl], a.V);
  }
  // Waves without a RoPE chunk of their own use a zero RoPE query, so their
  // (duplicate) RoPE product adds exactly zero and nothing depends on a branch.
  f16x8_t qh[CPW];
  bf16x8_t qr = {};
  {
    const float* qrow = a.qfull + (static_cast<int64_t>(b) * a.H + hg * 16 + r16) * DQ + g * 8;
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
      const float* p = qrow + (w * CPW + c) * 32;
      const float4 x0 = *reinterpret_cast<const float4*>(p);
      const float4 x1 = *reinterpret_cast<const float4*>(p + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) qh[c][e] = static_cast<_Float16>(x[e]);
    }
    if constexpr (RPW > 0) {
      const float* p = qrow + DC + rope_chunk * 32;
      const float4 x0 = *reinterpret_cast<const float4*>(p);
      const float4 x1 = *reinterpret_cast<const float4*>(p + 4);
      const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) qr[e] = static_cast<__bf16>(has_rope ? x[e] : 0.f);  // q^R is bf16: exact
    }
  }
  __syncthreads();

  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache) + g * 8;
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate) + g * 8;

  // Loads of tile k into `r`; every address comes from LDS.
  auto issue = [&](TileRegs<CPW, RPW>& r, int k) {
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      const int j = min(k * kTile + hf * 16 + r16, n - 1);  // past the end: repeat the last token (masked)
      const int sl = tok_slot[j];
      const int id = tok_id[j];
      const uint16_t* row = cache + static_cast<int64_t>(sl) * DQ;
      const uint16_t* grow = gate + static_cast<int64_t>(id) * DC;
#pragma unroll
      for (int c = 0; c < CPW; ++c) {
        r.gat[hf][c] = *reinterpret_cast<const u32x4_t*>(grow + (w * CPW + c) * 32);
        r.lat[hf][c] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(row + (w * CPW + c) * 32));
      }
      if constexpr (RPW > 0)
        r.rop[hf][0] = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(row + DC + rope_chunk * 32));
    }
  };

  // Every load is unconditional (indexes past the split repeat its last
  // token), so the compiler's wait counters track each tile exactly and D
  // tiles stay in flight; a branch around a load would make it wait for all.
  // Loads return in issue order, so tile k must also be issued before tile k + 1.
  TileRegs<CPW, RPW> ring[D];
#pragma unroll
  for (int k = 0; k < D; ++k) {
    issue(ring[k], k);
    __builtin_amdgcn_sched_barrier(0);
  }

  f32x4_t o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // running max of head r16 (log2 domain), identical in every wave
  float l_run = 0.f;        // this lane's share of the running sum
  uint16_t* ct = ct_all + w * CPW * 32 * CTS;  // this wave's [CPW*32 dims][CTS]

  // Tiles run in groups of D; those past the split are fully masked (their
  // probabilities are exactly 0 and the running max is unchanged).
  const int ngroups = (ntiles + D - 1) / D;
  for (int k0 = 0; k0 < ngroups * D; k0 += D) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      // Keep tiles in source order: hoisting a later tile's products above
      // this point would make the wave wait for that tile's loads too.
      __builtin_amdgcn_sched_barrier(0);
      const int k = k0 + u;
      TileRegs<CPW, RPW>& r = ring[u];
      const int nt = n - k * kTile;  // valid tokens of the tile (may be <= 0)

      // partial scores over this wave's dims
      f32x4_t sp[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int pos = ct_pos(hf, r16);
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < CPW; ++c) {
          uint32_t pk[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float p0 = bf16_lo(r.lat[hf][c][e]) * bf16_lo(r.gat[hf][c][e]);
            const float p1 = bf16_hi(r.lat[hf][c][e]) * bf16_hi(r.gat[hf][c][e]);
            pk[e] = pack_f16x2(p0, p1);
          }
          const u32x4_t hv = {pk[0], pk[1], pk[2], pk[3]};
          const f16x8_t av = __builtin_bit_cast(f16x8_t, hv);
          uint16_t* col = ct + (c * 32 + g * 8) * CTS + pos;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            col[(2 * e) * CTS] = static_cast<uint16_t>(pk[e] & 0xffffu);
            col[(2 * e + 1) * CTS] = static_cast<uint16_t>(pk[e] >> 16);
          }
          acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, qh[c], acc, 0, 0, 0);
        }
        if constexpr (RPW > 0)
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r.rop[hf][0]), qr, acc, 0, 0, 0);
        sp[hf] = acc;
      }
      // this tile's registers are free: issue tile k + D into them
      issue(r, k + D);

      // sum the partial scores of all waves
      float* sb = sbuf + ((k & 1) * NW) * 64 * 8;
      *reinterpret_cast<f32x4_t*>(sb + (w * 64 + lane) * 8) = sp[0];
      *reinterpret_cast<f32x4_t*>(sb + (w * 64 + lane) * 8 + 4) = sp[1];
      __syncthreads();
      f32x4_t sc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
#pragma unroll
      for (int v = 0; v < NW; ++v) {
        sc[0] += *reinterpret_cast<const f32x4_t*>(sb + (v * 64 + lane) * 8);
        sc[1] += *reinterpret_cast<const f32x4_t*>(sb + (v * 64 + lane) * 8 + 4);
      }

      // online softmax: lane holds head r16, tokens hf*16 + 4g + r
      float sv[8];
      float mt = -INFINITY;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int tk = hf * 16 + 4 * g + q;
          const float x = tk < nt ? sc[hf][q] * a.scale_log2 : -INFINITY;
          sv[hf * 4 + q] = x;
          mt = fmaxf(mt, x);
        }
      }
      mt = fmaxf(mt, __shfl_xor(mt, 16, 64));
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2f(m_run - m_new);
      m_run = m_new;
      float psum = 0.f;
      f16x8_t pb;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float p = exp2f(sv[i] - m_new);
        psum += p;
        pb[i] = static_cast<_Float16>(p);
      }
      l_run = l_run * alpha + psum;
#pragma unroll
      for (int i = 0; i < NDB; ++i) o[i] *= alpha;

      // value product over this wave's dims (its own LDS region)
      wave_lds_sync();
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const f16x8_t av = *reinterpret_cast<const f16x8_t*>(ct + (db * 16 + r16) * CTS + g * 8);
        o[db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, pb, o[db], 0, 0, 0);
      }
      wave_lds_sync();
    }
  }

  // ---- this wave's dims of the split's partial result ----
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t pbase = (static_cast<int64_t>(b) * a.s_max + s) * a.H + hg * 16;
  // lane holds O^T[dim = (w*CPW*2 + db)*16 + 4g + q][head r16]
#pragma unroll
  for (int db = 0; db < NDB; ++db) {
    float* dst = a.part_o + (pbase + r16) * DC + (w * NDB + db) * 16 + 4 * g;
    __builtin_nontemporal_store(o[db], reinterpret_cast<f32x4_t*>(dst));
  }
  if (w == 0 && g == 0) {
    __builtin_nontemporal_store(m_run, a.part_ml + (pbase + r16) * 2 + 0);
    __builtin_nontemporal_store(l_run, a.part_ml + (pbase + r16) * 2 + 1);
  }
}

}  // namespace egmla
