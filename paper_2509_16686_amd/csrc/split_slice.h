// Id-sliced MFMA split kernel of EG-MLA decode (bf16 storage, 16 heads per
// work-group, latent dim <= 128).  Included by decode.hip after SplitArgs.
//
// Work item: (sequence b, context split s, head group, id slice k).  With SL
// slices, the work item of slice k handles the split's tokens whose id is
// k mod SL, and the grid is ordered so that work-group x runs slice x % SL.
// The dispatcher hands work-groups to the 8 XCDs of an MI355X round-robin, so
// with SL = 8 every XCD gathers gate rows from one eighth of the gate table
// only (the rows of ids = k mod 8), which stays in that XCD's L2 cache
// instead of every XCD fetching its own copy of most of the table.  The
// softmax over a sequence does not depend on how its tokens are grouped:
// every slice emits a partial (max, sum, output) that the split merge
// combines exactly like the partials of different context splits.  SL = 1
// processes every token of the split (no slicing).
//
// Phase 1 (token list).  The split's positions are scanned in rows of 256
// (wave r % NW takes row r; lane l the 4 positions 4l .. 4l + 3): each
// position's cache slot (page table or contiguous) and token id are loaded,
// the tokens of this slice kept, and their (slot, id) written to an LDS list
// in position order.
// Phase 2 (units).  The list forms 16-token units; unit u belongs to wave
// u % NW.  For a unit the wave
//   * loads whole 128-byte lines: each latent and gate instruction covers 4
//     tokens x 256 bytes (16 lanes per token, 16 bytes each), each RoPE-key
//     instruction 8 tokens x 128 bytes;
//   * gates in fp32 (exact product of two bf16 values), rounds once to fp16
//     and stores the gated unit row-major ([token][latent fp16 | RoPE key
//     bf16]) in its own LDS tile;
//   * reads the tile back in the layout of the MFMA A operand (lane: token
//     lane % 16, 16 bytes = 8 consecutive dims of a 32-dim chunk) and
//     computes S^T[token][head]: the latent part on v_mfma_f32_16x16x32_f16
//     with the absorbed query rounded once to fp16, the RoPE part on
//     v_mfma_f32_16x16x32_bf16 (bf16 x bf16: exact);
//   * runs the online softmax on the accumulator layout (lane: one head, 4
//     tokens), rescaling only when a head's maximum grows by more than 2^8;
//   * reads each 16-dim block of the latent part with ds_read_b64_tr_b16,
//     whose 16-lane transpose is the A operand of v_mfma_f32_16x16x16_f16,
//     and accumulates O^T[dim][head] += C~^T x P^T (P in fp16).
// fp16's 11-bit significands keep rows dominated by a few keys within the
// element-wise bound with one product per chunk, where bf16 operands needed
// hi + lo products; magnitudes must stay below 65504.
// Every global load of a unit depends only on the LDS list and is issued D
// units ahead of its use, unconditionally (indexes past the list repeat its
// last token), so the compiler's wait counters track each unit.
// Phase 3.  The waves merge their (max, sum, output) and write the partial.
#pragma once

namespace egmla {

// Largest number of positions one work item of the sliced kernel scans.
constexpr int kMaxScanTokens = 4096;

template <int DC, int DR, int NW>
struct SsplitCfg {
  static constexpr int DQ = DC + DR;
  static constexpr int NC = DC / 32;                 // 32-dim latent chunks (score MFMA)
  static constexpr int NR = DR / 32;                 // 32-dim RoPE chunks
  static constexpr int NB = DC / 16;                 // 16-dim blocks of the value product
  static constexpr int LPT = DC / 8;                 // lanes per token of a latent / gate load
  static constexpr int TPL = 64 / LPT;               // tokens per latent / gate load instruction
  static constexpr int NLI = 16 / TPL;               // latent (and gate) load instructions per unit
  static constexpr int RPT = DR / 8;                 // lanes per token of a RoPE load
  static constexpr int TPR = RPT > 0 ? 64 / RPT : 1; // tokens per RoPE load instruction
  static constexpr int NRI = RPT > 0 ? 16 / TPR : 0; // RoPE load instructions per unit
  static constexpr int TS = DQ + 8;                  // tile row: latent (fp16) | RoPE key (bf16) | 16 bytes of padding
  static constexpr int ROWS = kMaxScanTokens / 256;  // scan rows of a work item, at most
  static constexpr int RPW = ROWS / NW;              // scan rows per wave, at most
  static constexpr int LDS_LIST = kMaxScanTokens * 8;            // slot + id of every kept token
  static constexpr int LDS_ROWS = ROWS * 4;                      // kept tokens per scan row
  static constexpr int LDS_TILE = NW * 16 * TS * 2;              // each wave's gated unit
  static constexpr int LDS_MERGE = NW * NB * 64 * 16;            // every wave's accumulators (aliases the above)
  static constexpr int LDS_A = LDS_LIST + LDS_ROWS + LDS_TILE;
  static constexpr int LDS_MAIN = LDS_A > LDS_MERGE ? LDS_A : LDS_MERGE;
  static constexpr int LDS_STAT = NW * 16 * 4 * 2;               // every wave's max and sum per head
  static constexpr int LDS_BYTES = LDS_MAIN + LDS_STAT;
  static_assert(DC % 32 == 0 && DR % 32 == 0 && DC <= 128 && 64 % LPT == 0 && (DR == 0 || 64 % RPT == 0),
                "sliced-kernel shapes");
  static_assert(ROWS % NW == 0, "scan rows per wave");
};

// One unit's loads: this lane's 16 bytes of every latent, gate and RoPE instruction.
template <int NLI, int NRI>
struct SliceRegs {
  u32x4_t lat[NLI];
  u32x4_t gat[NLI];
  u32x4_t rop[NRI > 0 ? NRI : 1];
};

// Exclusive prefix over the lanes of a wave, and the wave total, of a count
// in 0..7 (three ballots).
__device__ __forceinline__ void wave_count_prefix(int cnt, int& pre, int& tot) {
  const uint64_t m0 = __builtin_amdgcn_ballot_w64((cnt & 1) != 0);
  const uint64_t m1 = __builtin_amdgcn_ballot_w64((cnt & 2) != 0);
  const uint64_t m2 = __builtin_amdgcn_ballot_w64((cnt & 4) != 0);
  auto below = [](uint64_t m) {
    return static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(m >> 32),
                                                      __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(m), 0u)));
  };
  pre = below(m0) + 2 * below(m1) + 4 * below(m2);
  tot = __builtin_popcountll(m0) + 2 * __builtin_popcountll(m1) + 4 * __builtin_popcountll(m2);
}

// Cache slots of positions t0 + p[e] of sequence b, for e < ne (ne is
// uniform): with a page table, the page entries are all loaded before any is
// used, so the slots cost one round trip whatever N is; contiguous slots are
// arithmetic.  Clamped into the cache like cache_slot().
template <int N>
__device__ __forceinline__ void split_slots(const SplitArgs& a, int b, int t0, const int (&p)[N], int (&o)[N],
                                            int ne) {
  if (a.page_table) {
    const int32_t* pt = a.page_table + static_cast<int64_t>(b) * a.max_pages;
    int pg[N];
#pragma unroll
    for (int e = 0; e < N; ++e)
      if (e < ne) pg[e] = pt[(t0 + p[e]) / a.P];
#pragma unroll
    for (int e = 0; e < N; ++e)
      if (e < ne) o[e] = static_cast<int>(paged_slot(pg[e], t0 + p[e], a.P, a.num_slots));
  } else {
#pragma unroll
    for (int e = 0; e < N; ++e)
      if (e < ne) o[e] = static_cast<int>(contiguous_slot(b, t0 + p[e], a.P, a.max_pages, a.num_slots));
  }
}

// Absorption of one head inside the split kernel (256 threads, d_h = d_c =
// 128): q_lat[b][h][c] = sum_k q^C[b][h][k] W_UK[h][k][c].  Thread t takes
// columns 8 (t % 16) .. + 7 over rows 8 (t / 16) .. + 7 (exact bf16 products,
// fp32 sums); the 16 row groups are added in LDS (red: 16 x 128 floats) in a
// fixed order, so every work-group that absorbs a head produces the same
// bits.  Threads t < 128 store column t with device-coherent stores (they
// bypass this XCD's L2), for work-groups on any XCD to read once the stamp of
// this work-group says they are complete.
struct AbsorbRegs {
  u32x4_t wv[8];  // W_UK rows 8 (t / 16) .. + 7, columns 8 (t % 16) .. + 7
  u32x4_t qv;     // q^C[8 (t / 16) .. + 7]
};
__device__ __forceinline__ void absorb_load(const SplitArgs& a, int b, int h, AbsorbRegs& r) {
  constexpr int DH = 128, DCa = 128;
  const int tid = threadIdx.x, cg = tid & 15, kg = tid >> 4;
  const uint16_t* wrow = a.w_uk + (static_cast<int64_t>(h) * DH + 8 * kg) * DCa + 8 * cg;
#pragma unroll
  for (int k = 0; k < 8; ++k) r.wv[k] = *reinterpret_cast<const u32x4_t*>(wrow + k * DCa);
  r.qv = *reinterpret_cast<const u32x4_t*>(a.qin + (static_cast<int64_t>(b) * a.H + h) * (DH + a.DR) + 8 * kg);
}
__device__ __forceinline__ void absorb_finish(const SplitArgs& a, int b, int h, const AbsorbRegs& ar, float* red) {
  constexpr int DH = 128, DCa = 128;
  const int tid = threadIdx.x, cg = tid & 15, kg = tid >> 4;
  const u32x4_t* wv = ar.wv;
  const u32x4_t qv = ar.qv;
  float acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = 0.f;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const float qk = (r & 1) ? bf16_hi(qv[r >> 1]) : bf16_lo(qv[r >> 1]);
#pragma unroll
    for (int i = 0; i < 8; ++i) acc[i] = fmaf(qk, (i & 1) ? bf16_hi(wv[r][i >> 1]) : bf16_lo(wv[r][i >> 1]), acc[i]);
  }
  *reinterpret_cast<float4*>(red + kg * DCa + 8 * cg) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  *reinterpret_cast<float4*>(red + kg * DCa + 8 * cg + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
  __syncthreads();
  if (tid < DCa) {
    float v = 0.f;
#pragma unroll
    for (int k = 0; k < DH / 8; ++k) v += red[k * DCa + tid];
    float* qf = const_cast<float*>(a.qfull) + (static_cast<int64_t>(b) * a.H + h) * (a.DC + a.DR) + tid;
    __hip_atomic_store(qf, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();  // red is free again
}
__device__ __forceinline__ void absorb_head_128(const SplitArgs& a, int b, int h, float* red) {
  AbsorbRegs r;
  absorb_load(a, b, h, r);
  absorb_finish(a, b, h, r, red);
}

// FUSED (no id slices, d_h = 128): the work-groups of a sequence also absorb
// its query.  Split s of the ns non-empty splits of sequence b absorbs the heads
// j (of its group of 16) with j = s mod ns: their W_UK rows load with the page
// table entries, the products are formed and stored device-coherently
// before the token ids are loaded, and once the ids are in (vector memory
// operations complete in issue order, so the stores are then complete) the
// work-group publishes the call's stamp in qflags[b][group][s].  Before its first scores a work-group waits for the
// stamps of splits 0 .. min(ns, 16) - 1 (the other work-groups of the
// sequence run at the same time: one work-group per compute unit), polling at
// most spin_limit times; if one is missing it absorbs all 16 heads itself
// (the same bits), so the wait always ends.
template <int DC, int DR, int NW, int D, int SL, bool FUSED = false>
__global__ __launch_bounds__(NW * 64, 2) void split_slice_kernel(SplitArgs a) {
  using Cfg = SsplitCfg<DC, DR, NW>;
  constexpr int NC = Cfg::NC, NR = Cfg::NR, NB = Cfg::NB, DQ = Cfg::DQ, TS = Cfg::TS;
  constexpr int LPT = Cfg::LPT, TPL = Cfg::TPL, NLI = Cfg::NLI;
  constexpr int RPT = Cfg::RPT > 0 ? Cfg::RPT : 1, TPR = Cfg::TPR, NRI = Cfg::NRI;
  static_assert(SL == 1 || SL == 8, "id slices");
  __shared__ __attribute__((aligned(16))) unsigned char lds[Cfg::LDS_BYTES];
  int* l_slot = reinterpret_cast<int*>(lds);                   // [kMaxScanTokens]
  int* l_id = l_slot + kMaxScanTokens;                         // [kMaxScanTokens]
  int* rowcnt = l_id + kMaxScanTokens;                         // [ROWS]
  uint16_t* tile_all = reinterpret_cast<uint16_t*>(lds + Cfg::LDS_LIST + Cfg::LDS_ROWS);  // [NW][16][TS]
  f32x4_t* obuf = reinterpret_cast<f32x4_t*>(lds);             // [NW][NB][64], after the units
  float* mbuf = reinterpret_cast<float*>(lds + Cfg::LDS_MAIN); // [NW][16]
  float* lbuf = mbuf + NW * 16;                                // [NW][16]

  // work-group x runs slice x % SL (its XCD); the rest is the (b, s, group) item
  const int k = SL > 1 ? static_cast<int>(blockIdx.x % SL) : 0;
  const int item = SL > 1 ? static_cast<int>(blockIdx.x / SL) : xcd_logical_block(blockIdx.x, gridDim.x);
  const int hg = item % a.groups;
  const int s = (item / a.groups) % a.s_max;
  const int b = item / (a.groups * a.s_max);
  const int t0 = s * a.split;
  const int L = clamp_len(a.seq_lens[b], a.cap);
  if (t0 >= L) return;  // empty split: the merge reads no partial of it (uniform over the work-group)
  const int n = min(t0 + a.split, L) - t0;

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);

  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate);
  const int lt = lane / LPT, lc = 8 * (lane % LPT);  // token within a latent / gate instruction, first dim
  const int rt = lane / RPT, rcol = 8 * (lane % RPT);
  constexpr int NRL = NLI + NRI;  // row loads per unit
  // List entries (clamped to the list: past its end the last token repeats,
  // masked) whose rows this lane loads for this wave's unit i: latent
  // instruction c < NLI, then RoPE instruction c.
  auto row_entries = [&](int i, int nlist, int* jj) {
    const int j0 = (w + i * NW) * 16;
#pragma unroll
    for (int c = 0; c < NLI; ++c) jj[c] = min(j0 + TPL * c + lt, nlist - 1);
#pragma unroll
    for (int c = 0; c < NRI; ++c) jj[NLI + c] = min(j0 + TPR * c + rt, nlist - 1);
  };
  // Row loads of one unit given the cache slot of each of its row_entries.
  auto issue_rows = [&](SliceRegs<NLI, NRI>& rg, const int* sl) {
#pragma unroll
    for (int c = 0; c < NLI; ++c)
      rg.lat[c] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(cache + static_cast<int64_t>(sl[c]) * DQ + lc));
#pragma unroll
    for (int c = 0; c < NRI; ++c)
      rg.rop[c] = __builtin_nontemporal_load(
          reinterpret_cast<const u32x4_t*>(cache + static_cast<int64_t>(sl[NLI + c]) * DQ + DC + rcol));
  };
  auto issue_list_rows = [&](SliceRegs<NLI, NRI>& rg, int i, int nlist) {
    int jj[NRL], sl[NRL];
    row_entries(i, nlist, jj);
#pragma unroll
    for (int c = 0; c < NRL; ++c) sl[c] = l_slot[jj[c]];
    issue_rows(rg, sl);
  };
  auto issue_gates = [&](SliceRegs<NLI, NRI>& rg, int i, int nlist) {
    const int j0 = (w + i * NW) * 16;
#pragma unroll
    for (int c = 0; c < NLI; ++c) {
      const int j = min(j0 + TPL * c + lt, nlist - 1);
      rg.gat[c] = *reinterpret_cast<const u32x4_t*>(gate + static_cast<int64_t>(l_id[j]) * DC + lc);
    }
  };

  // This lane's query values (fp32: absorbed query chunks, then RoPE chunks),
  // loaded right after the ids so that waiting for them (loads complete in
  // issue order) does not wait for any cache row.
  float4 qraw[2 * (NC + NR)];
  auto load_q = [&]() {
    const float* qrow = a.qfull + (static_cast<int64_t>(b) * a.H + hg * 16 + r16) * DQ + g * 8;
#pragma unroll
    for (int c = 0; c < NC + NR; ++c) {
      qraw[2 * c] = *reinterpret_cast<const float4*>(qrow + c * 32);
      qraw[2 * c + 1] = *reinterpret_cast<const float4*>(qrow + c * 32 + 4);
    }
  };

  SliceRegs<NLI, NRI> ring[D];
  int ntok;
  if constexpr (SL == 1) {
    // ---- phase 1 without slices: the list is the split's positions ----
    // slot and id of every position (all loads first, clamped into the split)
    constexpr int PER = kMaxScanTokens / (NW * 64);
    const int nper = (n + NW * 64 - 1) / (NW * 64);  // uniform
    int pp[PER], psl[PER], pid[PER];
#pragma unroll
    for (int e = 0; e < PER; ++e) pp[e] = min(tid + e * NW * 64, n - 1);
    // FUSED: this split's heads j = s, s + ns, ... < 16 of the group; the
    // W_UK rows of the first two load together with the page table entries
    const int ns = (L + a.split - 1) / a.split;  // non-empty splits of sequence b (s < ns)
    AbsorbRegs pre[FUSED ? 2 : 1];
    if constexpr (FUSED) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (s + i * ns < 16) absorb_load(a, b, hg * 16 + s + i * ns, pre[i]);
    }
    split_slots(a, b, t0, pp, psl, nper);
    if constexpr (FUSED) {
      // (the LDS list is written after this)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        if (s + i * ns < 16) absorb_finish(a, b, hg * 16 + s + i * ns, pre[i], reinterpret_cast<float*>(lds));
      for (int j = s + 2 * ns; j < 16; j += ns) absorb_head_128(a, b, hg * 16 + j, reinterpret_cast<float*>(lds));
      __atomic_signal_fence(__ATOMIC_SEQ_CST);  // the stores above are issued before the loads below
    }
#pragma unroll
    for (int e = 0; e < PER; ++e)
      if (e < nper) pid[e] = a.ids[psl[e]];
    if constexpr (!FUSED) load_q();
    // The rows of this wave's first D units need no token id: issue them now,
    // after the ids (loads complete in issue order), so they stream while the
    // ids are on their way.
    {
      int rp[D * NRL], rs[D * NRL];
#pragma unroll
      for (int u = 0; u < D; ++u) row_entries(u, n, rp + u * NRL);
      split_slots(a, b, t0, rp, rs, D * NRL);
#pragma unroll
      for (int u = 0; u < D; ++u) issue_rows(ring[u], rs + u * NRL);
    }
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const int j = tid + e * NW * 64;
      if (e < nper && j < n) {
        l_slot[j] = psl[e];
        l_id[j] = clamp_id(pid[e], a.V);
      }
    }
    ntok = n;
    if constexpr (FUSED) {
      if (s < 16) {
        // Only the first rows' D * NRL loads, issued last, may still be in
        // flight: this thread's absorbed stores, issued before its ids, are
        // complete.  Then the stamp goes out.
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(D * NRL) : "memory");
        __syncthreads();
        if (tid == 0)
          __hip_atomic_store(a.qflags + (static_cast<int64_t>(b) * a.groups + hg) * a.s_max + s, a.stamp,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  } else {
    // ---- phase 1a: slots and ids of this wave's scan rows (all loads first) ----
    const int nrows = (n + 255) / 256;
    // 4 consecutive positions share one 16-byte id load when their slots are
    // consecutive and 16-byte aligned: contiguous rows with the capacity a
    // multiple of 4, or pages of a multiple of 4 tokens
    const bool vec = (reinterpret_cast<uintptr_t>(a.ids) % 16 == 0) &&
                     (a.page_table ? (a.P % 4 == 0) : (a.cap % 4 == 0));
    const int nrw = nrows > w ? (nrows - w + NW - 1) / NW : 0;  // this wave's scan rows (uniform)
    int sl[Cfg::RPW][4], id[Cfg::RPW][4];
    if (vec) {
      // one 16-byte id load per 4 positions, at the slot of the first
      int p4[Cfg::RPW], s4[Cfg::RPW];
#pragma unroll
      for (int i = 0; i < Cfg::RPW; ++i) p4[i] = min(256 * (w + i * NW) + 4 * lane, n - 1) & ~3;
      split_slots(a, b, t0, p4, s4, nrw);
#pragma unroll
      for (int i = 0; i < Cfg::RPW; ++i) {
        if (i < nrw) {
          const int4 v = *reinterpret_cast<const int4*>(a.ids + s4[i]);
          sl[i][0] = s4[i]; sl[i][1] = s4[i] + 1; sl[i][2] = s4[i] + 2; sl[i][3] = s4[i] + 3;
          id[i][0] = v.x; id[i][1] = v.y; id[i][2] = v.z; id[i][3] = v.w;
        }
      }
    } else {
      int p1[Cfg::RPW * 4], s1[Cfg::RPW * 4];
#pragma unroll
      for (int i = 0; i < Cfg::RPW; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) p1[4 * i + e] = min(256 * (w + i * NW) + 4 * lane + e, n - 1);
      split_slots(a, b, t0, p1, s1, 4 * nrw);
#pragma unroll
      for (int i = 0; i < Cfg::RPW; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (i < nrw) {
            sl[i][e] = s1[4 * i + e];
            id[i][e] = a.ids[sl[i][e]];
          }
    }
    load_q();
    // ---- phase 1b: keep this slice's tokens; count them per scan row ----
    int keep[Cfg::RPW], pre[Cfg::RPW];
#pragma unroll
    for (int i = 0; i < Cfg::RPW; ++i) {
      const int r = w + i * NW;
      keep[i] = 0;
      pre[i] = 0;
      if (r < nrows) {
        const int p0 = 256 * r + 4 * lane;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          id[i][e] = clamp_id(id[i][e], a.V);
          const bool kp = p0 + e < n && (id[i][e] & (SL - 1)) == k;
          keep[i] |= kp ? (1 << e) : 0;
        }
        int tot;
        wave_count_prefix(__builtin_popcount(keep[i]), pre[i], tot);
        if (lane == 0) rowcnt[r] = tot;
      }
    }
    __syncthreads();
    // ---- phase 1c: write the kept tokens at their place in the list ----
    ntok = 0;
    for (int r = 0; r < nrows; ++r) ntok += rowcnt[r];
#pragma unroll
    for (int i = 0; i < Cfg::RPW; ++i) {
      const int r = w + i * NW;
      if (r < nrows) {
        int off = pre[i];
        for (int rr = 0; rr < r; ++rr) off += rowcnt[rr];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (keep[i] & (1 << e)) {
            l_slot[off] = sl[i][e];
            l_id[off] = id[i][e];
            ++off;
          }
        }
      }
    }
  }
  // query chunks: absorbed query in fp16, RoPE query (a stored bf16 value: exact)
  f16x8_t qh[NC];
  bf16x8_t qr[NR > 0 ? NR : 1];
  if constexpr (FUSED) {
    __syncthreads();  // the list is complete (and the absorption's LDS is free)
    const int ns = (L + a.split - 1) / a.split;
    const int np = min(ns, 16);
    int* okp = reinterpret_cast<int*>(mbuf);
    if (w == 0) {
      const unsigned long long* fl = a.qflags + (static_cast<int64_t>(b) * a.groups + hg) * a.s_max;
      bool ok = false;
      for (int it = 0;; ++it) {
        const unsigned long long v =
            lane < np ? __hip_atomic_load(fl + lane, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : a.stamp;
        ok = __builtin_amdgcn_ballot_w64(v != a.stamp) == 0;
        if (ok || it >= a.spin_limit) break;
        __builtin_amdgcn_s_sleep(4);
      }
      if (lane == 0) okp[0] = ok ? 1 : 0;
    }
    __syncthreads();
    if (okp[0] == 0) {
      // a producer has not run yet: absorb the group's 16 heads here
      for (int j = 0; j < 16; ++j) absorb_head_128(a, b, hg * 16 + j, reinterpret_cast<float*>(tile_all));
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
    // latent part: device-coherent 16-byte loads of the absorbed rows; RoPE
    // part straight from the query
    const int h = hg * 16 + r16;
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.qfull), 0, static_cast<int>(static_cast<int64_t>(a.B) * a.H * (DC + DR) * 4), 0x00020000);
    const int qoff = static_cast<int>(((static_cast<int64_t>(b) * a.H + h) * (DC + DR) + 8 * g) * 4);
    f32x4_t xq[2 * NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      xq[2 * c] = __builtin_amdgcn_raw_buffer_load_b128(rq, qoff + 128 * c, 0, 16);
      xq[2 * c + 1] = __builtin_amdgcn_raw_buffer_load_b128(rq, qoff + 128 * c + 16, 0, 16);
    }
    const uint16_t* qrr = a.qin + (static_cast<int64_t>(b) * a.H + h) * (a.DH + DR) + a.DH + 8 * g;
#pragma unroll
    for (int c = 0; c < NR; ++c) qr[c] = *reinterpret_cast<const bf16x8_t*>(qrr + 32 * c);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int e = 0; e < 8; ++e) qh[c][e] = static_cast<_Float16>(xq[2 * c + (e >> 2)][e & 3]);
    }
  } else {
#pragma unroll
  for (int c = 0; c < NC + NR; ++c) {
    const float x[8] = {qraw[2 * c].x, qraw[2 * c].y, qraw[2 * c].z, qraw[2 * c].w,
                        qraw[2 * c + 1].x, qraw[2 * c + 1].y, qraw[2 * c + 1].z, qraw[2 * c + 1].w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (c < NC) qh[c][e] = static_cast<_Float16>(x[e]);
      else qr[c - NC][e] = static_cast<__bf16>(x[e]);
    }
  }
  }
  __syncthreads();

  const int nunits = (ntok + 15) / 16;  // every unit below nunits holds a kept token
  const int nu = nunits > w ? (nunits - w + NW - 1) / NW : 0;  // this wave's units

  f32x4_t o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY;  // reference maximum of head r16 (log2 domain), identical across g
  float l_run = 0.f;        // this lane's share of the sum relative to m_run

  if (nu > 0) {
    // loads of this wave's unit i from the list
    auto issue = [&](SliceRegs<NLI, NRI>& rg, int i) {
      issue_list_rows(rg, i, ntok);
      issue_gates(rg, i, ntok);
    };
    // the first D units: gate rows now that the ids are in LDS (and, with
    // slices, their cache rows too)
#pragma unroll
    for (int u = 0; u < D; ++u) {
      if constexpr (SL > 1) issue_list_rows(ring[u], u, ntok);
      issue_gates(ring[u], u, ntok);
      __builtin_amdgcn_sched_barrier(0);
    }

    uint16_t* tile = tile_all + w * 16 * TS;  // this wave's [16 tokens][TS]
    uint16_t* tread = tile + (4 * g + (r16 >> 2)) * TS + 4 * (r16 & 3);
    auto process = [&](SliceRegs<NLI, NRI>& rg, int i, bool refill) {
      const int nt = ntok - (w + i * NW) * 16;  // valid tokens of the unit (>= 1)
      // gate the latent (fp16); stage the unit row-major in this wave's tile
#pragma unroll
      for (int c = 0; c < NLI; ++c)
        *reinterpret_cast<u32x4_t*>(tile + (TPL * c + lt) * TS + lc) = gate_chunk_f16(rg.lat[c], rg.gat[c]);
#pragma unroll
      for (int c = 0; c < NRI; ++c) *reinterpret_cast<u32x4_t*>(tile + (TPR * c + rt) * TS + DC + rcol) = rg.rop[c];
      // this unit's registers are free: issue unit i + D into them
      if (refill) issue(rg, i + D);
      wave_lds_sync();
      // S^T[token 4g + q][head r16], two accumulator chains
      f32x4_t acc = {0.f, 0.f, 0.f, 0.f}, acc2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const f16x8_t av = *reinterpret_cast<const f16x8_t*>(tile + r16 * TS + c * 32 + g * 8);
        acc = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, qh[c], acc, 0, 0, 0);
      }
#pragma unroll
      for (int rc = 0; rc < NR; ++rc) {
        const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(tile + r16 * TS + DC + rc * 32 + g * 8);
        acc2 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, qr[rc], acc2, 0, 0, 0);
      }
      acc += acc2;

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
      const f16x4_t pb = __builtin_bit_cast(f16x4_t, u32x2_t{pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3])});

      // O^T[dim][head] += C~^T[dim][token] x P^T[token][head], 16 dims at a
      // time.  Lane r16 of group g reads dims 16 db + 4 (r16 % 4) .. + 3 of
      // token 4g + r16 / 4; the transposed read hands lane r16 of group g the
      // dim 16 db + r16 of tokens 4g .. 4g + 3.
#pragma unroll
      for (int db = 0; db < NB; ++db) {
        const s16x4_t at =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(tread + db * 16));
        o[db] = __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, at), pb, o[db], 0, 0, 0);
      }
      // every lane's reads of the tile are done before the next unit overwrites it
      wave_lds_sync();
    };

    // Full groups of D units (ring slot u holds units u, u + D, ...), then the
    // remaining nu % D units straight-line: one loop exit, and on every path
    // to it the same D units are in flight in the same order, so the
    // compiler's wait counters stay exact.
    const int nfull = nu / D;
    for (int i0 = 0; i0 < nfull * D; i0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        // keep units in source order: hoisting a later unit's work above this
        // point would make the wave wait for that unit's loads too
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

  // ---- phase 3: merge the waves' partial results; write the work item's partial ----
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);
  const int64_t pbase = ((static_cast<int64_t>(b) * a.s_max + s) * SL + k) * a.H + hg * 16;
  if (g == 0) mbuf[w * 16 + r16] = m_run;
  __syncthreads();  // also: every wave is done with the list and its tile (obuf aliases them)
  float M = -INFINITY;
#pragma unroll
  for (int v = 0; v < NW; ++v) M = fmaxf(M, mbuf[v * 16 + r16]);  // -inf only for a slice without tokens
  const float sc = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - M);
#pragma unroll
  for (int db = 0; db < NB; ++db) obuf[(w * NB + db) * 64 + lane] = o[db] * sc;
  if (g == 0) lbuf[w * 16 + r16] = l_run * sc;
  __syncthreads();
  // lane holds O^T[dim = 16 db + 4g + q][head r16]
  for (int db = w; db < NB; db += NW) {
    f32x4_t sum = obuf[db * 64 + lane];
#pragma unroll
    for (int v = 1; v < NW; ++v) sum += obuf[(v * NB + db) * 64 + lane];
    __builtin_nontemporal_store(sum, reinterpret_cast<f32x4_t*>(a.part_o + (pbase + r16) * DC + db * 16 + 4 * g));
  }
  if (w == 0 && g == 0) {
    float Ls = 0.f;
#pragma unroll
    for (int v = 0; v < NW; ++v) Ls += lbuf[v * 16 + r16];
    __builtin_nontemporal_store(M, a.part_ml + (pbase + r16) * 2 + 0);
    __builtin_nontemporal_store(Ls, a.part_ml + (pbase + r16) * 2 + 1);
  }
}

}  // namespace egmla
