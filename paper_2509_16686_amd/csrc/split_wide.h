// Wide split kernel of EG-MLA decode: latent dim 512, RoPE dim 64, bf16
// storage, heads in blocks of 64.  Included by decode.hip after SplitArgs.
//
// Work split.  One work-group of 8 waves per (token range, block of 64
// heads), in two roles; wave w runs on SIMD w % 4, so every SIMD holds one
// wave of each role and the VALU and LDS work of one overlaps the matrix
// products of the other.
//   * Score wave s (w = s < 4) owns latent dims 128 s .. 128 s + 127 of every
//     token.  It loads its 256 bytes of a token's cache row and gate row in
//     whole 128-byte lines (one instruction: 4 tokens, 16 lanes each) and the
//     RoPE line of tokens 4g + s, gates the latent (fp16), writes both into
//     the unit's tiles in LDS (row = token), reads its A operands (token
//     lane % 16, 8 dims) back and computes the partial scores
//     S_s^T[token][head] of the 64 heads on v_mfma_f32_16x16x32_f16, the
//     absorbed query of its dims held in registers.  A chunk's loads for the
//     unit two ahead go out as soon as the chunk has been gated.
//   * Value wave t (w = 4 + t) owns head tile t (heads 16 t .. 16 t + 15) for
//     the softmax and latent dims 128 t .. 128 t + 127 of the output: it adds
//     the four partials of its head tile and the RoPE part (its own product
//     over the 64 RoPE dims, A operand from the RoPE tile), runs the online
//     softmax of its 16 heads (log2 domain, lazy rescale), and accumulates
//     O^T[dim][head] += C~^T P^T for its dims and all 64 heads over pairs of
//     units on v_mfma_f32_16x16x32_f16 (k-slots of lane group g: tokens
//     4g .. 4g + 3 of both units; A operands read with ds_read_b64_tr_b16
//     from the gated tiles).  It loads nothing from global memory in the unit
//     loop.
// Each role runs its own loop (so their registers do not add up) and both
// meet the same barriers, one per unit of 16 tokens: the partials and tiles
// of unit u are written before barrier u; between barriers u and u + 1 the
// value waves run the softmax of unit u and half of the value product of the
// last complete pair of units (dims 64 h .. 64 h + 63 of their 128, h = u % 2)
// in one basic block, so that the two interleave, while the score waves
// compute unit u + 1.  Partial scores are double-buffered, probabilities kept
// per pair (two pairs), rescale factors per unit (four), RoPE keys in two
// buffers and gated tiles in five (a tile lives five unit steps).  Loads in
// whole lines matter: a load-only copy of the kernel's access pattern with
// 16 rows x 64 bytes per instruction takes about twice as long.
//
// Precision.  The latent part of the scores and the values run on the fp16
// MFMA: the absorbed query is one rounding of its fp32 sum to fp16, each gated
// latent one rounding of the exact fp32 product c * g, each probability one
// rounding to fp16 (11-bit significands: rows dominated by a few keys stay
// within the element-wise bound, which bf16 operands would need hi + lo
// products for); where the second unit of a pair raised a head's maximum,
// the first unit's probabilities are scaled by that factor (below 2^-8) in
// fp16, a second rounding of terms at most 2^-8 of the new maximum.  The RoPE
// part (bf16 x bf16) is exact.  Magnitudes must stay below 65504.
//
// The two head blocks of a 128-head layer run the same token range on the same
// XCD (block ids 8 apart), so the second fetch of a token's rows hits that
// XCD's L2 cache.
#pragma once

namespace egmla {

// Work-group barrier that orders LDS accesses; outstanding global loads stay
// in flight across it (the workgroup-scope fences wait for LDS only).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

struct WideCfg {
  static constexpr int DC = 512, DR = 64, DQ = DC + DR;
  static constexpr int NV = 4;             // value waves (= score waves)
  static constexpr int NW = 2 * NV;        // waves per work-group
  static constexpr int NT = NW * 64;       // threads per work-group
  static constexpr int HEADS = 64;         // heads per work-group
  static constexpr int NHT = HEADS / 16;   // head tiles: one per value wave
  static constexpr int DW = DC / NV;       // latent dims of a score wave / output dims of a value wave
  static constexpr int NCH = DW / 32;      // 32-dim score chunks of a score wave
  static constexpr int NRC = DR / 32;      // 32-dim RoPE chunks (value waves)
  static constexpr int NDB = DW / 16;      // 16-dim value blocks of a value wave
  static constexpr int TOK = 16;           // tokens per unit
  static constexpr int NHB = 5;            // gated-tile buffers (a unit's tile lives 5 unit steps)
  static constexpr int NRB = 2;            // RoPE-key buffers
  // tile row: 512 gated dims + 32 bytes, so that the row stride is 8 banks
  // (mod 64): the 16-byte row writes and the transposed 8-byte reads of 4
  // rows are free of bank conflicts
  static constexpr int TS = DC + 16;
  // RoPE tile row: 64 dims + 16 bytes (36 banks mod 64): the 16 rows of an
  // operand read fall on 16 distinct groups of 4 banks
  static constexpr int RS = DR + 8;
  static constexpr int HT = 0;                                // [NHB][16][TS] fp16: gated latent
  static constexpr int RT = HT + NHB * TOK * TS * 2;          // [NRB][16][RS] bf16: RoPE keys
  static constexpr int SB = RT + NRB * TOK * RS * 2;          // [2][NV][NHT][64] f32x4: partial scores
  static constexpr int PB = SB + 2 * NV * NHT * 64 * 16;      // [2][NHT][64][2] fp16 x 4: probabilities of unit pairs
  static constexpr int AL = PB + 2 * NHT * 64 * 16;           // [4][16][NHT] f32: rescale factor of head 16 ht + r
  static constexpr int LB = AL + 4 * HEADS * 4;               // [16][NHT] f32: softmax sum of head 16 ht + r
  static constexpr int LIST = LB + HEADS * 4;                 // int2 (slot, id) per token
  static constexpr int LISTCAP = 3072;                        // tokens listed at a time
  static constexpr int LDS_BYTES = LIST + LISTCAP * 8;
  static_assert(NHT == NV && NHT == 4, "one head tile per value wave; 16-byte factor reads");
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
  static_assert(LISTCAP % NT == 0 && LISTCAP % TOK == 0, "list chunk");
  static_assert(RT % 16 == 0 && SB % 16 == 0 && PB % 16 == 0 && LB % 16 == 0 && LIST % 16 == 0, "alignment");
  static_assert(TOK == 4 * NV, "a score wave loads the RoPE lines of 4 tokens per unit");
};

// Balanced schedule of the wide kernel.  The batch's tokens, taken sequence
// after sequence, form one range of N = sum of the clamped lengths; range g of
// G_eff = min(G, N) takes positions [g N / G_eff, (g + 1) N / G_eff), which
// may span several sequences, so every range gets the same number of tokens
// (+-1) whatever the length mix.  Its part of sequence b is a segment with its
// own partial result, stored at partial row g + b: along the staircase of
// (range, sequence) pairs that have tokens, g + b grows by one at every step,
// so the rows are distinct (at most G_eff + B - 1 of them) and those of
// sequence b are consecutive.  One work-group of NT threads (an extra
// work-group of the absorption kernel, which runs just before the split
// kernel) computes the prefix sums of the lengths and writes:
//   hdr[0] = N, hdr[1] = G_eff;
//   wg_start[g] = (sequence, offset) of position g N / G_eff;
//   seq_rows[b] = (first partial row, number of rows) of sequence b (0 rows
//                 for an empty sequence).
struct WideSchedArgs {
  const int32_t* seq_lens;
  int cap, G;
  int64_t* hdr;
  int2* wg_start;
  int2* seq_rows;
};

template <int NT>
__device__ __forceinline__ void wide_schedule(const WideSchedArgs& sa, int B) {
  const int32_t* __restrict__ seq_lens = sa.seq_lens;
  const int cap = sa.cap, G = sa.G;
  int64_t* __restrict__ hdr = sa.hdr;
  int2* __restrict__ wg_start = sa.wg_start;
  int2* __restrict__ seq_rows = sa.seq_rows;
  __shared__ int64_t wsum[NT / 64];
  __shared__ int64_t carry_s;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  constexpr int NWV = NT / 64;
  // inclusive prefix over the work-group of one value per thread; returns the
  // exclusive prefix and leaves the total in `tot`
  auto block_scan = [&](int64_t v, int64_t& tot) {
    int64_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int64_t y = __shfl_up(x, o, 64);
      if (lane >= o) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int64_t before = 0;
    tot = 0;
    for (int k = 0; k < NWV; ++k) {
      if (k < w) before += wsum[k];
      tot += wsum[k];
    }
    __syncthreads();
    return before + x - v;
  };
  int64_t N = 0;
  for (int base = 0; base < B; base += NT) {
    const int b = base + tid;
    int64_t tot;
    block_scan(b < B ? clamp_len(seq_lens[b], cap) : 0, tot);
    N += tot;
  }
  const int Ge = static_cast<int>(N < G ? N : G);
  if (tid == 0) {
    hdr[0] = N;
    hdr[1] = Ge;
    carry_s = 0;
  }
  __syncthreads();
  for (int base = 0; base < B; base += NT) {
    const int b = base + tid;
    const int L = b < B ? clamp_len(seq_lens[b], cap) : 0;
    int64_t tot;
    const int64_t P = carry_s + block_scan(L, tot);  // tokens before sequence b
    if (b < B) {
      if (L > 0) {
        // range of position p: the largest g with g N / G_eff <= p
        const int g_first = static_cast<int>(((P + 1) * Ge - 1) / N);
        const int g_last = static_cast<int>(((P + L) * Ge - 1) / N);
        seq_rows[b] = make_int2(g_first + b, g_last - g_first + 1);
        // ranges whose first position lies in sequence b
        for (int g = static_cast<int>((P * Ge + N - 1) / N); g <= g_last; ++g)
          wg_start[g] = make_int2(b, static_cast<int>(static_cast<int64_t>(g) * N / Ge - P));
      } else {
        seq_rows[b] = make_int2(0, 0);
      }
    }
    __syncthreads();
    if (tid == 0) carry_s += tot;
    __syncthreads();
  }
}

// Work-group id -> (token range, head block): with `groups` head blocks and
// G ranges (G a multiple of 8), block ids 8 apart share an XCD, so the head
// blocks of range g are block ids 8 (groups (g / 8) + hb) + g % 8.
__device__ __forceinline__ void wide_block(int bid, int groups, int& range, int& hb) {
  const int xcd = bid & 7, j = bid >> 3;
  hb = j % groups;
  range = (j / groups) * 8 + xcd;
}

// Walks this work-group's segments (its range's part of one sequence each)
// and their list chunks: seg_begin(b) before the first chunk of sequence b's
// segment, chunk(n, nunits) once the chunk's token list (n tokens, padded to
// nunits units of 16 by repeating its last token) is in LDS, seg_end(b) after
// the last chunk.  Every wave runs the same walk (the quantities it branches
// on are uniform over the work-group).
template <typename SegBegin, typename Chunk, typename SegEnd>
__device__ __forceinline__ void wide_walk(const SplitArgs& a, int wg, int2* list, SegBegin seg_begin, Chunk chunk,
                                          SegEnd seg_end) {
  using C = WideCfg;
  const int64_t N = a.sched_hdr[0];
  const int Ge = static_cast<int>(a.sched_hdr[1]);
  int64_t remaining = (static_cast<int64_t>(wg) + 1) * N / Ge - static_cast<int64_t>(wg) * N / Ge;
  int b = a.wg_start[wg].x, off = a.wg_start[wg].y;
  const int tid = threadIdx.x;
  while (remaining > 0 && b < a.B) {
    const int L = clamp_len(a.seq_lens[b], a.cap);
    const int take = static_cast<int>(min(static_cast<int64_t>(L - off), remaining));
    if (take > 0) {
      seg_begin(b);
      for (int c0 = 0; c0 < take; c0 += C::LISTCAP) {
        const int t0 = off + c0;
        const int n = min(C::LISTCAP, take - c0);
        const int nunits = (n + C::TOK - 1) / C::TOK;
        {
          constexpr int PER = C::LISTCAP / C::NT;
          const int npad = nunits * C::TOK;
          const int nper = (npad + C::NT - 1) / C::NT;  // uniform
          int pp[PER], psl[PER], pid[PER];
#pragma unroll
          for (int e = 0; e < PER; ++e) pp[e] = min(tid + e * C::NT, n - 1);
          split_slots(a, b, t0, pp, psl, nper);
#pragma unroll
          for (int e = 0; e < PER; ++e)
            if (e < nper) pid[e] = a.ids[psl[e]];
#pragma unroll
          for (int e = 0; e < PER; ++e) {
            const int j = tid + e * C::NT;
            if (e < nper && j < npad) list[j] = make_int2(psl[e], clamp_id(pid[e], a.V));
          }
        }
        __syncthreads();  // the list is complete; every wave is done with the previous chunk
        chunk(n, nunits);
      }
      seg_end(b);
    }
    remaining -= take > 0 ? take : 0;
    ++b;
    off = 0;
  }
}

// Unit steps (barriers) of a list chunk of nunits units: one per unit, then
// the two halves of the values of the last pair of units (a lone last unit
// is a pair whose second unit has no tokens).
__device__ __forceinline__ int wide_steps(int nunits) { return 2 * ((nunits + 1) / 2) + 2; }

// One wave's work in the split kernel: ROLE 0 = score wave s, ROLE 1 = value
// wave t (the index is `idx`).  Every wave of the work-group walks the same
// segments and chunks and meets the same barriers: one per unit, one more at
// the end of each chunk.
template <int ROLE, int D>
__device__ __forceinline__ void wide_wave(const SplitArgs& a, unsigned char* lds, int wg, int hblk, int idx) {
  using C = WideCfg;
  constexpr int DC = C::DC, DQ = C::DQ, DW = C::DW, NHT = C::NHT, NV = C::NV, TS = C::TS, TOK = C::TOK;
  constexpr int NCH = C::NCH, NDB = C::NDB, NRC = C::NRC;
  constexpr int QROW = DQ;  // absorbed query row: [q_lat fp16 | q^R bf16]
  int2* list = reinterpret_cast<int2*>(lds + C::LIST);
  f32x4_t* sbuf = reinterpret_cast<f32x4_t*>(lds + C::SB);  // [2][NV][NHT][64]
  s16x4_t* pbuf = reinterpret_cast<s16x4_t*>(lds + C::PB);  // [2][NHT][64][2]: pair (u / 2) % 2, unit u % 2
  float* abuf = reinterpret_cast<float*>(lds + C::AL);      // [4][16][NHT]: unit u % 4
  float* lbuf = reinterpret_cast<float*>(lds + C::LB);      // [16][NHT]
  auto htile = [&](int h) { return reinterpret_cast<uint16_t*>(lds + C::HT) + h * TOK * TS; };
  auto rtile = [&](int u) { return reinterpret_cast<uint16_t*>(lds + C::RT) + (u % C::NRB) * TOK * C::RS; };

  const int lane = threadIdx.x & 63, r16 = lane & 15, g = lane >> 4;
  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate);
  const uint16_t* __restrict__ qfull = reinterpret_cast<const uint16_t*>(a.qfull);
  const int64_t qbase = static_cast<int64_t>(hblk) * C::HEADS + r16;  // + b H: query row of head r16 of tile 0
  const int dcol = DW * idx + 8 * g;  // score waves: this lane's first dim of chunk 0

  if constexpr (ROLE == 0) {
    // ======================= score wave s = idx =======================
    f16x8_t qh[NCH][NHT];  // B operands: head 16 ht + r16, dims 8g .. 8g + 7 of chunk c
    // Loads in whole 128-byte lines: instruction j brings the 256 bytes of
    // this wave's dims of token 4g + j (lane r16: dims 8 r16 .. 8 r16 + 7) of
    // the cache row and of the gate row, and one more instruction the RoPE
    // line of token 4g + s (lane r16: dims 4 r16 .. 4 r16 + 3).  Gated, they
    // go to the unit's tiles in the same layout; the score products read their
    // A operands (token r16, 8 dims) back from the tile.
    struct Unit {
      u32x4_t lat[4];
      u32x4_t gat[4];
      u32x2_t rop;
    };
    const int lcol = DW * idx + 8 * r16;  // this lane's dims in the cache and gate rows
    auto seg_begin = [&](int b) {
#pragma unroll
      for (int ht = 0; ht < NHT; ++ht) {
        const uint16_t* qrow = qfull + (static_cast<int64_t>(b) * a.H + qbase + 16 * ht) * QROW + dcol;
#pragma unroll
        for (int c = 0; c < NCH; ++c) qh[c][ht] = *reinterpret_cast<const f16x8_t*>(qrow + 32 * c);
      }
    };
    auto chunk = [&](int, int nunits) {
      // Rows of the unit being refilled (a unit past the chunk takes the last
      // unit's rows, never used, so that every step issues the same loads);
      // the list entries of tokens 4g .. 4g + 3 are read one unit ahead.
      int4 en0 = *reinterpret_cast<const int4*>(list + 4 * g);
      int4 en1 = *reinterpret_cast<const int4*>(list + 4 * g + 2);
      const uint16_t* crow[4];
      const uint16_t* grow[4];
      const uint16_t* rrow = nullptr;
      auto next_rows = [&](int u) {
        const int sl[4] = {en0.x, en0.z, en1.x, en1.z};
        const int id[4] = {en0.y, en0.w, en1.y, en1.w};
        const int nx = TOK * min(u + 1, nunits - 1) + 4 * g;
        en0 = *reinterpret_cast<const int4*>(list + nx);
        en1 = *reinterpret_cast<const int4*>(list + nx + 2);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          crow[j] = cache + static_cast<int64_t>(sl[j]) * DQ + lcol;
          grow[j] = gate + static_cast<int64_t>(id[j]) * DC + lcol;
        }
        const int rs = idx == 0 ? sl[0] : idx == 1 ? sl[1] : idx == 2 ? sl[2] : sl[3];  // token 4g + s
        rrow = cache + static_cast<int64_t>(rs) * DQ + DC + 4 * r16;
      };
      auto issue_chunk = [&](Unit& U, int j) {
        U.lat[j] = *reinterpret_cast<const u32x4_t*>(crow[j]);
        U.gat[j] = *reinterpret_cast<const u32x4_t*>(grow[j]);
      };
      auto issue_rope = [&](Unit& U) { U.rop = *reinterpret_cast<const u32x2_t*>(rrow); };
      auto step = [&](Unit& U, int u) {
        uint16_t* tw = htile(u % C::NHB);
        f32x4_t acc[NHT];
#pragma unroll
        for (int ht = 0; ht < NHT; ++ht) acc[ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        next_rows(u + D);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const u32x4_t gv = gate_chunk_f16(U.lat[j], U.gat[j]);
          issue_chunk(U, j);  // unit u + D into the registers just consumed
          *reinterpret_cast<u32x4_t*>(tw + (4 * g + j) * TS + lcol) = gv;
          __builtin_amdgcn_sched_barrier(0);  // the loads go out here, not after the products
        }
        *reinterpret_cast<u32x2_t*>(rtile(u) + (4 * g + idx) * C::RS + 4 * r16) = U.rop;
        issue_rope(U);
        __builtin_amdgcn_sched_barrier(0);
        // A operands: token r16, dims 8g .. 8g + 7 of chunk c (this wave's own writes)
        f16x8_t h[NCH];
#pragma unroll
        for (int c = 0; c < NCH; ++c) h[c] = *reinterpret_cast<const f16x8_t*>(tw + r16 * TS + dcol + 32 * c);
#pragma unroll
        for (int c = 0; c < NCH; ++c)
#pragma unroll
          for (int ht = 0; ht < NHT; ++ht)
            acc[ht] = __builtin_amdgcn_mfma_f32_16x16x32_f16(h[c], qh[c][ht], acc[ht], 0, 0, 0);
        const int k = u & 1;
#pragma unroll
        for (int ht = 0; ht < NHT; ++ht) sbuf[((k * NV + idx) * NHT + ht) * 64 + lane] = acc[ht];
        lds_barrier();  // barrier u: partials, gated tile and RoPE keys of unit u visible
      };
      Unit ring[D];
#pragma unroll
      for (int u = 0; u < D; ++u) {
        next_rows(u);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          issue_chunk(ring[u], j);
          __builtin_amdgcn_sched_barrier(0);  // the loop's issue order, so that its waits stay exact
        }
        issue_rope(ring[u]);
        __builtin_amdgcn_sched_barrier(0);
      }
      // Full groups of D units (ring slot u holds units u, u + D, ...), then
      // the remaining nunits % D straight-line, so that on every path the
      // same units are in flight in the same order.
      const int nfull = nunits / D;
      for (int i0 = 0; i0 < nfull * D; i0 += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
          __builtin_amdgcn_sched_barrier(0);
          step(ring[u], i0 + u);
        }
      }
#pragma unroll
      for (int u = 0; u < D - 1; ++u) {
        __builtin_amdgcn_sched_barrier(0);
        if (nfull * D + u < nunits) step(ring[u], nfull * D + u);
      }
      // the value waves' steps past the last unit (their last values)
      for (int u = nunits; u < wide_steps(nunits); ++u) lds_barrier();
    };
    wide_walk(a, wg, list, seg_begin, chunk, [](int) {});
  } else {
    // ======================= value wave t = idx =======================
    bf16x8_t qr[NRC];                      // RoPE B operands: head 16 t + r16, dims 8g .. 8g + 7 of chunk c
    f32x4_t o[NDB][NHT];                   // O^T[dim 128 t + 16 db + 4g + i][head 16 ht + r16]
    float m_run = -INFINITY, l_run = 0.f;  // head 16 t + r16 (log2 domain); l: this lane's tokens
    auto seg_begin = [&](int b) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int ht = 0; ht < NHT; ++ht) o[db][ht] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      m_run = -INFINITY;
      l_run = 0.f;
      const uint16_t* qrow = qfull + (static_cast<int64_t>(b) * a.H + qbase + 16 * idx) * QROW + DC + 8 * g;
#pragma unroll
      for (int c = 0; c < NRC; ++c) qr[c] = *reinterpret_cast<const bf16x8_t*>(qrow + 32 * c);
    };
    auto chunk = [&](int n, int nunits) {
      // Values: O^T += C~^T P^T for the units ua (even) and ua + 1 (if
      // `pair`), their probabilities written before the last barrier, on the
      // K = 32 product: lane group g's 8 k-slots are tokens 4g .. 4g + 3 of
      // unit ua, then the same tokens of unit ua + 1 (a lone unit: zero
      // probabilities for the second half, its own tile read twice).
      // prep_reads reads the probabilities and the rescale factors,
      // prep_apply scales unit ua's probabilities by unit ub's factor and the
      // sums by both (a branch per head tile in which a head's maximum grew:
      // rare).
      auto prep_reads = [&](int ua, bool pair, f16x8_t (&pb)[NHT], float4& aa, float4& ab) {
        const int ub = pair ? ua + 1 : ua;
        aa = *reinterpret_cast<const float4*>(abuf + ((ua & 3) * 16 + r16) * NHT);
        ab = *reinterpret_cast<const float4*>(abuf + ((ub & 3) * 16 + r16) * NHT);
        const int pr = (ua >> 1) & 1;
#pragma unroll
        for (int ht = 0; ht < NHT; ++ht)
          pb[ht] = *reinterpret_cast<const f16x8_t*>(pbuf + ((pr * NHT + ht) * 64 + lane) * 2);
      };
      auto prep_apply = [&](bool pair, f16x8_t (&pb)[NHT], const float4& aa, const float4& ab) {
        const float aas[NHT] = {aa.x, aa.y, aa.z, aa.w};
        const float abs_[NHT] = {ab.x, ab.y, ab.z, ab.w};
        if (!pair) {
#pragma unroll
          for (int ht = 0; ht < NHT; ++ht)
#pragma unroll
            for (int e = 4; e < 8; ++e) pb[ht][e] = static_cast<_Float16>(0.f);
        }
#pragma unroll
        for (int ht = 0; ht < NHT; ++ht) {
          const float fbh = pair ? abs_[ht] : 1.f;
          if (__builtin_amdgcn_ballot_w64(fbh != 1.f)) {
            const _Float16 sb = static_cast<_Float16>(fbh);
#pragma unroll
            for (int e = 0; e < 4; ++e) pb[ht][e] *= sb;
          }
          const float f = aas[ht] * fbh;
          if (__builtin_amdgcn_ballot_w64(f != 1.f)) {
#pragma unroll
            for (int db = 0; db < NDB; ++db) o[db][ht] *= f;
          }
        }
      };
      // lane r16 of group g reads dims 16 db + 4 (r16 % 4) .. + 3 of token
      // 4g + r16 / 4; the transposed read hands it dim 16 db + r16 of tokens 4g .. 4g + 3
      const int toff = (4 * g + (r16 >> 2)) * TS + DW * idx + 4 * (r16 & 3);
      auto vals_reads = [&](int ua, bool pair, int d0, s16x4_t (&ta)[4], s16x4_t (&tb)[4]) {
        const uint16_t* tra = htile(ua % C::NHB) + toff;
        const uint16_t* trb = htile((pair ? ua + 1 : ua) % C::NHB) + toff;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          ta[d] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(tra + 16 * (d0 + d)));
          tb[d] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(trb + 16 * (d0 + d)));
        }
      };
      auto vals_mfma = [&](int d0, const s16x4_t (&ta)[4], const s16x4_t (&tb)[4], const f16x8_t (&pb)[NHT]) {
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const f16x8_t av =
              __builtin_bit_cast(f16x8_t, __builtin_shufflevector(ta[d], tb[d], 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int ht = 0; ht < NHT; ++ht)
            o[d0 + d][ht] = __builtin_amdgcn_mfma_f32_16x16x32_f16(av, pb[ht], o[d0 + d][ht], 0, 0, 0);
        }
      };
      // Softmax of head tile t over unit u: the RoPE part of the scores (A
      // operand: token r16, dims 8g .. 8g + 7 of chunk c) and this head
      // tile's four partials are read by soft_reads; soft_math is free of
      // branches, so that its VALU work interleaves with the value products.
      auto soft_reads = [&](int u, bf16x8_t (&ra)[NRC], f32x4_t (&sv)[NV]) {
        const uint16_t* rr = rtile(u) + r16 * C::RS + 8 * g;
#pragma unroll
        for (int c = 0; c < NRC; ++c) ra[c] = *reinterpret_cast<const bf16x8_t*>(rr + 32 * c);
#pragma unroll
        for (int v = 0; v < NV; ++v) sv[v] = sbuf[(((u & 1) * NV + v) * NHT + idx) * 64 + lane];
      };
      auto soft_math = [&](int u, const bf16x8_t (&ra)[NRC], const f32x4_t (&sv)[NV]) {
        f32x4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NRC; ++c) sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ra[c], qr[c], sc, 0, 0, 0);
        sc += (sv[0] + sv[1]) + (sv[2] + sv[3]);
        const int nt = n - TOK * u;  // valid tokens of the unit (>= 1)
        float x[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) x[q] = 4 * g + q < nt ? sc[q] * a.scale_log2 : -INFINITY;
        const float mt = max_over_row_groups(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
        const float m_new = fmaxf(m_run, mt);  // finite: the unit has a valid token
        const bool grow = m_new > m_run + kLazyRescale;  // false while both are -inf
        const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;  // exp2(-inf) = 0
        m_run = grow ? m_new : m_run;
        l_run *= alpha;
        float p[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          p[q] = __builtin_amdgcn_exp2f(x[q] - m_run);  // masked: exp2(-inf) = 0
          l_run += p[q];
        }
        // B operand of the value product: k = token 4g + i of the unit's half,
        // j = head r16; the factor of head r16 (the four lanes of a head
        // write the same value)
        pbuf[((((u >> 1) & 1) * NHT + idx) * 64 + lane) * 2 + (u & 1)] =
            __builtin_bit_cast(s16x4_t, u32x2_t{pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3])});
        abuf[((u & 3) * 16 + r16) * NHT + idx] = alpha;
      };
      // After barrier u: the softmax of unit u (past the last unit every
      // token is masked, which leaves the running maximum and sum as they
      // are) and half h = u % 2 of the values of the pair of units k2, k2 + 1
      // (k2 = 2 (u / 2) - 2): dims 64 h .. 64 h + 63 of this wave's 128,
      // interleaved with the softmax.  The steps go in pairs, straight-line,
      // so that each accumulator has one product site and stays in place; in
      // the first pair of steps no pair of units is complete, and the
      // products add zero (probabilities zero, unit 0's tile read).
      // pb: the probabilities of the pair, read on the first step of the two
      auto step = [&](int u, int d0, f16x8_t (&pb)[NHT]) {
        lds_barrier();  // barrier u
        const bool live = u >= 2;
        const int k2 = live ? (u & ~1) - 2 : 0;
        const bool pair = live && k2 + 1 < nunits;
        // every LDS read of the step first (one round trip), then the
        // branches of the rescale, then the products and the softmax
        float4 aa, ab;
        if (d0 == 0) prep_reads(k2, pair, pb, aa, ab);
        bf16x8_t ra[NRC];
        f32x4_t sv[NV];
        s16x4_t ta[4], tb[4];
        soft_reads(u, ra, sv);
        vals_reads(k2, pair, d0, ta, tb);
        if (d0 == 0) {
          if (live) {
            prep_apply(pair, pb, aa, ab);
          } else {
#pragma unroll
            for (int ht = 0; ht < NHT; ++ht)
#pragma unroll
              for (int e = 0; e < 8; ++e) pb[ht][e] = static_cast<_Float16>(0.f);
          }
        }
        vals_mfma(d0, ta, tb, pb);
        soft_math(u, ra, sv);
        // the softmax sums of this head tile (final: the last unit's softmax
        // ran at step nunits - 1), for the normalised partial rows written
        // after the last barrier
        if (u == wide_steps(nunits) - 2) {
          const float lt = sum_over_row_groups(l_run);
          if (g == 0) lbuf[r16 * NHT + idx] = lt;
        }
      };
      for (int u = 0; u < wide_steps(nunits); u += 2) {
        f16x8_t pb[NHT];
        step(u, 0, pb);
        step(u + 1, 4, pb);
      }
    };
    // The segment's partial: each row O / l in fp16 (the sums of all four head
    // tiles were written to LDS before the last barrier) and, for this head
    // tile, (m, l) in fp32.
    auto seg_end = [&](int b) {
      const int64_t pbase = (static_cast<int64_t>(wg) + b) * a.H + hblk * C::HEADS;
      const float4 lt = *reinterpret_cast<const float4*>(lbuf + r16 * NHT);
      const float lts[NHT] = {lt.x, lt.y, lt.z, lt.w};
      uint16_t* part = reinterpret_cast<uint16_t*>(a.part_o);
#pragma unroll
      for (int ht = 0; ht < NHT; ++ht) {
        const float inv = 1.f / lts[ht];  // >= 1: the maximum's own term
        uint16_t* orow = part + (pbase + 16 * ht + r16) * DC + DW * idx + 4 * g;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const f32x4_t v = o[db][ht];
          const u32x2_t h = {pack_f16x2(v[0] * inv, v[1] * inv), pack_f16x2(v[2] * inv, v[3] * inv)};
          __builtin_nontemporal_store(h, reinterpret_cast<u32x2_t*>(orow + 16 * db));
        }
      }
      if (g == 0) {
        __builtin_nontemporal_store(m_run, a.part_ml + (pbase + 16 * idx + r16) * 2 + 0);
        __builtin_nontemporal_store(lts[idx], a.part_ml + (pbase + 16 * idx + r16) * 2 + 1);
      }
    };
    wide_walk(a, wg, list, seg_begin, chunk, seg_end);
  }
}

// D: units of 16 tokens in flight per score wave (34 VGPRs of rows each; the
// value waves load nothing from global memory inside the unit loop).
template <int D>
__global__ __launch_bounds__(WideCfg::NT, 1) void split_wide_kernel(SplitArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[WideCfg::LDS_BYTES];
  int wg, hblk;
  wide_block(blockIdx.x, a.groups, wg, hblk);
  if (wg >= static_cast<int>(a.sched_hdr[1])) return;  // uniform over the work-group
  const int w = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  if (w < WideCfg::NV)
    wide_wave<0, D>(a, lds, wg, hblk, w);
  else
    wide_wave<1, D>(a, lds, wg, hblk, w - WideCfg::NV);
}

}  // namespace egmla
