// Wide split kernel of EG-MLA decode: latent dim 512, RoPE dim 64, bf16
// storage, heads in blocks of 64.  Included by decode.hip after SplitArgs.
//
// Work split.  One work-group of 4 waves (one per SIMD) per (token range, block
// of 64 heads); wave w holds heads 16 w .. 16 w + 15 of the block over all 576
// score dims and all 512 value dims, so no wave needs another wave's scores.
// The two head blocks of a 128-head layer run the same token range on the same
// XCD (blocks 8 apart), so the second fetch of a token's rows hits that XCD's
// L2 cache.
//
// Precision.  The absorbed query (fp32) is held as bf16 hi + lo, and each gated
// latent c * g (an exact fp32 product of two bf16 values, 16 significant bits)
// as bf16 hi + lo whose sum is the product exactly.  A score's latent part is
// hi.q_hi + hi.q_lo + lo.q_hi (the lo.lo product, below 2^-16 of the score, is
// left out), so a score carries fp32-level error even when the logits are
// large and the softmax is sharp; the RoPE part (bf16 x bf16) is exact.  The
// value product takes the gated latent's hi part and bf16 probabilities.
//
// Staging.  Tokens are taken 16 at a time (a slot); a ring of 4 slots holds two
// pairs of slots, one computed while the other's rows travel.  Cache rows and
// gate rows go from HBM straight into LDS with global_load_lds_dwordx4 (no
// registers): per token one 1024-byte latent DMA (into the slot's HI region),
// one 1024-byte gate DMA (into its LO region) and a 128-byte RoPE key.  Wave w
// fetches and then gates tokens 4 w .. 4 w + 3 of every slot in place: HI
// receives bf16(c g), LO the remainder.
//
// Scores.  S^T[token][head] of a slot on v_mfma_f32_16x16x32_bf16: the A
// operand (token lane % 16, 8 dims) is read from the slot, the B operand is
// the query (16 heads) held in registers: 3 latent products per 32-dim chunk
// on three accumulator chains, then the RoPE chunks.
//
// Softmax and values.  Per pair of slots the lane holds 8 scores of its head
// (4 tokens of each slot); online softmax in the log2 domain with a lazy
// rescale.  O^T[dim][head] += C~^T P^T on v_mfma_f32_16x16x32_bf16 with K = the
// pair's 32 tokens: each lane's own 8 probabilities are its B operand, and two
// ds_read_b64_tr_b16 (one per slot, the same 4 token rows) are its A operand,
// so the token order inside K is the same for both operands.
//
// Registers per wave: query hi + lo 128 (its RoPE chunks wait in LDS), value
// accumulators 128 (32 blocks of 16 dims x 16 heads), the score chain and the
// operands in flight: one wave per SIMD.  Each phase (gating, scores, values)
// reads its LDS operands at most two steps ahead of their use.
#pragma once

namespace egmla {

// LDS DMA of 16 bytes per lane from sbase + voff: lane l's bytes land at LDS
// byte address lds_base + 16 l (M0 holds lds_base; one wait state separates
// its write from the DMA).  The instruction is not visible to the compiler's
// wait counters: the caller waits for it with s_waitcnt vmcnt before reading
// the destination, and before the work-group exits.
// (No memory clobber: the DMA's LDS writes become visible only through
// wait_vmcnt, which is a compiler memory barrier, and the work-group barriers
// order every access to a ring slot before the DMA that refills it.)
__device__ __forceinline__ void lds_dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(lds_base), "v"(voff),
               "s"(sbase));
}

// The same with a full 64-bit address per lane (lanes of one instruction may
// read different rows); inactive lanes move nothing.
__device__ __forceinline__ void lds_dma16_addr(uint64_t addr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_base), "v"(addr));
}


// s_waitcnt with only the vector-memory counter constrained; also a compiler
// memory barrier, so that no LDS access moves across it.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier that orders LDS accesses but does not wait for
// outstanding global loads (the ring's DMA stays in flight across it).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

// Rows in a slot's HI and LO regions are stored with their 16-byte pieces
// permuted: logical piece p of slot row r sits at piece p ^ lat_swz(r)
// (lat_swz(r) < 16 takes 16 distinct values over r = 0..15).  The score read
// (16 rows, one piece each: 4-bank group (p ^ lat_swz(r)) mod 16) and the
// transposed value read (4 rows x one 32-byte pair each: pair index
// (p / 2) ^ (lat_swz(r) / 2) differs over each group of 4 rows) are then free
// of bank conflicts.
__device__ __forceinline__ int lat_swz(int r) { return ((0xCA60 >> (4 * (r & 3))) & 15) ^ (r >> 2); }

struct WideCfg {
  static constexpr int DC = 512, DR = 64, DQ = DC + DR;
  static constexpr int NW = 4, NT = NW * 64;
  static constexpr int HEADS = 64;        // heads per work-group
  static constexpr int TOK = 16;          // tokens per slot
  static constexpr int NS = 4;            // ring slots (two pairs)
  static constexpr int LROW = DC * 2;     // bytes per latent row in LDS (pieces swizzled, see lat_swz)
  static constexpr int HI = 0;                       // [16][LROW] latent, then bf16(c g)
  static constexpr int LO = HI + TOK * LROW;         // [16][LROW] gate row, then c g - bf16(c g)
  static constexpr int ROPE = LO + TOK * LROW;       // [16][128 B] RoPE keys, 16-byte pieces swizzled
  static constexpr int SLOT = ROPE + TOK * DR * 2;   // bytes per slot
  static constexpr int RING = NS * SLOT;
  static constexpr int LIST = RING;                  // int2 (slot, id) per token
  static constexpr int LISTCAP = 1024;               // tokens listed at a time (a multiple of 32)
  static constexpr int QROPE = LIST + LISTCAP * 8;   // [NW][2 chunks][64 lanes] bf16x8: RoPE query (B operand)
  static constexpr int LDS_BYTES = QROPE + NW * 2 * 64 * 16;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
  static_assert(SLOT % 16 == 0 && LIST % 16 == 0, "alignment");
};

// Balanced schedule of the wide kernel.  The batch's tokens, taken sequence
// after sequence, form one range of N = sum of the clamped lengths; range g of
// G_eff = min(G, N) takes positions [g N / G_eff, (g + 1) N / G_eff), which
// may span several sequences, so every range gets the same number of tokens
// (+-1) whatever the length mix.  Its part of sequence b is a segment with its
// own partial result, stored at partial row g + b: along the staircase of
// (range, sequence) pairs that have tokens, g + b grows by one at every step,
// so the rows are distinct (at most G_eff + B - 1 of them) and those of
// sequence b are consecutive.  One work-group of 1024 threads computes the
// prefix sums of the lengths and writes:
//   hdr[0] = N, hdr[1] = G_eff;
//   wg_start[g] = (sequence, offset) of position g N / G_eff;
//   seq_rows[b] = (first partial row, number of rows) of sequence b (0 rows
//                 for an empty sequence).
constexpr int kSchedThreads = 1024;

__global__ __launch_bounds__(kSchedThreads) void wide_schedule_kernel(const int32_t* __restrict__ seq_lens, int B,
                                                                      int cap, int G, int64_t* __restrict__ hdr,
                                                                      int2* __restrict__ wg_start,
                                                                      int2* __restrict__ seq_rows) {
  __shared__ int64_t wsum[kSchedThreads / 64];
  __shared__ int64_t carry_s;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  constexpr int NWV = kSchedThreads / 64;
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
  for (int base = 0; base < B; base += kSchedThreads) {
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
  for (int base = 0; base < B; base += kSchedThreads) {
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

__global__ __launch_bounds__(WideCfg::NT, 1) void split_wide_kernel(SplitArgs a) {
  using C = WideCfg;
  constexpr int DC = C::DC, DQ = C::DQ, LROW = C::LROW;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::LDS_BYTES];
  const int2* list = reinterpret_cast<const int2*>(lds + C::LIST);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));

  int wg, hblk;
  wide_block(blockIdx.x, a.groups, wg, hblk);
  const int64_t N = a.sched_hdr[0];
  const int Ge = static_cast<int>(a.sched_hdr[1]);
  if (wg >= Ge) return;  // uniform over the work-group
  int64_t remaining = (static_cast<int64_t>(wg) + 1) * N / Ge - static_cast<int64_t>(wg) * N / Ge;
  int b = a.wg_start[wg].x, off = a.wg_start[wg].y;

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int head0 = hblk * C::HEADS + 16 * w;  // first head of this wave

  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate);
  // latent / gate DMA of slot row 4w + k: lane l fetches logical piece l ^ lat_swz(4w + k)
  uint32_t dma_off[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) dma_off[k] = static_cast<uint32_t>(16 * (lane ^ lat_swz(4 * w + k)));
  // RoPE DMA (lanes 0..31): lane l fills 16-byte position l % 8 of slot row
  // 4w + l / 8 with logical piece (l % 8) ^ (row % 8)
  const int rope_row = 4 * w + ((lane >> 3) & 3);
  const uint32_t rope_src = static_cast<uint32_t>(2 * DC + 16 * ((lane & 7) ^ (rope_row & 7)));
  // gating: lane l takes physical piece l of this wave's rows
  const int off_gate = (4 * w) * LROW + 16 * lane;
  // scores: lane (token r16, group g) reads logical piece 4 c + g of slot row r16
  const int sa_x = g ^ lat_swz(r16);
  const int off_sa = r16 * LROW + 16 * (sa_x & 3);                               // + 64 (c ^ (sa_x >> 2))
  const int off_sr = C::ROPE + r16 * 128 + 16 * ((4 * 0 + g) ^ (r16 & 7));        // RoPE chunk 0
  const int off_sr1 = C::ROPE + r16 * 128 + 16 * ((4 * 1 + g) ^ (r16 & 7));       // RoPE chunk 1
  // values: lane r16 of group g reads dims 16 db + 4 (r16 % 4) .. + 3 of slot row
  // 4g + r16 / 4 (logical piece 2 db + (r16 % 4) / 2, half r16 % 2)
  const int tr_row = 4 * g + (r16 >> 2);
  const int tr_f = lat_swz(tr_row);
  const int tr_s = ((r16 & 3) >> 1) ^ (tr_f & 1);
  const int off_tr = tr_row * LROW + 16 * tr_s + 8 * (r16 & 1);                    // + 32 (db ^ (tr_f >> 1))
  const int tr_fh = tr_f >> 1;

  bf16x8_t qh[16], ql[16];  // B operands: head r16, dims 8g .. 8g + 7 of each 32-dim chunk
  bf16x8_t* qrope = reinterpret_cast<bf16x8_t*>(lds + C::QROPE) + w * 2 * 64 + lane;  // RoPE chunks c: [64 c]
  f32x4_t o[32];                   // O^T[dim 16 db + 4g + i][head r16]
  float m_run, l_run;              // head r16 (log2 domain); l: this lane's tokens

  while (remaining > 0 && b < a.B) {  // one segment: this range's part of sequence b
    const int L = clamp_len(a.seq_lens[b], a.cap);
    const int take = static_cast<int>(min(static_cast<int64_t>(L - off), remaining));
    if (take > 0) {
#pragma unroll
      for (int db = 0; db < 32; ++db) o[db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      m_run = -INFINITY;
      l_run = 0.f;
      // query of this lane's head for sequence b, as the absorption wrote it:
      // [q hi | q^R | q lo] in bf16
      {
        const uint16_t* qrow = reinterpret_cast<const uint16_t*>(a.qfull) +
                               (static_cast<int64_t>(b) * a.H + head0 + r16) * (DC + DQ) + 8 * g;
#pragma unroll
        for (int c = 0; c < 16; ++c) {
          qh[c] = *reinterpret_cast<const bf16x8_t*>(qrow + 32 * c);
          ql[c] = *reinterpret_cast<const bf16x8_t*>(qrow + DQ + 32 * c);
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) qrope[64 * c] = *reinterpret_cast<const bf16x8_t*>(qrow + DC + 32 * c);  // own region
      }
      for (int c0 = 0; c0 < take; c0 += C::LISTCAP) {
        const int t0 = off + c0;
        const int n = min(C::LISTCAP, take - c0);
        const int npairs = (n + 31) / 32;
        // ---- token list: (slot, id) of positions t0 .. t0 + 32 npairs - 1 (past
        // the segment the last token repeats; masked) ----
        {
          constexpr int PER = C::LISTCAP / C::NT;
          const int npad = npairs * 32;
          const int nper = (npad + C::NT - 1) / C::NT;  // uniform
          int pp[PER], psl[PER], pid[PER];
#pragma unroll
          for (int e = 0; e < PER; ++e) pp[e] = min(tid + e * C::NT, n - 1);
          split_slots(a, b, t0, pp, psl, nper);
#pragma unroll
          for (int e = 0; e < PER; ++e)
            if (e < nper) pid[e] = a.ids[psl[e]];
          int2* lw = reinterpret_cast<int2*>(lds + C::LIST);
#pragma unroll
          for (int e = 0; e < PER; ++e) {
            const int j = tid + e * C::NT;
            if (e < nper && j < npad) lw[j] = make_int2(psl[e], clamp_id(pid[e], a.V));
          }
        }
        __syncthreads();  // the list is complete; every wave is done with the previous chunk's slots

        // This wave's DMAs of pair p: tokens 4w .. 4w + 3 of slots 2p and 2p + 1,
        // per slot 4 latent rows, 4 gate rows and one RoPE instruction (18 in
        // all).  pair_entries reads the pair's list entries (wave-uniform, into
        // scalar registers); dma_step(j) issues instruction j, so that the issue
        // can be spread between the score products.  A pair index past the
        // chunk takes the last pair's entries (its rows land in ring slots that
        // are free, and are never read).
        int psl[8], pid[8];
        auto pair_entries = [&](int p) {
          const int pe = min(p, npairs - 1);
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const int4 e01 = reinterpret_cast<const int4*>(list)[(16 * (2 * pe + k) + 4 * w) / 2];
            const int4 e23 = reinterpret_cast<const int4*>(list)[(16 * (2 * pe + k) + 4 * w) / 2 + 1];
            psl[4 * k + 0] = __builtin_amdgcn_readfirstlane(e01.x);
            psl[4 * k + 1] = __builtin_amdgcn_readfirstlane(e01.z);
            psl[4 * k + 2] = __builtin_amdgcn_readfirstlane(e23.x);
            psl[4 * k + 3] = __builtin_amdgcn_readfirstlane(e23.z);
            pid[4 * k + 0] = __builtin_amdgcn_readfirstlane(e01.y);
            pid[4 * k + 1] = __builtin_amdgcn_readfirstlane(e01.w);
            pid[4 * k + 2] = __builtin_amdgcn_readfirstlane(e23.y);
            pid[4 * k + 3] = __builtin_amdgcn_readfirstlane(e23.w);
          }
        };
        auto dma_step = [&](int p, int j) {
          const int k = j / 9, i = j % 9;  // slot 2p + k of the ring, instruction i
          const uint32_t sb = lds0 + ((2 * p + k) % C::NS) * C::SLOT;
          if (i < 4) {
            lds_dma16(cache + static_cast<int64_t>(psl[4 * k + i]) * DQ, dma_off[i], sb + C::HI + (4 * w + i) * LROW);
          } else if (i < 8) {
            lds_dma16(gate + static_cast<int64_t>(pid[4 * k + i - 4]) * DC, dma_off[i - 4],
                      sb + C::LO + (4 * w + i - 4) * LROW);
          } else {
            // RoPE keys of the 4 rows: lane l < 32 reads row 4w + l / 8 (its own list entry)
            const int slk = list[16 * (2 * min(p, npairs - 1) + k) + rope_row].x;
            const uint64_t addr = reinterpret_cast<uint64_t>(cache + static_cast<int64_t>(slk) * DQ) + rope_src;
            if (lane < 32) lds_dma16_addr(addr, sb + C::ROPE + 4 * w * 128);
          }
        };

        // gate this wave's rows of pair p in place: HI <- bf16(c g), LO <- c g - HI
        // (per slot, the 8 reads of its 4 rows first, then the products)
        auto gate_pair = [&](int p) {
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            unsigned char* sp = lds + ((2 * p + k) % C::NS) * C::SLOT + off_gate;
            u32x4_t lat[4], gat[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              lat[r] = *reinterpret_cast<const u32x4_t*>(sp + C::HI + r * LROW);
              gat[r] = *reinterpret_cast<const u32x4_t*>(sp + C::LO + r * LROW);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              u32x4_t hi, lo;
              gate_chunk_hilo(lat[r], gat[r], hi, lo);
              *reinterpret_cast<u32x4_t*>(sp + C::HI + r * LROW) = hi;
              *reinterpret_cast<u32x4_t*>(sp + C::LO + r * LROW) = lo;
            }
            __builtin_amdgcn_sched_barrier(0);
          }
        };
        // S^T[token 4g + q][head r16] of the pair's two slots (unscaled), on
        // four accumulator chains (slot x query part) whose products alternate,
        // so no product waits for the one before it.  The operands of chunk
        // c + 1 are read while chunk c's products run, and nothing is hoisted
        // further (every chunk's reads would otherwise be live at once).  Two of
        // the next pair's DMAs go out with each of the first 9 chunks.
        auto scores = [&](int s0, f32x4_t& sa, f32x4_t& sb, int pn) {
          const unsigned char* spa = lds + (s0 % C::NS) * C::SLOT;
          const unsigned char* spb = lds + ((s0 + 1) % C::NS) * C::SLOT;
          f32x4_t a0 = {0.f, 0.f, 0.f, 0.f}, a1 = a0, b0 = a0, b1 = a0;
          bf16x8_t ah[2], al[2], bh[2], bl[2];
          auto rd = [&](int c) {
            const int pc = off_sa + 64 * (c ^ (sa_x >> 2));
            ah[c & 1] = *reinterpret_cast<const bf16x8_t*>(spa + C::HI + pc);
            al[c & 1] = *reinterpret_cast<const bf16x8_t*>(spa + C::LO + pc);
            bh[c & 1] = *reinterpret_cast<const bf16x8_t*>(spb + C::HI + pc);
            bl[c & 1] = *reinterpret_cast<const bf16x8_t*>(spb + C::LO + pc);
          };
          rd(0);
#pragma unroll
          for (int c = 0; c < 16; ++c) {
            if (c + 1 < 16) rd(c + 1);
            if (c < 9) {
              dma_step(pn, 2 * c);
              dma_step(pn, 2 * c + 1);
            }
            __builtin_amdgcn_sched_barrier(0);
            a0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[c & 1], qh[c], a0, 0, 0, 0);
            b0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[c & 1], qh[c], b0, 0, 0, 0);
            a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[c & 1], ql[c], a1, 0, 0, 0);
            b1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[c & 1], ql[c], b1, 0, 0, 0);
            a0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[c & 1], qh[c], a0, 0, 0, 0);
            b0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl[c & 1], qh[c], b0, 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
          }
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const int off = c ? off_sr1 : off_sr;
            const bf16x8_t ar = *reinterpret_cast<const bf16x8_t*>(spa + off);
            const bf16x8_t br = *reinterpret_cast<const bf16x8_t*>(spb + off);
            a1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ar, qrope[64 * c], a1, 0, 0, 0);
            b1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(br, qrope[64 * c], b1, 0, 0, 0);
          }
          sa = a0 + a1;
          sb = b0 + b1;
        };

        // Pair 0's DMAs go out now; pair p + 1's during the scores of pair p
        // (into the slots of pair p - 1, free once every wave has passed pair
        // p's barrier), so when iteration p starts, pair p's are the only loads
        // in flight.
        pair_entries(0);
#pragma unroll
        for (int j = 0; j < 18; ++j) dma_step(0, j);
        for (int p = 0; p < npairs; ++p) {
          wait_vmcnt<0>();
          gate_pair(p);
          lds_barrier();  // pair p gated and visible; every wave is done with pair p - 1
          pair_entries(p + 1);
          __builtin_amdgcn_sched_barrier(0);

          f32x4_t sa, sb;
          scores(2 * p, sa, sb, p + 1);
          float x[8];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            x[q] = sa[q] * a.scale_log2;
            x[4 + q] = sb[q] * a.scale_log2;
          }
          const int nt = n - 32 * p;  // valid tokens of the pair (1..32)
          if (nt < 32) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (4 * g + q >= nt) x[q] = -INFINITY;
              if (16 + 4 * g + q >= nt) x[4 + q] = -INFINITY;
            }
          }
          // online softmax of head r16 over the pair's 32 tokens
          float mt = x[0];
#pragma unroll
          for (int q = 1; q < 8; ++q) mt = fmaxf(mt, x[q]);
          mt = max_over_row_groups(mt);
          const float m_new = fmaxf(m_run, mt);  // finite: the pair has a valid token
          const bool grow = m_new > m_run + kLazyRescale;  // false while both are -inf
          if (__builtin_amdgcn_ballot_w64(grow)) {
            const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;  // exp2(-inf) = 0
            m_run = grow ? m_new : m_run;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < 32; ++db) o[db] *= alpha;
          }
          float pr[8];
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            pr[q] = __builtin_amdgcn_exp2f(x[q] - m_run);  // masked: exp2(-inf) = 0
            l_run += pr[q];
          }
          // B operand: k = 8g + i <-> slot 2p token 4g + i (i < 4), slot 2p + 1 token 4g + i - 4
          const bf16x8_t pb = __builtin_bit_cast(
              bf16x8_t, u32x4_t{pack_bf16x2(pr[0], pr[1]), pack_bf16x2(pr[2], pr[3]), pack_bf16x2(pr[4], pr[5]),
                                pack_bf16x2(pr[6], pr[7])});
          // O^T += C~^T P^T, A operand: dim 16 db + r16 of the same 8 tokens
          const unsigned char* sp0 = lds + ((2 * p) % C::NS) * C::SLOT + C::HI + off_tr;
          const unsigned char* sp1 = lds + ((2 * p + 1) % C::NS) * C::SLOT + C::HI + off_tr;
          // (the operands of block db + 3 are read while block db's product runs)
          s16x4_t v0[4], v1[4];
          auto rdv = [&](int db) {
            const int pd = 32 * (db ^ tr_fh);
            v0[db & 3] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(sp0 + pd));
            v1[db & 3] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(sp1 + pd));
          };
          rdv(0);
          rdv(1);
          rdv(2);
#pragma unroll
          for (int db = 0; db < 32; ++db) {
            if (db + 3 < 32) rdv(db + 3);
            __builtin_amdgcn_sched_barrier(0);
            const bf16x8_t av =
                __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(v0[db & 3], v1[db & 3], 0, 1, 2, 3, 4, 5, 6, 7));
            o[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, pb, o[db], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
        // the last pair's DMAs (issued past the chunk, never read) land before
        // the list is rebuilt or the work-group exits
        wait_vmcnt<0>();
      }
      // ---- partial result of this segment: this wave's 16 heads ----
      const int64_t pbase = (static_cast<int64_t>(wg) + b) * a.H + head0;
      const float l = sum_over_row_groups(l_run);
      if (g == 0) {
        __builtin_nontemporal_store(m_run, a.part_ml + (pbase + r16) * 2 + 0);
        __builtin_nontemporal_store(l, a.part_ml + (pbase + r16) * 2 + 1);
      }
      float* obase = a.part_o + (pbase + r16) * DC + 4 * g;
#pragma unroll
      for (int db = 0; db < 32; ++db)
        __builtin_nontemporal_store(o[db], reinterpret_cast<f32x4_t*>(obase + 16 * db));
    }
    remaining -= take > 0 ? take : 0;
    ++b;
    off = 0;
  }
}

}  // namespace egmla
