// Wide split kernel of EG-MLA decode: 128 heads per work-group, latent dim
// 512, RoPE dim 64, bf16 storage.  Included by decode.hip after SplitArgs.
//
// One work-group of 8 waves (two per SIMD) per (sequence b, context split s,
// block of 128 heads).  Wave w = 2 hg + dh pairs a head group hg (32 heads) with
// a dimension half dh (latent dims 256 dh .. + 255 and RoPE dims 32 dh .. + 31,
// 288 of the 576 score dims).  The split's tokens are taken 16 at a time (a
// tile).
//
// Staging.  Cache rows and gate rows go from HBM straight into LDS with
// global_load_lds_dwordx4 (no registers): a ring of 3 tile slots, two tiles in
// flight ahead of the one being computed.  Wave w fetches tokens 2w and 2w + 1
// of every tile: per token one instruction for the 1024-byte latent row, one
// for the 1024-byte gate row and one (8 lanes) for the 128-byte RoPE key.
// It then gates those 2 tokens in place (exact fp32 product, one bf16
// rounding), so the tile holds [token][gated latent] and [token][RoPE key].
//
// Scores.  Wave (hg, dh) computes the partial S^T[token][head] of its 32 heads
// over its 288 dims with v_mfma_f32_16x16x32_bf16: the A operand (token lane%16,
// 8 dims) read from the tile, the B operand the absorbed query (written in
// bf16 by the absorption) held in registers (64 per lane; its RoPE chunk in
// LDS).  The two waves of a head group
// exchange their partial sums through LDS; both add them in the same order, so
// both hold the same scores and run the same online softmax (log2 domain,
// lazy rescale).  The exchange synchronises only the two waves of the pair
// (a flag in LDS), so pairs drift apart and one pair's softmax overlaps
// another pair's score products on the same SIMDs.
//
// Values.  Wave (hg, dh) accumulates O^T[dim][head] for its 32 heads and its
// 256 latent dims on v_mfma_f32_32x32x16_bf16 (128 accumulators per lane).  The
// A operand is two ds_read_b64_tr_b16 of the gated latent (16-lane transposes:
// one dim, 4 tokens each); the B operand is the probabilities, moved from the
// score accumulator layout into the operand layout with v_permlane16_swap.
//
// Registers: 128 accumulators + 64 query + the tile's temporaries fit the 256
// of a wave at two waves per SIMD in one register file.
//
// LDS traffic per tile (bytes): tile data 35 K written by the DMA, gating 32 K
// read and 16 K written, scores 74 K read, exchange 16 K written and read,
// values 64 K read.
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

typedef __attribute__((ext_vector_type(16))) float f32x16_t;

// Latent rows in LDS are stored with their 16-byte pieces permuted: logical
// piece p of tile row r sits at piece p ^ lat_swz(r).  The permutation keeps
// both MFMA operand reads free of bank conflicts (32 or 64 banks): the score
// read (16 rows, one piece each) hits 16 distinct 4-bank groups, and the
// transposed value read (4 rows x 32 bytes per 16 lanes) 4 distinct pairs.
__device__ __forceinline__ int lat_swz(int r) { return ((0xCA60 >> (4 * (r & 3))) & 15) ^ (r >> 2); }

struct WideCfg {
  static constexpr int DC = 512, DR = 64, DQ = DC + DR;
  static constexpr int NW = 8, NT = NW * 64;
  static constexpr int HEADS = 128;       // heads per work-group
  static constexpr int NS = 3;            // ring slots
  static constexpr int LROW = DC * 2;       // bytes per latent row in LDS (pieces swizzled, see lat_swz)
  static constexpr int LAT = 0;                       // [16][LROW]   latent, gated in place
  static constexpr int ROPE = LAT + 16 * LROW;        // [16][128 B]  RoPE keys, 16-byte pieces swizzled
  static constexpr int GATE = ROPE + 16 * DR * 2;     // [16][1024 B] gate rows
  static constexpr int SLOT = GATE + 16 * DC * 2;     // bytes per slot
  static constexpr int RING = NS * SLOT;
  static constexpr int LIST = RING;                               // int2 (slot, id) per token
  static constexpr int XBUF = LIST + kMaxSplitTokensDevice * 8;   // [NW][2][64] f32x4 partial scores
  static constexpr int QROPE = XBUF + NW * 2 * 64 * 16;           // [NW][2][64] bf16x8 RoPE query (B operand)
  static constexpr int FLAGS = QROPE + NW * 2 * 64 * 16;          // [NW] int: exchanges published per wave
  static constexpr int LDS_BYTES = FLAGS + NW * 4;
  static constexpr int SPIN_LIMIT = 1 << 16;  // polls of a partner's flag before giving up (never reached)
  static constexpr int DMA_PER_TILE = 6;  // per wave: 2 latent, 2 gate, 2 RoPE
  static_assert(LDS_BYTES <= 160 * 1024, "LDS budget");
  static_assert(SLOT % 16 == 0 && LIST % 16 == 0 && XBUF % 16 == 0 && QROPE % 16 == 0, "alignment");
};

// Balanced schedule of the wide kernel.  The batch's tokens, taken sequence
// after sequence, form one range of N = sum of the clamped lengths; work-group
// g of G_eff = min(G, N) takes positions [g N / G_eff, (g + 1) N / G_eff), which
// may span several sequences, so every work-group gets the same number of
// tokens (+-1) whatever the length mix.  Its part of sequence b is a segment
// with its own partial result, stored at partial row g + b: along the
// staircase of (work-group, sequence) pairs that have tokens, g + b grows by one
// at every step, so the rows are distinct (at most G_eff + B - 1 of them) and
// those of sequence b are consecutive.  One work-group of 1024 threads computes
// the prefix sums of the lengths and writes:
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
        // work-group of position p: the largest g with g N / G_eff <= p
        const int g_first = static_cast<int>(((P + 1) * Ge - 1) / N);
        const int g_last = static_cast<int>(((P + L) * Ge - 1) / N);
        seq_rows[b] = make_int2(g_first + b, g_last - g_first + 1);
        // work-groups whose first position lies in sequence b
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

__global__ __launch_bounds__(WideCfg::NT, 1) void split_wide_kernel(SplitArgs a) {
  using C = WideCfg;
  constexpr int DC = C::DC, DQ = C::DQ, NS = C::NS, LROW = C::LROW;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::LDS_BYTES];
  int2* list = reinterpret_cast<int2*>(lds + C::LIST);
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));

  const int hb128 = blockIdx.x % a.groups;
  const int wg = blockIdx.x / a.groups;
  const int64_t N = a.sched_hdr[0];
  const int Ge = static_cast<int>(a.sched_hdr[1]);
  if (wg >= Ge) return;  // uniform over the work-group
  int64_t remaining = (static_cast<int64_t>(wg) + 1) * N / Ge - static_cast<int64_t>(wg) * N / Ge;
  int b = a.wg_start[wg].x, off = a.wg_start[wg].y;

  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int hg = w >> 1, dh = w & 1;
  const int head0 = hb128 * C::HEADS + hg * 32;  // first head of this wave's head group
  const int chunk = a.split;                     // list capacity per rebuild (<= kMaxSplitTokensDevice)

  const uint16_t* __restrict__ cache = static_cast<const uint16_t*>(a.cache);
  const uint16_t* __restrict__ gate = static_cast<const uint16_t*>(a.gate);
  // RoPE keys of tokens 2w and 2w + 1: lane l < 16 fills 16-byte position
  // l % 8 of token 2w + l / 8 with piece (l % 8) ^ (token % 8), one DMA per
  // token (lanes 0-7, then lanes 8-15)
  const uint32_t rope_off = 2 * DC + 16 * ((lane & 7) ^ ((2 * w + ((lane >> 3) & 1)) & 7));
  // latent / gate DMA of token 2w + k: lane l fetches logical piece l ^ lat_swz(2w + k)
  const uint32_t lane16s[2] = {static_cast<uint32_t>(16 * (lane ^ lat_swz(2 * w))),
                               static_cast<uint32_t>(16 * (lane ^ lat_swz(2 * w + 1)))};
  // Loop-invariant per-lane byte offsets inside a slot.
  const int off_gl = C::LAT + 2 * w * LROW + 16 * lane;       // gating: latent piece of token 2w
  const int off_gg = C::GATE + 2 * w * DC * 2 + 16 * lane;    // gating: gate piece of token 2w
  // values: lane r16 of 16-lane group R reads 4 dims (8 bytes) of token
  // 8 (R / 2) + 4 j + r16 / 4 and receives dim 16 (R % 2) + r16 of tokens
  // 8 (R / 2) + 4 j .. + 3; logical piece 32 dh + 4 db + tr_s of that row
  const int tr_row0 = 8 * (lane >> 5) + (r16 >> 2);
  const int tr_s = 2 * ((lane >> 4) & 1) + ((r16 & 3) >> 1);
  const int tr_f[2] = {lat_swz(tr_row0), lat_swz(tr_row0 + 4)};
  const int off_tr = C::LAT + tr_row0 * LROW + 512 * dh + 8 * (r16 & 1);
  // scores: lane (token r16, g) reads logical piece 32 dh + 4 c + g
  const int sa_x = g ^ lat_swz(r16);
  const int off_sa = C::LAT + r16 * LROW + 512 * dh + 16 * (sa_x & 3);
  const int off_sr = C::ROPE + r16 * 128 + 16 * ((4 * dh + g) ^ (r16 & 7));    // scores: RoPE A operand
  f32x4_t* xbuf = reinterpret_cast<f32x4_t*>(lds + C::XBUF);
  int* flags = reinterpret_cast<int*>(lds + C::FLAGS);
  if (lane == 0) flags[w] = 0;  // ordered before any poll by the first list barrier
  int exchanges = 0;            // this wave's published exchanges (the same count in every wave)

  bf16x8_t qb[2][8];  // B operand: head 16 hb + r16, dims 8g .. 8g + 7 of latent chunk c
  bf16x8_t* qrope = reinterpret_cast<bf16x8_t*>(lds + C::QROPE) + w * 2 * 64 + lane;  // RoPE chunk, [hb * 64]
  f32x16_t o[8];      // O^T[dim 256 dh + 32 db + row][head lane % 32]
  float m_run[2], l_run[2];  // head 16 hb + r16 (log2 domain); l: this lane's 4 tokens of each tile
  bf16x8_t pb;  // B operand of the value product: head lane % 32, tokens 8 (lane / 32) .. + 7

  // gate this wave's 2 tokens of the tile at slot byte offset sbase (in place)
  auto gate_tile = [&](int sbase) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      u32x4_t* lp = reinterpret_cast<u32x4_t*>(lds + sbase + off_gl + k * LROW);
      const u32x4_t gv = *reinterpret_cast<const u32x4_t*>(lds + sbase + off_gg + k * DC * 2);
      *lp = gate_chunk(*lp, gv);
    }
  };
  // O^T += C~^T P^T over the 16 tokens of the tile at slot byte offset sbase
  auto values = [&](int sbase) {
    const unsigned char* tp = lds + sbase + off_tr;
#pragma unroll
    for (int db = 0; db < 8; ++db) {
      // physical piece (4 db + tr_s) ^ f = 4 (db ^ (f >> 2)) + (tr_s ^ (f & 3))
      const int p0 = 4 * (db ^ (tr_f[0] >> 2)) + (tr_s ^ (tr_f[0] & 3));
      const int p1 = 4 * (db ^ (tr_f[1] >> 2)) + (tr_s ^ (tr_f[1] & 3));
      const s16x4_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(tp + 16 * p0));
      const s16x4_t a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
          (__attribute__((address_space(3))) s16x4_t*)(tp + 4 * LROW + 16 * p1));
      const bf16x8_t av = __builtin_bit_cast(
          bf16x8_t, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, pb, o[db], 0, 0, 0);
    }
  };

  while (remaining > 0 && b < a.B) {  // one segment: this work-group's part of sequence b
    const int L = clamp_len(a.seq_lens[b], a.cap);
    const int take = static_cast<int>(min(static_cast<int64_t>(L - off), remaining));
    if (take > 0) {
#pragma unroll
      for (int db = 0; db < 8; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        m_run[hb] = -INFINITY;
        l_run[hb] = 0.f;
      }
      // query of this lane for sequence b (bf16, as the absorption wrote it)
      {
        const uint16_t* q16 = reinterpret_cast<const uint16_t*>(a.qfull);
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
          const uint16_t* qrow = q16 + (static_cast<int64_t>(b) * a.H + head0 + hb * 16 + r16) * DQ;
#pragma unroll
          for (int c = 0; c < 8; ++c) qb[hb][c] = *reinterpret_cast<const bf16x8_t*>(qrow + 256 * dh + 32 * c + 8 * g);
          qrope[hb * 64] = *reinterpret_cast<const bf16x8_t*>(qrow + DC + 32 * dh + 8 * g);  // this wave's LDS region
        }
      }
      for (int c0 = 0; c0 < take; c0 += chunk) {
        const int t0 = off + c0;
        const int n = min(chunk, take - c0);
        const int ntiles = (n + 15) / 16;
        // ---- token list: (slot, id) of positions t0 .. t0 + 16 ntiles - 1 (past
        // the segment the last token repeats; masked) ----
        {
          constexpr int PER = kMaxSplitTokensDevice / C::NT;
          const int npad = ntiles * 16;
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
        __syncthreads();  // the list is complete; every wave is done with the previous chunk's tiles

        // DMA of tile i given its list entries for this wave's tokens 2w, 2w + 1
        // ((slot, id) each; one 16-byte LDS read per tile)
        auto entries = [&](int i) { return reinterpret_cast<const int4*>(list)[i * 8 + w]; };
        auto issue_tile = [&](int i, int4 e) {
          const uint32_t slot = lds0 + (i % NS) * C::SLOT;
          const int sl[2] = {__builtin_amdgcn_readfirstlane(e.x), __builtin_amdgcn_readfirstlane(e.z)};
          const int id[2] = {__builtin_amdgcn_readfirstlane(e.y), __builtin_amdgcn_readfirstlane(e.w)};
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            lds_dma16(cache + static_cast<int64_t>(sl[k]) * DQ, lane16s[k], slot + C::LAT + (2 * w + k) * LROW);
            lds_dma16(gate + static_cast<int64_t>(id[k]) * DC, lane16s[k], slot + C::GATE + (2 * w + k) * DC * 2);
          }
#pragma unroll
          for (int k = 0; k < 2; ++k)
            if ((lane >> 3) == k) lds_dma16(cache + static_cast<int64_t>(sl[k]) * DQ, rope_off, slot + C::ROPE + 2 * w * 128);
        };

        issue_tile(0, entries(0));
        if (ntiles > 1) issue_tile(1, entries(1));
        int4 next_e = entries(min(2, ntiles - 1));  // list entries of tile t + 2
        // this wave's tokens of tile 0 (that of tile 1 may be in flight)
        if (ntiles > 1) wait_vmcnt<C::DMA_PER_TILE>();
        else wait_vmcnt<0>();
        gate_tile(0);

        // Tile t: scores, exchange, softmax and values of tile t, with the
        // gating of tile t + 1 overlapping the softmax.
        for (int t = 0; t < ntiles; ++t) {
          const int sbase = __builtin_amdgcn_readfirstlane((t % NS) * C::SLOT);
          lds_barrier();  // tile t gated and visible; every wave is done with tile t - 1
          if (t + 2 < ntiles) issue_tile(t + 2, next_e);  // into the slot of tile t - 1
          next_e = entries(min(t + 3, ntiles - 1));         // read now, used next iteration
          __builtin_amdgcn_sched_barrier(0);

          // partial scores over this wave's dims
          // two accumulators per head block (even and odd chunks): four
          // independent MFMA chains instead of two
          f32x4_t acc[2], acc2[2];
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) acc[hb] = acc2[hb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int c = 0; c < 9; ++c) {
            // physical piece (4 c + g) ^ f = 4 (c ^ (sa_x >> 2)) + (sa_x & 3)
            const unsigned char* ap = c < 8 ? lds + sbase + off_sa + 64 * (c ^ (sa_x >> 2)) : lds + sbase + off_sr;
            const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(ap);
#pragma unroll
            for (int hb = 0; hb < 2; ++hb) {
              f32x4_t& ac = (c & 1) ? acc2[hb] : acc[hb];
              ac = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, c < 8 ? qb[hb][c] : qrope[hb * 64], ac, 0, 0, 0);
            }
          }
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) acc[hb] += acc2[hb];
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) xbuf[(w * 2 + hb) * 64 + lane] = acc[hb];
          // Publish the partial scores to the partner wave (w ^ 1) and wait
          // for its own: LDS writes of a wave complete in order, and the flag
          // is written after the scores are.
          ++exchanges;
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
          if (lane == 0) __hip_atomic_store(flags + w, exchanges, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          for (int spin = 0; spin < C::SPIN_LIMIT; ++spin) {
            const int seen = __builtin_amdgcn_readfirstlane(
                __hip_atomic_load(flags + (w ^ 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP));
            if (seen >= exchanges) break;
            __builtin_amdgcn_s_sleep(1);
          }
          asm volatile("" ::: "memory");
          __builtin_amdgcn_sched_barrier(0);
          if (t + 1 < ntiles) {
            // this wave's tokens of tile t + 1 (that of tile t + 2 may be in flight)
            if (t + 2 < ntiles) wait_vmcnt<C::DMA_PER_TILE>();
            else wait_vmcnt<0>();
            gate_tile(__builtin_amdgcn_readfirstlane(((t + 1) % NS) * C::SLOT));
          }
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) {
            const f32x4_t other = xbuf[((w ^ 1) * 2 + hb) * 64 + lane];
            // the same order in both waves of the pair: dim half 0 + dim half 1
            acc[hb] = dh == 0 ? acc[hb] + other : other + acc[hb];
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[hb][q] *= a.scale_log2;
          }
          const int nt = n - t * 16;  // valid tokens of the tile (1..16)
          if (nt < 16) {
#pragma unroll
            for (int hb = 0; hb < 2; ++hb)
#pragma unroll
              for (int q = 0; q < 4; ++q)
                if (4 * g + q >= nt) acc[hb][q] = -INFINITY;
          }
          // online softmax per head (lane: head 16 hb + r16, tokens 4g .. 4g + 3)
          float alpha[2];
          bool any_grow = false;
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) {
            const float mt = max_over_row_groups(fmaxf(fmaxf(acc[hb][0], acc[hb][1]), fmaxf(acc[hb][2], acc[hb][3])));
            const float m_new = fmaxf(m_run[hb], mt);  // finite: the tile has a valid token
            const bool grow = m_new > m_run[hb] + kLazyRescale;
            alpha[hb] = grow ? __builtin_amdgcn_exp2f(m_run[hb] - m_new) : 1.0f;
            m_run[hb] = grow ? m_new : m_run[hb];
            l_run[hb] *= alpha[hb];
            any_grow |= grow;
          }
          if (__builtin_amdgcn_ballot_w64(any_grow)) {
            // accumulator lane holds head lane % 32 = 16 ((lane / 16) % 2) + r16
            const float al = (lane >> 4) & 1 ? alpha[1] : alpha[0];
#pragma unroll
            for (int db = 0; db < 8; ++db) o[db] *= al;
          }
          uint32_t pk[2][2];
#pragma unroll
          for (int hb = 0; hb < 2; ++hb) {
            float p[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              p[q] = __builtin_amdgcn_exp2f(acc[hb][q] - m_run[hb]);
              l_run[hb] += p[q];
            }
            pk[hb][0] = pack_bf16x2(p[0], p[1]);
            pk[hb][1] = pack_bf16x2(p[2], p[3]);
          }
          // rows (16-lane groups) 2k and 2k + 1 of head blocks 0 and 1 ->
          // lane L: head L % 32, tokens 8 (L / 32) .. + 7
          {
            const auto s0 = __builtin_amdgcn_permlane16_swap(pk[0][0], pk[1][0], false, false);
            const auto s1 = __builtin_amdgcn_permlane16_swap(pk[0][1], pk[1][1], false, false);
            pb = __builtin_bit_cast(bf16x8_t, u32x4_t{s0[0], s1[0], s0[1], s1[1]});
          }
          values(sbase);
          __builtin_amdgcn_sched_barrier(0);
        }

      }
      // ---- partial result of this segment: this wave's heads and dims ----
      const int64_t pbase = (static_cast<int64_t>(wg) + b) * a.H + head0;
      if (dh == 0) {
#pragma unroll
        for (int hb = 0; hb < 2; ++hb) {
          const float l = sum_over_row_groups(l_run[hb]);
          if (g == 0) {
            __builtin_nontemporal_store(m_run[hb], a.part_ml + (pbase + 16 * hb + r16) * 2 + 0);
            __builtin_nontemporal_store(l, a.part_ml + (pbase + 16 * hb + r16) * 2 + 1);
          }
        }
      }
      {
        float* obase = a.part_o + pbase * DC + 256 * dh;  // uniform
        const uint32_t loff = (lane & 31) * DC + 4 * (lane >> 5);
#pragma unroll
        for (int db = 0; db < 8; ++db)
#pragma unroll
          for (int r4 = 0; r4 < 4; ++r4)
            __builtin_nontemporal_store(
                f32x4_t{o[db][4 * r4], o[db][4 * r4 + 1], o[db][4 * r4 + 2], o[db][4 * r4 + 3]},
                reinterpret_cast<f32x4_t*>(obase + loff + 32 * db + 8 * r4));
      }
    }
    remaining -= take > 0 ? take : 0;
    ++b;
    off = 0;
  }
}

}  // namespace egmla
