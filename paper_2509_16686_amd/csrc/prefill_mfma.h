// Causal prefill of EG-MLA on gfx950 MFMA, in the absorbed form of App. C
// Eq. (C.13) with the latent-space gate of Sec. 3.1 Eq. (5), for d_c = 128,
// d_r = 64, d_h = d_v = 128 and 16 heads (bf16 storage).  Included by
// prefill.hip.
//
// Every query row (token t, head h) attends to the gated latents c~_j and RoPE
// keys k^R_j of its own sequence's tokens j <= t:
//   s = tau (q_lat[t,h] . c~_j + q^R[t,h] . k^R_j),   q_lat = W_UK[h]^T q^C,
//   o_lat[t,h] = sum_j softmax_j(s) c~_j,   out[t,h] = W_UV[h] o_lat[t,h].
// All 16 heads share one key and value per token (the latent), so a tile of
// keys serves every head of a work-group's tokens at once (128 query rows):
// the kernel is a multi-query flash attention with 192-dim keys and 128-dim
// values.
//
// Five launches: a map from each token to its sequence's first token; the
// gated latent of every token (fp16, once: the attention's keys and values);
// the absorption (q_lat in fp16, q^R copied in bf16, for every token); the
// attention kernel below, which writes o_lat / l in fp16; and the
// up-projection by W_UV per head (W_UV converted exactly to fp16).
//
// Precision: the latent part of the attention runs on the fp16 MFMA.  q_lat
// is one rounding of its fp32 sum to fp16, the gated latent one rounding of
// the exact fp32 product to fp16, and so is each probability: 11-bit
// significands, where bf16 keys would need a second (lo) product to keep rows
// dominated by a few keys within the element-wise bound.  The RoPE part runs
// on the bf16 MFMA (bf16 q^R and k^R: exact products).  Values must stay
// below 65504 in magnitude.
//
// Attention kernel.  A work-group (4 waves; two per CU, whose barriers are
// independent, so that one's softmax overlaps the other's products on the
// same SIMDs) takes 8 consecutive tokens of the
// packed token stream (a block may straddle sequences: each row masks keys
// outside its own sequence) and walks tiles of 64 keys from the first token's
// sequence start to the block's last token.  Blocks are launched heaviest
// first (last in the stream first).
//  * Tile: the gated latent rows (fp16) and RoPE keys (bf16) of the next tile
//    go straight from global memory into the other of two LDS buffers while
//    the current one is computed (buffer_load_dwordx4 ... lds through buffer
//    resources based at the tile's first key: lane L's 16 bytes land at the
//    instruction's LDS base + 16 L, so each lane fetches the piece that
//    belongs in its slot).  Rows of 256 bytes hold the 16-byte pieces
//    XOR-swizzled by f(key) = 4 (key % 4) + (key / 4) % 4, RoPE rows of 128
//    bytes by (key / 2) % 8: the 16 lanes of a 16-byte read cycle and the 32
//    lanes of a transposed 8-byte read cycle each hit distinct banks.  The two
//    buffers are separate LDS objects and the tile loop is unrolled by two, so
//    that the compiler knows a tile's copies do not alias the other buffer's
//    reads (and does not wait for them before those reads).
//  * Scores: wave w holds rows (tokens 2w, 2w + 1) x 16 heads = 32 rows, its
//    query in registers as the B operand of v_mfma_f32_32x32x16_f16 (latent
//    part) and v_mfma_f32_32x32x16_bf16 (RoPE part) (lane: row lane % 32, dims
//    8 (lane / 32) + 16 c).  S^T[key][row] comes from 12 products per 32 keys
//    with the tile rows as the A operand, each chunk's operands read one chunk
//    ahead of its products.
//  * Online softmax per row in the log2 domain, lazy rescale (as the decode).
//    A lane holds 16 of each 32 keys' scores of its row; the other 16 are in
//    lane ^ 32 (one permlane32 swap for the maximum; the sums are combined
//    once at the end).
//  * Values: O^T[dim][row] += C~^T P^T.  In the score accumulator lane L holds
//    keys 8q + 4 (L / 32) + 0..3 (q = 0..3) of each 32; the value product sums
//    over keys in any order that its two operands share, so the B operand of
//    16-key chunk m is the lane's own probabilities of q = 2m, 2m + 1 (no lane
//    exchange), and the A operand is two ds_read_b64_tr_b16 of the tile (one
//    dim per lane, keys 16 m + 4 (L / 32) + 0..3 and 16 m + 8 + 4 (L / 32) + 0..3).
#pragma once

namespace egmla {

constexpr int kPfTokens = 8;      // query tokens per work-group (x 16 heads = 128 rows)
constexpr int kPfHeads = 16;
constexpr int kPfKeys = 64;       // keys per tile
constexpr int kPfThreads = 256;   // 4 waves, 32 query rows each; two work-groups per CU
constexpr int kPfDC = 128, kPfDR = 64, kPfDQ = kPfDC + kPfDR;
constexpr int kPfLatRow = 2 * kPfDC;    // bytes per key row of the gated latent
constexpr int kPfRopeRow = 2 * kPfDR;   // bytes per key row of the RoPE key
constexpr int kPfLatBytes = kPfKeys * kPfLatRow;
constexpr int kPfRopeOff = kPfLatBytes;                           // after the latent rows
constexpr int kPfBufBytes = kPfRopeOff + kPfKeys * kPfRopeRow;    // one tile buffer (24 KB; two per work-group)
static_assert(2 * 2 * kPfBufBytes <= 160 * 1024, "two work-groups of two tile buffers per compute unit");
constexpr int kPfUvTokens = 128;  // absorption and up-projection: tokens per chunk (4 waves x 32)
constexpr int kPfSideChunks = 4;  // chunks per work-group: the head's weights are staged once for them

typedef __attribute__((ext_vector_type(16))) float pf_f32x16_t;

__device__ __forceinline__ int pf_lat_swz(int key) { return ((key & 3) << 2) | ((key >> 2) & 3); }
__device__ __forceinline__ int pf_rope_swz(int key) { return (key >> 1) & 7; }

// Maximum and sum of lanes i and i ^ 32, the same value (same order) in both.
__device__ __forceinline__ float pf_pair_max(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(s[0]), __uint_as_float(s[1]));
}
__device__ __forceinline__ float pf_pair_sum(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto s = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(s[0]) + __uint_as_float(s[1]);
}

// seq_start[t] = the first token of t's sequence (cu_seqlens[b] for the last b
// with cu_seqlens[b] <= t), clamped into [0, t].
__global__ __launch_bounds__(256) void prefill_seqmap_kernel(const int32_t* __restrict__ cu, int B, int T,
                                                             int32_t* __restrict__ seq_start) {
  const int t = blockIdx.x * 256 + threadIdx.x;
  if (t >= T) return;
  int lo = 0, hi = B - 1;  // largest b in [0, B) with cu[b] <= t (b = 0 if none)
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= t) lo = mid;
    else hi = mid - 1;
  }
  seq_start[t] = min(max(cu[lo], 0), t);
}

// ct[t] = c_t (.) G[id_t] in fp16 (the exact fp32 products, each rounded
// once): 16 threads per token, 8 dims each.
__global__ __launch_bounds__(256) void prefill_gate_kernel(const uint16_t* __restrict__ latent,
                                                           const int32_t* __restrict__ ids,
                                                           const uint16_t* __restrict__ gate,
                                                           uint16_t* __restrict__ ct, int T, int V) {
  const int i = blockIdx.x * 256 + threadIdx.x, t = i >> 4, p = i & 15;
  if (t >= T) return;
  const u32x4_t c = *reinterpret_cast<const u32x4_t*>(latent + static_cast<int64_t>(t) * kPfDQ + 8 * p);
  const u32x4_t g = *reinterpret_cast<const u32x4_t*>(gate + static_cast<int64_t>(clamp_id(ids[t], V)) * kPfDC + 8 * p);
  *reinterpret_cast<u32x4_t*>(ct + static_cast<int64_t>(t) * kPfDC + 8 * p) = gate_chunk_f16(c, g);
}

// Word 3 of a raw buffer resource on gfx9 (32-bit data format; stride 0, so
// the record count is a byte count and offsets past it read zeros).
constexpr int kPfBufRsrcWord3 = 0x00020000;

struct PrefillArgs {
  const uint16_t* qf;          // [T][16][192]: q_lat fp16 | q^R bf16
  const uint16_t* latent;      // [T][192] bf16: c | k^R
  const uint16_t* ct;          // [T][128] fp16: gated latent
  const int32_t* seq_start;    // [T]
  uint16_t* olat;              // [T][16][128] fp16: o_lat / l
  int T;
  float scale_log2;            // tau log2(e)
};

__global__ __launch_bounds__(kPfThreads, 2) void prefill_attn_mfma_kernel(PrefillArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds0[kPfBufBytes];  // two tile buffers
  __shared__ __attribute__((aligned(16))) unsigned char lds1[kPfBufBytes];
  const int nblk = (a.T + kPfTokens - 1) / kPfTokens;
  const int q0 = (nblk - 1 - static_cast<int>(blockIdx.x)) * kPfTokens;  // heaviest blocks first
  const int q_last = min(q0 + kPfTokens, a.T) - 1;
  const int kbeg = min(max(a.seq_start[q0], 0), q0);                 // keys from here ...
  const int kend = q_last + 1;                                       // ... to here (exclusive)
  const int s_max = min(max(a.seq_start[q_last], kbeg), q_last);     // latest sequence start in the block
  const int ntiles = (kend - kbeg + kPfKeys - 1) / kPfKeys;

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int r16 = lane & 15, R1 = (lane >> 4) & 1;
  // this lane's query row; rows past the stream repeat its last token and are not stored
  const int t_row = q0 + 2 * w + (r32 >> 4);
  const bool row_ok = t_row < a.T;
  const int t_c = min(t_row, a.T - 1);
  const int head = r32 & 15;
  const int s_row = min(max(a.seq_start[t_c], kbeg), t_c);

  f16x8_t qv[kPfDC / 16];   // q_lat (fp16)
  bf16x8_t qr[kPfDR / 16];  // q^R (bf16)
  {
    const uint16_t* qrow = a.qf + (static_cast<int64_t>(t_c) * kPfHeads + head) * kPfDQ + 8 * h;
#pragma unroll
    for (int c = 0; c < kPfDC / 16; ++c) qv[c] = *reinterpret_cast<const f16x8_t*>(qrow + 16 * c);
#pragma unroll
    for (int c = 0; c < kPfDR / 16; ++c) qr[c] = *reinterpret_cast<const bf16x8_t*>(qrow + kPfDC + 16 * c);
  }

  // tile copies into LDS: wave w issues latent instructions I = 4 w + j (keys
  // 4 I .. 4 I + 3; lane: key 4 I + lane / 16, slot lane % 16) and RoPE
  // instructions I = 2 w + j (keys 8 I .. 8 I + 7; lane: key 8 I + lane / 8,
  // slot lane % 8); slot s of a row holds logical piece s ^ swizzle(key)
  constexpr int NLI = kPfKeys / 4 / 4, NRI = kPfKeys / 8 / 4;
  auto key_at = [&](int tile, int k) { return min(kbeg + tile * kPfKeys + k, kend - 1); };
  auto lds_ptr = [](unsigned char* p) { return (__attribute__((address_space(3))) void*)p; };
  auto issue_tile = [&](int tile, unsigned char* base) {
    const int t0 = kbeg + tile * kPfKeys;
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.ct + static_cast<int64_t>(t0) * kPfDC), 0, kPfKeys * kPfLatRow, kPfBufRsrcWord3);
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.latent + static_cast<int64_t>(t0) * kPfDQ + kPfDC), 0, kPfKeys * kPfDQ * 2,
        kPfBufRsrcWord3);
#pragma unroll
    for (int j = 0; j < NLI; ++j) {
      const int I = NLI * w + j, key = 4 * I + (lane >> 4), piece = (lane & 15) ^ pf_lat_swz(key);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, lds_ptr(base + 4 * I * kPfLatRow), 16,
                                               (key_at(tile, key) - t0) * kPfLatRow + 16 * piece, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < NRI; ++j) {
      const int I = NRI * w + j, key = 8 * I + (lane >> 3), piece = (lane & 7) ^ pf_rope_swz(key);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rr, lds_ptr(base + kPfRopeOff + 8 * I * kPfRopeRow), 16,
                                               (key_at(tile, key) - t0) * kPfDQ * 2 + 16 * piece, 0, 0, 0);
    }
  };
  // this wave's copies have landed; the barrier after it covers every wave's
  auto tile_landed = []() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  // per-lane LDS offsets (bytes within a tile buffer)
  const int off_sl = r32 * kPfLatRow;               // score A: key row 32 kb + r32 (+ 32 kb rows)
  const int swz_sl = pf_lat_swz(r32);
  const int off_sr = kPfRopeOff + r32 * kPfRopeRow;
  const int swz_sr = pf_rope_swz(r32);
  // value A (transposed reads): rows 16 m + 4 h + r16 / 4 (+ 8), byte 8 (r16 % 2) of the piece
  const int off_v = (4 * h + (r16 >> 2)) * kPfLatRow + 8 * (r16 & 1);
  const int vlo = 2 * R1 + ((r16 & 3) >> 1);  // low 2 bits of the logical piece

  pf_f32x16_t o[kPfDC / 32];
#pragma unroll
  for (int db = 0; db < kPfDC / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m_run = -1e30f, l_run = 0.f;  // finite start: a fully masked tile leaves both unchanged

  issue_tile(0, lds0);
  tile_landed();
  __syncthreads();

  // step i computes tile i from buffer tb and copies tile i + 1 into nb (last
  // read in step i - 1, which ended in a barrier)
  auto step = [&](int i, const unsigned char* tb, unsigned char* nb) {
    if (i + 1 < ntiles) issue_tile(i + 1, nb);
    const int k_lo = kbeg + i * kPfKeys;

    // ---- scores S^T[key][row] for keys k_lo + 32 kb + (0..31) ----
    pf_f32x16_t s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
    for (int c = 0; c < kPfDC / 16; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const f16x8_t av =
            *reinterpret_cast<const f16x8_t*>(tb + off_sl + 32 * kb * kPfLatRow + 16 * ((2 * c + h) ^ swz_sl));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, qv[c], s[kb], 0, 0, 0);
      }
#pragma unroll
    for (int c = 0; c < kPfDR / 16; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(tb + off_sr + 32 * kb * kPfRopeRow +
                                                                16 * ((2 * c + h) ^ swz_sr));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qr[c], s[kb], 0, 0, 0);
      }
    // issue order: the A operands of a chunk (both key blocks) one chunk ahead
    // of its two products
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
    for (int c = 0; c < kPfDQ / 16 - 1; ++c) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    // keys outside [s_row, t_row] (or past the block) only in tiles that reach
    // past the block's first token or start before its latest sequence start
    if (k_lo + kPfKeys - 1 > q0 || k_lo < s_max) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k_lo + 32 * kb + 8 * (r >> 2) + 4 * h + (r & 3);
          if (key < s_row || key > t_c) s[kb][r] = -INFINITY;
        }
    }

    // ---- online softmax (row = lane % 32; keys split between lanes L and L ^ 32) ----
    // the scale (tau log2 e > 0) commutes with the maximum; it is applied inside the exponent
    float mt = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mt = fmaxf(mt, s[kb][r]);
    mt = pf_pair_max(mt) * a.scale_log2;
    const float m_new = fmaxf(m_run, mt);
    const bool grow = m_new > m_run + kLazyRescale;
    const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - m_new) : 1.0f;
    m_run = grow ? m_new : m_run;
    l_run *= alpha;
    if (__builtin_amdgcn_ballot_w64(grow)) {
#pragma unroll
      for (int db = 0; db < kPfDC / 32; ++db) o[db] *= alpha;
    }
    f16x8_t pb[2][2];  // [kb][16-key chunk m]: keys 16 m + 8 (e / 4) + 4 h + e % 4 of element e
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        float p[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][8 * m + e], a.scale_log2, -m_run));
          l_run += p[e];
        }
        pb[kb][m] = __builtin_bit_cast(f16x8_t, u32x4_t{pack_f16x2(p[0], p[1]), pack_f16x2(p[2], p[3]),
                                                        pack_f16x2(p[4], p[5]), pack_f16x2(p[6], p[7])});
      }

    // ---- values O^T[dim][row] += C~^T P^T ----
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const unsigned char* vp = tb + off_v + (32 * kb + 16 * m) * kPfLatRow;
#pragma unroll
        for (int db = 0; db < kPfDC / 32; ++db) {
          // logical piece 4 db + vlo; rows +0 and +8 swizzle with 4 (r16 / 4) + h and + 2
          const int p0 = 4 * (db ^ (r16 >> 2)) + (vlo ^ h);
          const int p1 = 4 * (db ^ (r16 >> 2)) + (vlo ^ (h + 2));
          const s16x4_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(vp + 16 * p0));
          const s16x4_t a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(vp + 8 * kPfLatRow + 16 * p1));
          const f16x8_t av = __builtin_bit_cast(f16x8_t, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, pb[kb][m], o[db], 0, 0, 0);
        }
      }

    tile_landed();
    __syncthreads();
  };
  for (int i = 0; i < ntiles; i += 2) {
    step(i, lds0, lds1);
    if (i + 1 < ntiles) step(i + 1, lds1, lds0);
  }

  // ---- o_lat / l: lane holds dims 32 db + 8 q + 4 h + 0..3 of its row ----
  const float inv = 1.0f / pf_pair_sum(l_run);
  if (row_ok) {
    uint16_t* orow = a.olat + (static_cast<int64_t>(t_row) * kPfHeads + head) * kPfDC + 4 * h;
#pragma unroll
    for (int db = 0; db < kPfDC / 32; ++db)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<u32x2_t*>(orow + 32 * db + 8 * q) =
            u32x2_t{pack_f16x2(o[db][4 * q] * inv, o[db][4 * q + 1] * inv),
                    pack_f16x2(o[db][4 * q + 2] * inv, o[db][4 * q + 3] * inv)};
  }
}

// q_lat[t, h, :] = W_UK[h]^T q^C[t, h, :] in fp16, and q^R copied in bf16, for up to
// 4 chunks of 128 tokens of one head per work-group (4 waves of 32 tokens; the
// next chunk's rows load while a chunk computes and stores).  W_UK[h]
// ([d_h][d_c] row-major, rows padded to 288 bytes) is staged in LDS once and
// read back as the A operand of v_mfma_f32_32x32x16_bf16 with
// ds_read_b64_tr_b16 (one output column per lane, 4 consecutive rows per
// read); the query rows come straight from global as the B operand, and the
// accumulator holds q_lat^T, stored 4 consecutive columns at a time.
__global__ __launch_bounds__(256) void prefill_absorb_kernel(const uint16_t* __restrict__ q,
                                                             const uint16_t* __restrict__ w_uk,
                                                             uint16_t* __restrict__ qf, int T) {
  constexpr int DH = 128, RS = kPfDC + 16, DQin = DH + kPfDR;
  __shared__ __attribute__((aligned(16))) uint16_t wk[DH * RS];
  const int hh = blockIdx.y;
  const int c0 = blockIdx.x * kPfSideChunks;
  const int nch = min(kPfSideChunks, (T + kPfUvTokens - 1) / kPfUvTokens - c0);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int r16 = lane & 15, R1 = (lane >> 4) & 1;
  // a chunk's operands: the lane's token's q^C (B operand) and, per thread, 32
  // dims (4 x 16 bytes) of q^R of token t0 + tid / 2 (copied through)
  bf16x8_t qb[DH / 16];
  u32x4_t rq[4];
  auto load = [&](int chunk) {
    const int t0 = chunk * kPfUvTokens;
    const int tc = min(t0 + 32 * w + r32, T - 1);
    const uint16_t* qrow = q + (static_cast<int64_t>(tc) * kPfHeads + hh) * DQin + 8 * h;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c) qb[c] = *reinterpret_cast<const bf16x8_t*>(qrow + 16 * c);
    const int rt = min(t0 + (tid >> 1), T - 1);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      rq[j] = *reinterpret_cast<const u32x4_t*>(q + (static_cast<int64_t>(rt) * kPfHeads + hh) * DQin + DH +
                                                32 * (tid & 1) + 8 * j);
  };
  load(c0);
  for (int p = tid; p < DH * kPfDC / 8; p += 256) {
    const int k = p / (kPfDC / 8), c8 = (p % (kPfDC / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(wk + k * RS + c8) =
        *reinterpret_cast<const u32x4_t*>(w_uk + (static_cast<int64_t>(hh) * DH + k) * kPfDC + c8);
  }
  __syncthreads();
  // A operand of chunk c, column block cb: lane (column 32 cb + 16 R1 + r16) gets
  // rows 16 c + 8 h + 0..7; lane r16 of a 16-lane group addresses row + r16 / 4,
  // columns 4 (r16 % 4) .. + 3 of the group's 16
  const uint16_t* abase = wk + (8 * h + (r16 >> 2)) * RS + 16 * R1 + 4 * (r16 & 3);
  for (int k = 0; k < nch; ++k) {
    const int t0 = (c0 + k) * kPfUvTokens;
    const int t = t0 + 32 * w + r32;
    pf_f32x16_t acc[kPfDC / 32];
#pragma unroll
    for (int cb = 0; cb < kPfDC / 32; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;
#pragma unroll
    for (int c = 0; c < DH / 16; ++c)
#pragma unroll
      for (int cb = 0; cb < kPfDC / 32; ++cb) {
        const uint16_t* ap = abase + 16 * c * RS + 32 * cb;
        const s16x4_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)ap);
        const s16x4_t a1 =
            __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(ap + 4 * RS));
        const bf16x8_t av = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7));
        acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qb[c], acc[cb], 0, 0, 0);
      }
    const u32x4_t r0 = rq[0], r1 = rq[1], r2 = rq[2], r3 = rq[3];
    // the next chunk's rows travel while this one is stored (the last chunk loads itself again)
    __builtin_amdgcn_sched_barrier(0);
    load(c0 + min(k + 1, nch - 1));
    __builtin_amdgcn_sched_barrier(0);
    if (t < T) {
      uint16_t* dst = qf + (static_cast<int64_t>(t) * kPfHeads + hh) * kPfDQ + 4 * h;
#pragma unroll
      for (int cb = 0; cb < kPfDC / 32; ++cb)
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
          *reinterpret_cast<u32x2_t*>(dst + 32 * cb + 8 * qq) =
              u32x2_t{pack_f16x2(acc[cb][4 * qq], acc[cb][4 * qq + 1]),
                      pack_f16x2(acc[cb][4 * qq + 2], acc[cb][4 * qq + 3])};
    }
    if (t0 + (tid >> 1) < T) {
      uint16_t* dr = qf + (static_cast<int64_t>(t0 + (tid >> 1)) * kPfHeads + hh) * kPfDQ + kPfDC + 32 * (tid & 1);
      *reinterpret_cast<u32x4_t*>(dr) = r0;
      *reinterpret_cast<u32x4_t*>(dr + 8) = r1;
      *reinterpret_cast<u32x4_t*>(dr + 16) = r2;
      *reinterpret_cast<u32x4_t*>(dr + 24) = r3;
    }
  }
}

// out[t, h, :] = W_UV[h] o_lat[t, h, :] for up to 4 chunks of 128 tokens of
// one head per work-group (4 waves of 32 tokens; the next chunk's rows load
// while a chunk is stored): W_UV[h] ([d_v][d_c], rows padded by 16 bytes)
// converted to fp16 (exact for magnitudes between 2^-14 and 65504; smaller
// weights become fp16 subnormals, an absolute error below 2^-25) in LDS as the
// A operand, the fp16 o_lat rows straight from global as the B operand of
// v_mfma_f32_32x32x16_f16; the accumulator holds out^T, stored 4 consecutive v
// at a time.
__global__ __launch_bounds__(256) void prefill_uv_kernel(const uint16_t* __restrict__ olat,
                                                         const uint16_t* __restrict__ w_uv,
                                                         uint16_t* __restrict__ out, int T) {
  constexpr int DV = 128, RS = kPfDC + 8;
  __shared__ __attribute__((aligned(16))) uint16_t wl[DV * RS];
  const int hh = blockIdx.y;
  const int c0 = blockIdx.x * kPfSideChunks;
  const int nch = min(kPfSideChunks, (T + kPfUvTokens - 1) / kPfUvTokens - c0);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  f16x8_t ov[kPfDC / 16];  // the lane's token's o_lat, dims 16 c + 8 h .. + 7
  auto load = [&](int chunk) {
    const int tc = min(chunk * kPfUvTokens + 32 * w + r32, T - 1);
    const uint16_t* orow = olat + (static_cast<int64_t>(tc) * kPfHeads + hh) * kPfDC + 8 * h;
#pragma unroll
    for (int c = 0; c < kPfDC / 16; ++c) ov[c] = *reinterpret_cast<const f16x8_t*>(orow + 16 * c);
  };
  load(c0);
  for (int p = tid; p < DV * kPfDC / 8; p += 256) {
    const int v = p / (kPfDC / 8), k8 = (p % (kPfDC / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(wl + v * RS + k8) =
        bf16x8_to_f16x8(*reinterpret_cast<const u32x4_t*>(w_uv + (static_cast<int64_t>(hh) * DV + v) * kPfDC + k8));
  }
  __syncthreads();
  for (int k = 0; k < nch; ++k) {
    const int t = (c0 + k) * kPfUvTokens + 32 * w + r32;
    f16x8_t ob[kPfDC / 16];
#pragma unroll
    for (int c = 0; c < kPfDC / 16; ++c) ob[c] = ov[c];
    pf_f32x16_t acc[DV / 32];
#pragma unroll
    for (int vb = 0; vb < DV / 32; ++vb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[vb][r] = 0.f;
#pragma unroll
    for (int c = 0; c < kPfDC / 16; ++c)
#pragma unroll
      for (int vb = 0; vb < DV / 32; ++vb) {
        const f16x8_t av = *reinterpret_cast<const f16x8_t*>(wl + (32 * vb + r32) * RS + 16 * c + 8 * h);
        acc[vb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, ob[c], acc[vb], 0, 0, 0);
      }
    // the next chunk's rows travel while this one is stored (the last chunk loads itself again)
    __builtin_amdgcn_sched_barrier(0);
    load(c0 + min(k + 1, nch - 1));
    __builtin_amdgcn_sched_barrier(0);
    if (t < T) {
      uint16_t* dst = out + (static_cast<int64_t>(t) * kPfHeads + hh) * DV + 4 * h;
#pragma unroll
      for (int vb = 0; vb < DV / 32; ++vb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<u32x2_t*>(dst + 32 * vb + 8 * q) = u32x2_t{
              pack_bf16x2(acc[vb][4 * q], acc[vb][4 * q + 1]), pack_bf16x2(acc[vb][4 * q + 2], acc[vb][4 * q + 3])};
    }
  }
}

}  // namespace egmla
