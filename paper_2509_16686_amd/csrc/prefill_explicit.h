// Causal prefill of EG-MLA on gfx950 MFMA in the explicit form of App. C
// Eq. (C.2), (C.6), (C.11)-(C.13), with the latent-space gate of Sec. 3.1
// Eq. (5), for layers with many heads and a wide latent (d_c = 512 with 128
// heads: there the absorbed form costs 2 (d_c + d_r + d_c) = 2176 flops per
// (row, key) pair and head, the explicit one 2 (d_h + d_r + d_v) = 640).
// Included by prefill.hip.  bf16 storage, d_h = d_v = 128, d_r = 64, d_c a
// multiple of 64.
//
//   K^C[h][t] = W_UK[h] c~_t,  V[h][t] = W_UV[h] c~_t,  c~_t = c_t (.) G[id_t]
//   out[t,h]  = sum_{j <= t, same sequence} softmax_j(tau (q^C[t,h].K^C[h][j] + q^R[t,h].k^R_j)) V[h][j]
//
// Two launches after the sequence map: the projection (a GEMM over d_c) and
// the attention (a causal flash attention per head with 192-dim keys, the
// RoPE key shared by all heads, and 128-dim values).
//
// Precision.  The gated latent enters the projection as bf16 hi + lo (their
// sum is the fp32 product c * g exactly, two products per step), so K^C and V
// carry only the rounding of their fp32 sums, which is to fp16 (11-bit
// significand; values must stay below 65504 in magnitude, true of layers whose
// keys and values are of order one to thousands).  The attention runs on the
// fp16 MFMA for the latent part of the scores and for the values (the bf16
// query converts to fp16 exactly for magnitudes between 2^-14 and 65504) and on
// the bf16 MFMA for the RoPE part (bf16 query and key: exact products); P is
// rounded to fp16, and the output is rounded once to bf16.
#pragma once

namespace egmla {

constexpr int kPxDH = 128, kPxDR = 64, kPxDK = kPxDH + kPxDR;  // key dims per head (K^C | k^R)
// Word 3 of a raw buffer resource on gfx9 (32-bit data format; stride 0, so
// the record count is a byte count and offsets past it read zeros).
constexpr int kBufRsrcWord3 = 0x00020000;

// ---------------------------------------------------------------------------
// Gated latent, once per token: c~_t = c_t (.) G[id_t] as bf16 hi + lo rows
// (ct_hi[t] + ct_lo[t] is the exact fp32 product), 8 dims per thread.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void prefill_x_gate_kernel(const uint16_t* __restrict__ latent,
                                                             const int32_t* __restrict__ ids,
                                                             const uint16_t* __restrict__ gate,
                                                             uint16_t* __restrict__ ct_hi, uint16_t* __restrict__ ct_lo,
                                                             int T, int DC, int V) {
  const int per = DC / 8;  // threads per token
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int t = static_cast<int>(i / per), p = static_cast<int>(i % per);
  if (t >= T) return;
  const u32x4_t c = *reinterpret_cast<const u32x4_t*>(latent + static_cast<int64_t>(t) * (DC + kPxDR) + 8 * p);
  const u32x4_t g = *reinterpret_cast<const u32x4_t*>(gate + static_cast<int64_t>(clamp_id(ids[t], V)) * DC + 8 * p);
  u32x4_t hi, lo;
  gate_chunk_hilo(c, g, hi, lo);
  *reinterpret_cast<u32x4_t*>(ct_hi + static_cast<int64_t>(t) * DC + 8 * p) = hi;
  *reinterpret_cast<u32x4_t*>(ct_lo + static_cast<int64_t>(t) * DC + 8 * p) = lo;
}

// ---------------------------------------------------------------------------
// Projection.  Work-group (tt, h) forms K^C[h] and V[h] of tokens
// 128 tt .. + 127: a product of the 128 gated latent rows (B operand, as hi
// and lo) with the 256 rows W_UK[h] | W_UV[h] (A operand) over d_c, in steps
// of 32.  Each step's rows (64 bytes each: hi rows, lo rows, weights) go
// straight from global memory into the other of two LDS buffers while the
// current step is computed (buffer_load_dwordx4 ... lds: one instruction
// fills 16 rows; lane L's 16 bytes land at the instruction's LDS base + 16 L,
// so each lane fetches the piece that belongs in its slot); the four 16-byte
// pieces of a row are XOR-swizzled by (row / 4) % 4, so that the operand
// reads of 8 rows by 8 lanes hit distinct banks.  The two buffers are
// separate LDS objects and the step loop is unrolled by two (the compiler
// then knows the copies into one do not alias the other's reads).  Wave
// (wt, wo) = (w % 2, w / 2) forms tokens 64 wt .. + 63 of K^C (wo = 0) or V
// (wo = 1): 2 x 4 tiles of v_mfma_f32_32x32x16_bf16, two products per tile
// and step.
// ---------------------------------------------------------------------------
constexpr int kPxTok = 128, kPxOut = 256, kPxK = 32;
constexpr int kPxRowB = 2 * kPxK;                          // bytes per staged row (64)
constexpr int kPxRows = 2 * kPxTok + kPxOut;               // hi, lo, weights
constexpr int kPxProjBuf = kPxRows * kPxRowB;              // bytes per buffer (32 KB)
static_assert(2 * 2 * kPxProjBuf <= 160 * 1024, "two work-groups per compute unit");

__device__ __forceinline__ int px_swz(int row) { return (row >> 2) & 3; }

__global__ __launch_bounds__(256, 2) void prefill_x_proj_kernel(const uint16_t* __restrict__ ct_hi,
                                                                const uint16_t* __restrict__ ct_lo,
                                                                const uint16_t* __restrict__ w_uk,
                                                                const uint16_t* __restrict__ w_uv,
                                                                uint16_t* __restrict__ kc, uint16_t* __restrict__ vv,
                                                                int T, int DC) {
  __shared__ __attribute__((aligned(16))) unsigned char st0[kPxProjBuf];
  __shared__ __attribute__((aligned(16))) unsigned char st1[kPxProjBuf];
  const int tt = blockIdx.x, hh = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wt = w & 1, wo = w >> 1;
  const int t0 = kPxTok * tt;
  // buffer resources: the block's hi and lo rows, and the head's weight rows
  const int ntok = min(kPxTok, T - t0);
  const __amdgpu_buffer_rsrc_t rh =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(ct_hi + static_cast<int64_t>(t0) * DC), 0, ntok * DC * 2,
                                        kBufRsrcWord3);
  const __amdgpu_buffer_rsrc_t rl =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(ct_lo + static_cast<int64_t>(t0) * DC), 0, ntok * DC * 2,
                                        kBufRsrcWord3);
  const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(w_uk + static_cast<int64_t>(hh) * kPxDH * DC), 0, kPxDH * DC * 2, kBufRsrcWord3);
  const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(w_uv + static_cast<int64_t>(hh) * kPxDH * DC), 0, kPxDH * DC * 2, kBufRsrcWord3);
  // copies of a step: wave w fills rows 16 I .. 16 I + 15 for I = 8 w + j
  // (j < 8): region w of the four of 128 rows (hi, lo, W_UK, W_UV); lane: row
  // 16 I + lane / 4, slot lane % 4, which holds piece slot ^ swizzle(row)
  auto lds_ptr = [](unsigned char* p) { return (__attribute__((address_space(3))) void*)p; };
  auto issue_step = [&](int step, unsigned char* base) {
    const int kb = kPxRowB * step;  // byte offset of the step's 32 k in a row
    // wave w (uniform) takes one region: 0 hi rows, 1 lo rows, 2 W_UK rows, 3 W_UV rows
    const __amdgpu_buffer_rsrc_t rs = w == 0 ? rh : w == 1 ? rl : w == 2 ? rk : rv;
    const int nrow = w < 2 ? ntok : kPxDH;  // rows of the region (latent rows past the end repeat the last)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int I = 8 * w + j, row = 16 * I + (lane >> 2), piece = (lane & 3) ^ px_swz(row);
      const int r = min(row & (kPxTok - 1), nrow - 1);  // row within the region
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, lds_ptr(base + 16 * I * kPxRowB), 16, r * DC * 2 + kb + 16 * piece,
                                               0, 0, 0);
    }
  };
  auto step_landed = []() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };
  pf_f32x16_t acc[2][4];
#pragma unroll
  for (int tb = 0; tb < 2; ++tb)
#pragma unroll
    for (int ob = 0; ob < 4; ++ob)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[tb][ob][r] = 0.f;
  // operand rows of this lane: latent row 64 wt + 32 tb + r32, weight row 128 wo + 32 ob + r32
  auto compute = [&](const unsigned char* b) {
#pragma unroll
    for (int kk = 0; kk < kPxK / 16; ++kk) {
      bf16x8_t bh[2], bl[2], av[4];
#pragma unroll
      for (int tb = 0; tb < 2; ++tb) {
        const int row = 64 * wt + 32 * tb + r32;
        const int off = row * kPxRowB + 16 * ((2 * kk + h) ^ px_swz(row));
        bh[tb] = *reinterpret_cast<const bf16x8_t*>(b + off);
        bl[tb] = *reinterpret_cast<const bf16x8_t*>(b + kPxTok * kPxRowB + off);
      }
#pragma unroll
      for (int ob = 0; ob < 4; ++ob) {
        const int row = 2 * kPxTok + 128 * wo + 32 * ob + r32;
        av[ob] = *reinterpret_cast<const bf16x8_t*>(b + row * kPxRowB + 16 * ((2 * kk + h) ^ px_swz(row)));
      }
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int ob = 0; ob < 4; ++ob) {
          acc[tb][ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[ob], bh[tb], acc[tb][ob], 0, 0, 0);
          acc[tb][ob] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[ob], bl[tb], acc[tb][ob], 0, 0, 0);
        }
    }
  };
  // step s computes from one buffer while step s + 1 is copied into the other
  // (last read in step s - 1, which ended in a barrier); the step count is even
  const int steps = DC / kPxK;
  issue_step(0, st0);
  step_landed();
  __syncthreads();
  // (a scheduling barrier after each issue keeps the copies at the start of
  // the step instead of sunk below its products)
  for (int s0 = 0; s0 < steps; s0 += 2) {
    issue_step(s0 + 1, st1);
    __builtin_amdgcn_sched_barrier(0);
    compute(st0);
    step_landed();
    __syncthreads();
    if (s0 + 2 < steps) issue_step(s0 + 2, st0);
    __builtin_amdgcn_sched_barrier(0);
    compute(st1);
    step_landed();
    __syncthreads();
  }
  // lane holds dims 32 ob + 8 q + 4 h + (0..3) of token 64 wt + 32 tb + r32 in acc[tb][ob][4 q + (0..3)]
  uint16_t* dst = wo == 0 ? kc : vv;
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int t = t0 + 64 * wt + 32 * tb + r32;
    if (t >= T) break;
    uint16_t* row = dst + (static_cast<int64_t>(hh) * T + t) * kPxDH + 4 * h;
#pragma unroll
    for (int ob = 0; ob < 4; ++ob)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<u32x2_t*>(row + 32 * ob + 8 * q) =
            u32x2_t{pack_f16x2(acc[tb][ob][4 * q], acc[tb][ob][4 * q + 1]),
                    pack_f16x2(acc[tb][ob][4 * q + 2], acc[tb][ob][4 * q + 3])};
  }
}

// ---------------------------------------------------------------------------
// Attention.  Work-group (block, h) takes the 128 consecutive tokens
// 128 block .. + 127 of the packed stream for head h (a block may straddle
// sequences: each row masks keys outside its own sequence) and walks tiles of
// 64 keys from the first token's sequence start to the block's last token
// (a head's blocks on one XCD, last-in-the-stream first).  Wave w holds the rows of tokens
// 32 w .. + 31 of the block, its query (fp16) in registers as the B operand of
// v_mfma_f32_32x32x16_f16 (lane: row lane % 32, dims 8 (lane / 32) + 16 c).
//  * Tile: K^C rows (256 bytes, fp16), k^R rows (128 bytes, bf16) and V rows
//    (256 bytes, fp16) of the next tile go straight from global memory into
//    the other of two LDS buffers while the current one is computed
//    (buffer_load_dwordx4 ... lds through buffer resources based at the
//    tile's first key: lane L's 16 bytes land at the instruction's LDS base +
//    16 L, so each lane fetches the piece that belongs in its slot); 16-byte
//    pieces XOR-swizzled by f(key) = 4 (key % 4) + (key / 4) % 4 in the
//    256-byte rows and (key / 2) % 8 in the RoPE rows.  No register holds a
//    tile in flight, and the buffer form (unlike the global one) leaves the
//    compiler's waits for LDS reads exact while the copies are in flight.
//  * The A operands of each score chunk are read two chunks ahead of its
//    products (scheduling hints), so a pair of products waits for reads
//    issued two pairs earlier.
//  * Scores S^T[key][row]: 12 products per 32 keys, the tile rows as the A
//    operand (8 of K^C on the fp16 MFMA, 4 of k^R on the bf16 MFMA).
//  * Online softmax per row in the log2 domain with lazy rescale; a lane holds
//    16 of each 32 keys' scores of its row, the other 16 are in lane ^ 32.
//  * Values O^T[dim][row] += V^T P^T: the B operand is the lane's own
//    probabilities (fp16), the A operand two ds_read_b64_tr_b16 of the V rows.
// ---------------------------------------------------------------------------
constexpr int kPxQTok = 128;                       // query tokens per work-group (4 waves x 32)
constexpr int kPxKeys = 64;                        // keys per tile
constexpr int kPxKcRow = 2 * kPxDH;                // bytes per K^C / V row
constexpr int kPxRopeRow = 2 * kPxDR;              // bytes per k^R row
constexpr int kPxRopeOff = kPxKeys * kPxKcRow;
constexpr int kPxVOff = kPxRopeOff + kPxKeys * kPxRopeRow;
constexpr int kPxTileBytes = kPxVOff + kPxKeys * kPxKcRow;   // 40 KB; two per work-group
static_assert(2 * 2 * kPxTileBytes <= 160 * 1024, "two work-groups of two tile buffers per compute unit");

struct PrefillXArgs {
  const uint16_t* q;           // [T][H][192] bf16: q^C | q^R
  const uint16_t* latent;      // [T][d_c + 64] bf16: c | k^R
  const uint16_t* kc;          // [H][T][128] fp16
  const uint16_t* vv;          // [H][T][128] fp16
  const int32_t* seq_start;    // [T]
  uint16_t* out;               // [T][H][128] bf16
  int T, H, DC;
  float scale_log2;            // tau log2(e)
};

__global__ __launch_bounds__(256, 2) void prefill_x_attn_kernel(PrefillXArgs a) {
  // two tile buffers, distinct objects: the compiler then knows that a tile's
  // copies into one do not alias the reads of the other, and does not wait for
  // the copies before those reads
  __shared__ __attribute__((aligned(16))) unsigned char lds0[kPxTileBytes];
  __shared__ __attribute__((aligned(16))) unsigned char lds1[kPxTileBytes];
  // one XCD takes whole heads (a contiguous range of the head-major order), so
  // the blocks of a head read its K^C and V tiles through one L2 cache; within
  // a head the last blocks of the stream (the heaviest) come first
  const int nblk = (a.T + kPxQTok - 1) / kPxQTok;
  const int lb = xcd_logical_block(static_cast<int>(blockIdx.x), nblk * a.H);
  const int hh = lb / nblk;
  const int q0 = (nblk - 1 - lb % nblk) * kPxQTok;
  const int q_last = min(q0 + kPxQTok, a.T) - 1;
  const int kbeg = min(max(a.seq_start[q0], 0), q0);                 // keys from here ...
  const int kend = q_last + 1;                                       // ... to here (exclusive)
  const int s_max = min(max(a.seq_start[q_last], kbeg), q_last);     // latest sequence start in the block
  const int ntiles = (kend - kbeg + kPxKeys - 1) / kPxKeys;
  const int DQ = a.DC + kPxDR;

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r32 = lane & 31, h = lane >> 5;
  const int r16 = lane & 15, R1 = (lane >> 4) & 1;
  // this lane's query row; rows past the stream repeat its last token and are not stored
  const int t_row = q0 + 32 * w + r32;
  const bool row_ok = t_row < a.T;
  const int t_c = min(t_row, a.T - 1);
  const int s_row = min(max(a.seq_start[t_c], kbeg), t_c);

  f16x8_t qv[kPxDH / 16];   // latent part (fp16)
  bf16x8_t qr[kPxDR / 16];  // RoPE part (bf16)
  {
    const uint16_t* qrow = a.q + (static_cast<int64_t>(t_c) * a.H + hh) * kPxDK + 8 * h;
#pragma unroll
    for (int c = 0; c < kPxDH / 16; ++c)
      qv[c] = __builtin_bit_cast(f16x8_t, bf16x8_to_f16x8(*reinterpret_cast<const u32x4_t*>(qrow + 16 * c)));
#pragma unroll
    for (int c = 0; c < kPxDR / 16; ++c) qr[c] = *reinterpret_cast<const bf16x8_t*>(qrow + kPxDH + 16 * c);
  }

  // tile loads into LDS: wave w issues K^C and V instructions I = 4 w + j
  // (keys 4 I .. 4 I + 3; lane: key 4 I + lane / 16, slot lane % 16) and RoPE
  // instructions I = 2 w + j (keys 8 I .. 8 I + 7; lane: key 8 I + lane / 8,
  // slot lane % 8); slot s of a row holds logical piece s ^ swizzle(key)
  constexpr int NKI = kPxKeys / 4 / 4, NRI = kPxKeys / 8 / 4;
  auto key_at = [&](int tile, int k) { return min(kbeg + tile * kPxKeys + k, kend - 1); };
  const uint16_t* kc_h = a.kc + static_cast<int64_t>(hh) * a.T * kPxDH;
  const uint16_t* vv_h = a.vv + static_cast<int64_t>(hh) * a.T * kPxDH;
  auto lds_ptr = [](unsigned char* p) { return (__attribute__((address_space(3))) void*)p; };
  auto issue_tile = [&](int tile, unsigned char* base) {
    // buffer resources from the tile's first key (offsets within the tile's rows)
    const int t0 = kbeg + tile * kPxKeys;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(kc_h + static_cast<int64_t>(t0) * kPxDH), 0, kPxKeys * kPxKcRow, kBufRsrcWord3);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(vv_h + static_cast<int64_t>(t0) * kPxDH), 0, kPxKeys * kPxKcRow, kBufRsrcWord3);
    const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(a.latent + static_cast<int64_t>(t0) * DQ + a.DC), 0, kPxKeys * DQ * 2, kBufRsrcWord3);
#pragma unroll
    for (int j = 0; j < NKI; ++j) {
      const int I = NKI * w + j, key = 4 * I + (lane >> 4), piece = (lane & 15) ^ pf_lat_swz(key);
      const int off = (key_at(tile, key) - t0) * kPxKcRow + 16 * piece;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, lds_ptr(base + 4 * I * kPxKcRow), 16, off, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, lds_ptr(base + kPxVOff + 4 * I * kPxKcRow), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < NRI; ++j) {
      const int I = NRI * w + j, key = 8 * I + (lane >> 3), piece = (lane & 7) ^ pf_rope_swz(key);
      const int off = (key_at(tile, key) - t0) * DQ * 2 + 16 * piece;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rr, lds_ptr(base + kPxRopeOff + 8 * I * kPxRopeRow), 16, off, 0, 0, 0);
    }
  };
  // the tile's copies have landed (this wave's); the barrier after it covers every wave's
  auto tile_landed = []() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); };

  // per-lane LDS offsets (bytes within a tile buffer)
  const int off_sk = r32 * kPxKcRow;                // score A: key row 32 kb + r32
  const int swz_sk = pf_lat_swz(r32);
  const int off_sr = kPxRopeOff + r32 * kPxRopeRow;
  const int swz_sr = pf_rope_swz(r32);
  // value A (transposed reads): rows 16 m + 4 h + r16 / 4 (+ 8), byte 8 (r16 % 2) of the piece
  const int off_v = kPxVOff + (4 * h + (r16 >> 2)) * kPxKcRow + 8 * (r16 & 1);
  const int vlo = 2 * R1 + ((r16 & 3) >> 1);  // low 2 bits of the logical piece

  pf_f32x16_t o[kPxDH / 32];
#pragma unroll
  for (int db = 0; db < kPxDH / 32; ++db)
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
    const int k_lo = kbeg + i * kPxKeys;

    // ---- scores S^T[key][row] for keys k_lo + 32 kb + (0..31) ----
    pf_f32x16_t s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
    for (int c = 0; c < kPxDH / 16; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const f16x8_t av = *reinterpret_cast<const f16x8_t*>(tb + off_sk + 32 * kb * kPxKcRow +
                                                              16 * ((2 * c + h) ^ swz_sk));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(av, qv[c], s[kb], 0, 0, 0);
      }
#pragma unroll
    for (int c = 0; c < kPxDR / 16; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(tb + off_sr + 32 * kb * kPxRopeRow +
                                                                16 * ((2 * c + h) ^ swz_sr));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, qr[c], s[kb], 0, 0, 0);
      }
    // issue order: the A operands of a chunk (both key blocks) two chunks ahead
    // of its two products, so that each pair of products waits for reads issued
    // two pairs earlier
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int c = 0; c < (kPxDH + kPxDR) / 16 - 1 - 1; ++c) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    // keys outside [s_row, t_row] only in tiles that reach past the block's
    // first token or start before its latest sequence start
    if (k_lo + kPxKeys - 1 > q0 || k_lo < s_max) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k_lo + 32 * kb + 8 * (r >> 2) + 4 * h + (r & 3);
          if (key < s_row || key > t_c) s[kb][r] = -INFINITY;
        }
    }

    // ---- online softmax (row = lane % 32; keys split between lanes L and L ^ 32) ----
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
      for (int db = 0; db < kPxDH / 32; ++db) o[db] *= alpha;
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

    // ---- values O^T[dim][row] += V^T P^T ----
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const unsigned char* vp = tb + off_v + (32 * kb + 16 * m) * kPxKcRow;
#pragma unroll
        for (int db = 0; db < kPxDH / 32; ++db) {
          // logical piece 4 db + vlo; rows +0 and +8 swizzle with 4 (r16 / 4) + h and + 2
          const int p0 = 4 * (db ^ (r16 >> 2)) + (vlo ^ h);
          const int p1 = 4 * (db ^ (r16 >> 2)) + (vlo ^ (h + 2));
          const s16x4_t a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(vp + 16 * p0));
          const s16x4_t a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) s16x4_t*)(vp + 8 * kPxKcRow + 16 * p1));
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

  // ---- out = O / l in bf16: lane holds dims 32 db + 8 q + 4 h + 0..3 of its row ----
  const float inv = 1.0f / pf_pair_sum(l_run);
  if (row_ok) {
    uint16_t* orow = a.out + (static_cast<int64_t>(t_row) * a.H + hh) * kPxDH + 4 * h;
#pragma unroll
    for (int db = 0; db < kPxDH / 32; ++db)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<u32x2_t*>(orow + 32 * db + 8 * q) =
            u32x2_t{pack_bf16x2(o[db][4 * q] * inv, o[db][4 * q + 1] * inv),
                    pack_bf16x2(o[db][4 * q + 2] * inv, o[db][4 * q + 3] * inv)};
  }
}

}  // namespace egmla
