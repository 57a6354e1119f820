// Gate rows from the token embedding on gfx950 (Sec. 3.1 Eq. (3)-(4)):
//   out[i, :] = W^UE Emb[ids[i], :]        (e = emb_dim in, d_c out, fp32 sums)
// Over every vocabulary id this is the offline fold G = Emb W^UE^T of the
// table-lookup variant (Sec. 5.2) that the decode takes as its gate table;
// over the ids of a step's context it is the unfolded model's own gate
// computation.
//
// MFMA kernel (bf16, e a multiple of 128, d_c a multiple of 32): a slice of
// CB = 32 NCB rows of W^UE (output columns) sits in LDS for the whole kernel
// (rows padded by 16 bytes, so the 16 lanes of an LDS read cycle hit 16
// distinct 4-bank groups; slice rows past d_c are zero).  Each of the 8 waves
// takes 32 output rows at a time: their embedding rows go straight from HBM
// into registers as the B operand of v_mfma_f32_32x32x16_bf16 (lane: row
// lane%32, components 16c + 8(lane/32) .. +7 of chunk c), and each A fragment
// read from LDS (output column lane%32, the same components) feeds 32 rows.
// The accumulator holds out^T, so a lane stores 4 consecutive columns of one
// row at a time.  For e <= 512 a block's components all sit in registers: its
// loads go out together at the top of the block (the next block's row ids one
// block ahead), and the other wave on the SIMD computes while they travel.
// Issuing them earlier, at the end of the previous block, measured slower.
// Larger e takes passes of 256 (or 128) components.
//
// Work-groups are persistent and grouped by XCD: with S column slices, the S
// work-groups that share a set of row blocks are launched onto one XCD
// (work-groups go to the 8 XCDs round-robin), so an embedding row that the
// first of them fetches is in that XCD's L2 for the others.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr int kGateThreads = 256;        // VALU kernel
constexpr int kGateWaves = 8;            // MFMA kernel: waves per work-group (2 per SIMD)
constexpr int kGateLdsBudget = 150 * 1024;  // bytes of W^UE slice in LDS, at most


typedef __attribute__((ext_vector_type(16))) float gate_f32x16_t;

// One half-pass of a 32-row block: chunks 0 .. NH-1 of bq against W^UE
// components k0 + 16 c, with each slice's A fragment read one chunk ahead.
template <int NH, int NCB>
__device__ __forceinline__ void gate_products(const bf16x8_t (&bq)[NH], const uint16_t* arow, int RS, int k0,
                                              gate_f32x16_t (&acc)[NCB]) {
  bf16x8_t a_cur[NCB], a_nxt[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) a_cur[cb] = *reinterpret_cast<const bf16x8_t*>(arow + cb * 32 * RS + k0);
#pragma unroll
  for (int c = 0; c < NH; ++c) {
    if (c + 1 < NH) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        a_nxt[cb] = *reinterpret_cast<const bf16x8_t*>(arow + cb * 32 * RS + k0 + 16 * (c + 1));
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
      acc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a_cur[cb], bq[c], acc[cb], 0, 0, 0);
    // the next chunk's LDS reads go out first, then this chunk's products
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) a_cur[cb] = a_nxt[cb];
  }
}

// Stores a finished 32-row block: lane holds out^T[column 32 cb + 8 q + 4 h + t][row]
// in acc[cb][4 q + t].
template <int NCB>
__device__ __forceinline__ void gate_store(const gate_f32x16_t (&acc)[NCB], uint16_t* out, int64_t orow, bool live,
                                           int DC, int c0, int nc, int h) {
  if (!live) return;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
    if (32 * cb < nc) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<u32x2_t*>(out + orow * DC + c0 + 32 * cb + 8 * q + 4 * h) =
            u32x2_t{pack_bf16x2(acc[cb][4 * q], acc[cb][4 * q + 1]),
                    pack_bf16x2(acc[cb][4 * q + 2], acc[cb][4 * q + 3])};
    }
}

// TABLE: `ids` is the list of distinct ids that gate_claim_kernel built, its
// length counts[parity] (read on the device; n bounds it), and row i writes
// out[ids[i]], a [V, d_c] table.  Thread 0 zeroes counts[parity ^ 1], the
// slot of the next call.
template <int EP, int NCB, bool ONE_PASS, bool TABLE = false>
__global__ __launch_bounds__(64 * kGateWaves, 1) void gate_rows_mfma_kernel(const int32_t* __restrict__ ids,
                                                                            const uint16_t* __restrict__ emb,
                                                                            const uint16_t* __restrict__ w_ue,
                                                                            uint16_t* __restrict__ out, int64_t n,
                                                                            int E, int DC, int V, int S,
                                                                            unsigned int* __restrict__ counts,
                                                                            unsigned int parity) {
  if constexpr (TABLE) {
    n = min(n, static_cast<int64_t>(counts[parity]));
    if (blockIdx.x == 0 && threadIdx.x == 0) counts[parity ^ 1u] = 0u;
  }
  if (n <= 0) return;  // uniform over the work-group
  constexpr int CB = 32 * NCB;
  constexpr int NC = EP / 16;  // 16-component chunks per pass
  extern __shared__ __attribute__((aligned(16))) uint16_t wl[];  // [CB][E + 8]
  const int RS = E + 8;
  const int tid = threadIdx.x;
  const int xcd = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int slice = j % S, team = (j / S) * 8 + xcd;
  const int nteams = gridDim.x / S;
  const int c0 = slice * CB;
  const int nc = min(CB, DC - c0);  // a multiple of 32

  const int lane = tid & 63, w = tid >> 6, i32 = lane & 31, h = lane >> 5;
  const int64_t nrb = (n + 31) / 32;
  const uint16_t* arow = wl + i32 * RS + 8 * h;
  // this work-group's blocks: team, team + nteams, ...; wave w takes every 8th of them
  const int64_t step = static_cast<int64_t>(nteams) * kGateWaves;
  int64_t rb = team + static_cast<int64_t>(nteams) * w;
  // a block's row ids; past the end of the rows (or of the blocks) the last row
  // repeats, so every load stays in bounds and nothing past n is stored
  auto row_id = [&](int64_t blk) { return clamp_id(ids[min(blk * 32 + i32, n - 1)], V); };
  auto erow_of = [&](int id) { return emb + static_cast<int64_t>(id) * E + 8 * h; };
  constexpr int NH = NC / 2;  // ONE_PASS: E == EP

  // the first block's ids travel while W^UE is staged
  const int id_first = row_id(min(rb, nrb - 1));
  const int per_row = E / 8;
  for (int p = tid; p < CB * per_row; p += 64 * kGateWaves) {
    const int r = p / per_row, k8 = (p % per_row) * 8;
    u32x4_t v = u32x4_t{0u, 0u, 0u, 0u};
    if (r < nc) v = *reinterpret_cast<const u32x4_t*>(w_ue + static_cast<int64_t>(c0 + r) * E + k8);
    *reinterpret_cast<u32x4_t*>(wl + r * RS + k8) = v;
  }
  bf16x8_t bA[NH], bB[NH];
  int id_next = id_first;
  __syncthreads();

  if constexpr (ONE_PASS) {
    for (; rb < nrb; rb += step) {
      const uint16_t* erow = erow_of(id_next);
      const int id_after = row_id(min(rb + step, nrb - 1));
      gate_f32x16_t acc[NCB];
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;
#pragma unroll
      for (int c = 0; c < NH; ++c) bA[c] = *reinterpret_cast<const bf16x8_t*>(erow + 16 * c);
#pragma unroll
      for (int c = 0; c < NH; ++c) bB[c] = *reinterpret_cast<const bf16x8_t*>(erow + 16 * (NH + c));
      __builtin_amdgcn_sched_barrier(0);
      gate_products<NH, NCB>(bA, arow, RS, 0, acc);
      gate_products<NH, NCB>(bB, arow, RS, 16 * NH, acc);
      gate_store<NCB>(acc, out, TABLE ? id_next : rb * 32 + i32, rb * 32 + i32 < n, DC, c0, nc, h);
      id_next = id_after;
    }
  } else {
  // e above one pass: each block takes E / EP passes, every load of a pass in flight at once
  for (; rb < nrb; rb += step) {
    const int id = row_id(rb);
    const uint16_t* erow = erow_of(id);
    gate_f32x16_t acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] = 0.f;
    for (int p0 = 0; p0 < E; p0 += EP) {
#pragma unroll
      for (int c = 0; c < NH; ++c) bA[c] = *reinterpret_cast<const bf16x8_t*>(erow + p0 + 16 * c);
#pragma unroll
      for (int c = 0; c < NH; ++c) bB[c] = *reinterpret_cast<const bf16x8_t*>(erow + p0 + 16 * (NH + c));
      __builtin_amdgcn_sched_barrier(0);
      gate_products<NH, NCB>(bA, arow, RS, p0, acc);
      gate_products<NH, NCB>(bB, arow, RS, p0 + 16 * NH, acc);
    }
    gate_store<NCB>(acc, out, TABLE ? id : rb * 32 + i32, rb * 32 + i32 < n, DC, c0, nc, h);
  }
  }
}

// Stamp slots one 128-byte line apart, so that claims of different ids do
// not queue on one line.
constexpr int kMarkStride = 32;
constexpr int kClaimThreads = 1024;

// Distinct ids of a list (pass 1 of eg_mla_gate_table): row i claims its id
// with an atomic exchange of `stamp` into marks[id kMarkStride]; a row that
// finds another value appends the id to `list`.  The work-group gathers its
// winners in LDS and reserves their places with one atomic add (the
// counter is one address: an add per wave queued ~2000 of them there).
// counts[stamp % 2] counts the list and must be zero on entry; the pass over
// the list zeroes the other slot for the next call.
__global__ __launch_bounds__(kClaimThreads) void gate_claim_kernel(const int32_t* __restrict__ ids, int64_t n, int V,
                                                                   unsigned int* __restrict__ marks,
                                                                   unsigned int stamp, int32_t* __restrict__ list) {
  __shared__ unsigned int wave_n[kClaimThreads / 64];
  __shared__ unsigned int wg_base;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kClaimThreads + threadIdx.x;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int id = 0;
  bool win = false;
  if (i < n) {
    id = clamp_id(ids[i], V);
    win = atomicExch(marks + static_cast<int64_t>(id) * kMarkStride, stamp) != stamp;
  }
  const uint64_t mask = __builtin_amdgcn_ballot_w64(win);
  if (lane == 0) wave_n[w] = static_cast<unsigned int>(__builtin_popcountll(mask));
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned int tot = 0;
    for (int k = 0; k < kClaimThreads / 64; ++k) tot += wave_n[k];
    wg_base = tot > 0 ? atomicAdd(marks + static_cast<int64_t>(V) * kMarkStride + (stamp & 1u), tot) : 0u;
  }
  __syncthreads();
  unsigned int before = wg_base;
  for (int k = 0; k < w; ++k) before += wave_n[k];
  const unsigned int pos = before + static_cast<unsigned int>(__builtin_popcountll(mask & ((uint64_t{1} << lane) - 1)));
  if (win && pos < static_cast<unsigned int>(V)) list[pos] = id;  // a counter left nonzero cannot overrun
}

// TABLE: row i writes out[ids[i]] (rows with the same id write the same bits)
template <bool BF16, bool TABLE = false>
__global__ __launch_bounds__(kGateThreads) void gate_rows_valu_kernel(const int32_t* __restrict__ ids,
                                                                       const void* __restrict__ emb,
                                                                       const void* __restrict__ w_ue,
                                                                       void* __restrict__ out, int E, int DC, int V) {
  extern __shared__ float erow[];  // [E]
  const int64_t i = blockIdx.x;
  const int id = clamp_id(ids[i], V);
  for (int k = threadIdx.x; k < E; k += kGateThreads) erow[k] = ld<BF16>(emb, static_cast<int64_t>(id) * E + k);
  __syncthreads();
  const int c = blockIdx.y * kGateThreads + threadIdx.x;
  if (c >= DC) return;
  float acc = 0.f;
  for (int k = 0; k < E; ++k) acc = fmaf(ld<BF16>(w_ue, static_cast<int64_t>(c) * E + k), erow[k], acc);
  st<BF16>(out, (TABLE ? static_cast<int64_t>(id) : i) * DC + c, acc);
}

}  // namespace egmla

using namespace egmla;

namespace {

// Column slices and LDS of the MFMA kernel for this shape (0 slices: the VALU
// kernel runs).
struct GateShape {
  int ncb = 0, S = 0, ep = 0;
  bool one = false;
  size_t lds = 0;
};

GateShape gate_shape(const eg_mla_dims& d, int E) {
  GateShape g;
  const int DC = d.latent_dim;
  // slice width: as many 32-column blocks (up to 4) as d_c needs and the LDS holds
  int ncb = DC >= 96 ? 4 : (DC >= 64 ? 2 : 1);
  while (ncb > 1 && static_cast<int64_t>(32 * ncb) * (E + 8) * 2 > kGateLdsBudget) ncb /= 2;
  if (!(d.dtype == EG_MLA_BF16 && E % 128 == 0 && DC % 32 == 0 &&
        static_cast<int64_t>(32 * ncb) * (E + 8) * 2 <= kGateLdsBudget))
    return g;
  g.S = (DC + 32 * ncb - 1) / (32 * ncb);
  // one pass when the whole embedding row fits the registers (e <= 512),
  // else passes of 256 (or 128) components
  g.one = E <= 512;
  g.ep = g.one ? E : (E % 256 == 0 ? 256 : 128);
  if (g.one && ncb == 1) ncb = 2;  // d_c 32: a padded 64-column slice (fits: e <= 512)
  g.ncb = ncb;
  g.lds = static_cast<size_t>(32 * ncb) * (E + 8) * 2;
  return g;
}

eg_mla_status launch_gate(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n, const int32_t* ids,
                          const void* emb, const void* w_ue, void* out, bool table, unsigned int* marks,
                          unsigned int stamp, void* stream_) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  (void)hipGetLastError();
  const int E = emb_dim, DC = dims->latent_dim;
  const bool bf = dims->dtype == EG_MLA_BF16;
  const GateShape gs = gate_shape(*dims, E);
  const bool mfma = gs.S > 0 && reinterpret_cast<uintptr_t>(emb) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(w_ue) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 8 == 0;
  unsigned int* counts = nullptr;
  if (mfma && table) {
    // pass 1: the distinct ids into a list (marks: [V] stamp lines, [2] counts, [V] list)
    if (n > (int64_t{1} << 40)) return EG_MLA_ERR_UNSUPPORTED;
    unsigned int* cnt = marks + static_cast<int64_t>(emb_vocab) * kMarkStride;
    int32_t* list = reinterpret_cast<int32_t*>(cnt + 2);
    hipLaunchKernelGGL(gate_claim_kernel, dim3(static_cast<unsigned>((n + kClaimThreads - 1) / kClaimThreads)),
                       dim3(kClaimThreads), 0, stream, ids, n, emb_vocab, marks, stamp, list);
    counts = cnt;
    ids = list;
    n = std::min<int64_t>(n, emb_vocab);  // the list holds distinct ids only
  }
  if (mfma) {
    const int S = gs.S, ncb = gs.ncb, ep = gs.ep;
    const bool one = gs.one;
    const int64_t nrb = (n + 31) / 32;
    // one work-group per compute unit: 8 XCDs x k teams x S slices, with no
    // more teams than give each of a work-group's waves a row block
    const int per_xcd = std::max(1, device_cus() / 8 / S);
    // (the distinct-id pass too: 2 or 4 blocks per wave measured slower, each
    // work-group staging its W^UE slice first)
    const int64_t want = (nrb + kGateWaves - 1) / kGateWaves;
    const int k = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(per_xcd, (want + 7) / 8)));
    const int grid = 8 * k * S;
    const size_t lds = gs.lds;
    const void* fn = nullptr;
#define EGMLA_GATE_CASE(EPV, NCBV, ONE)                                                                    \
    if (ep == EPV && ncb == NCBV && one == ONE)                                                           \
      fn = table ? reinterpret_cast<const void*>(gate_rows_mfma_kernel<EPV, NCBV, ONE, true>)              \
                 : reinterpret_cast<const void*>(gate_rows_mfma_kernel<EPV, NCBV, ONE, false>);
    EGMLA_GATE_CASE(512, 4, true) EGMLA_GATE_CASE(512, 2, true)
    EGMLA_GATE_CASE(384, 4, true) EGMLA_GATE_CASE(384, 2, true)
    EGMLA_GATE_CASE(256, 4, true) EGMLA_GATE_CASE(256, 2, true)
    EGMLA_GATE_CASE(128, 4, true) EGMLA_GATE_CASE(128, 2, true)
    EGMLA_GATE_CASE(256, 4, false) EGMLA_GATE_CASE(256, 2, false) EGMLA_GATE_CASE(256, 1, false)
    EGMLA_GATE_CASE(128, 4, false) EGMLA_GATE_CASE(128, 2, false) EGMLA_GATE_CASE(128, 1, false)
#undef EGMLA_GATE_CASE
    if (fn == nullptr) return EG_MLA_ERR_UNSUPPORTED;
    if (lds > 65536 &&
        hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)) != hipSuccess)
      return EG_MLA_ERR_HIP;
    const int32_t* ids_c = ids;
    const uint16_t* emb_c = static_cast<const uint16_t*>(emb);
    const uint16_t* w_c = static_cast<const uint16_t*>(w_ue);
    uint16_t* out_c = static_cast<uint16_t*>(out);
    int V = emb_vocab, Ev = E, DCv = DC, Sv = S;
    unsigned int* counts_c = counts;
    unsigned int parity = stamp & 1u;
    void* args[] = {&ids_c, &emb_c, &w_c, &out_c, &n, &Ev, &DCv, &V, &Sv, &counts_c, &parity};
    if (hipLaunchKernel(fn, dim3(grid), dim3(64 * kGateWaves), args, lds, stream) != hipSuccess)
      return EG_MLA_ERR_HIP;
  } else {
    if (n > 0x7fffffff) return EG_MLA_ERR_UNSUPPORTED;
    const size_t lds = static_cast<size_t>(E) * sizeof(float);
    dim3 grid(static_cast<unsigned>(n), (DC + kGateThreads - 1) / kGateThreads);
    const void* fn = bf ? (table ? reinterpret_cast<const void*>(gate_rows_valu_kernel<true, true>)
                                 : reinterpret_cast<const void*>(gate_rows_valu_kernel<true, false>))
                        : (table ? reinterpret_cast<const void*>(gate_rows_valu_kernel<false, true>)
                                 : reinterpret_cast<const void*>(gate_rows_valu_kernel<false, false>));
    if (lds > 65536 &&
        hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)) != hipSuccess)
      return EG_MLA_ERR_HIP;
    int Ev = E, DCv = DC, V = emb_vocab;
    const int32_t* ids_c = ids;
    const void* emb_c = emb;
    const void* w_c = w_ue;
    void* out_c = out;
    void* args[] = {&ids_c, &emb_c, &w_c, &out_c, &Ev, &DCv, &V};
    if (hipLaunchKernel(fn, grid, dim3(kGateThreads), args, lds, stream) != hipSuccess) return EG_MLA_ERR_HIP;
  }
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}

}  // namespace

extern "C" eg_mla_status eg_mla_gate_rows(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                          const int32_t* ids, const void* emb, const void* w_ue, void* out,
                                          void* stream) {
  eg_mla_status st = validate_gate_rows(dims, emb_dim, emb_vocab, n, ids, emb, w_ue, out);
  if (st != EG_MLA_OK || n == 0) return st;
  return launch_gate(dims, emb_dim, emb_vocab, n, ids, emb, w_ue, out, false, nullptr, 0u, stream);
}

extern "C" size_t eg_mla_gate_table_marks_size(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab) {
  if (validate_gate_rows(dims, emb_dim, emb_vocab, 0, nullptr, nullptr, nullptr, nullptr) != EG_MLA_OK) return 0;
  // a stamp line per id, two counts, the id list
  return ((kMarkStride + 1) * static_cast<size_t>(emb_vocab) + 2) * sizeof(unsigned int);
}

extern "C" eg_mla_status eg_mla_gate_table(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                           const int32_t* ids, const void* emb, const void* w_ue, void* table,
                                           void* marks, size_t marks_bytes, uint32_t stamp, void* stream) {
  eg_mla_status st = validate_gate_rows(dims, emb_dim, emb_vocab, n, ids, emb, w_ue, table);
  if (st != EG_MLA_OK) return st;
  if (stamp == 0) return EG_MLA_ERR_INVALID_ARG;
  if (n == 0) return EG_MLA_OK;
  if (!marks || reinterpret_cast<uintptr_t>(marks) % 4 != 0 ||
      marks_bytes < eg_mla_gate_table_marks_size(dims, emb_dim, emb_vocab))
    return EG_MLA_ERR_WORKSPACE;
  return launch_gate(dims, emb_dim, emb_vocab, n, ids, emb, w_ue, table, true, static_cast<unsigned int*>(marks),
                     stamp, stream);
}
