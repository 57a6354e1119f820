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
__device__ __forceinline__ void gate_store(const gate_f32x16_t (&acc)[NCB], uint16_t* out, int64_t orow, int64_t n,
                                           int DC, int c0, int nc, int h) {
  if (orow >= n) return;
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

template <int EP, int NCB, bool ONE_PASS>
__global__ __launch_bounds__(64 * kGateWaves, 1) void gate_rows_mfma_kernel(const int32_t* __restrict__ ids,
                                                                            const uint16_t* __restrict__ emb,
                                                                            const uint16_t* __restrict__ w_ue,
                                                                            uint16_t* __restrict__ out, int64_t n,
                                                                            int E, int DC, int V, int S) {
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
      gate_store<NCB>(acc, out, rb * 32 + i32, n, DC, c0, nc, h);
      id_next = id_after;
    }
  } else {
  // e above one pass: each block takes E / EP passes, every load of a pass in flight at once
  for (; rb < nrb; rb += step) {
    const uint16_t* erow = erow_of(row_id(rb));
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
    gate_store<NCB>(acc, out, rb * 32 + i32, n, DC, c0, nc, h);
  }
  }
}

template <bool BF16>
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
  st<BF16>(out, i * DC + c, acc);
}

}  // namespace egmla

using namespace egmla;

extern "C" eg_mla_status eg_mla_gate_rows(const eg_mla_dims* dims, int32_t emb_dim, int32_t emb_vocab, int64_t n,
                                          const int32_t* ids, const void* emb, const void* w_ue, void* out,
                                          void* stream_) {
  eg_mla_status st = validate_gate_rows(dims, emb_dim, emb_vocab, n, ids, emb, w_ue, out);
  if (st != EG_MLA_OK || n == 0) return st;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  (void)hipGetLastError();
  const int E = emb_dim, DC = dims->latent_dim;
  const bool bf = dims->dtype == EG_MLA_BF16;
  // slice width: as many 32-column blocks (up to 4) as d_c needs and the LDS holds
  int ncb = DC >= 96 ? 4 : (DC >= 64 ? 2 : 1);
  while (ncb > 1 && static_cast<int64_t>(32 * ncb) * (E + 8) * 2 > kGateLdsBudget) ncb /= 2;
  const bool mfma = bf && E % 128 == 0 && DC % 32 == 0 && static_cast<int64_t>(32 * ncb) * (E + 8) * 2 <= kGateLdsBudget &&
                    reinterpret_cast<uintptr_t>(emb) % 16 == 0 && reinterpret_cast<uintptr_t>(w_ue) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(out) % 8 == 0;
  if (mfma) {
    const int S = (DC + 32 * ncb - 1) / (32 * ncb);
    const int64_t nrb = (n + 31) / 32;
    // one work-group per compute unit: 8 XCDs x k teams x S slices, with no
    // more teams than give each of a work-group's waves a row block
    const int per_xcd = std::max(1, device_cus() / 8 / S);
    const int64_t want = (nrb + kGateWaves - 1) / kGateWaves;
    const int k = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(per_xcd, (want + 7) / 8)));
    const int grid = 8 * k * S;
    // one pass when the whole embedding row fits the registers (e <= 512),
    // else passes of 256 (or 128) components
    const bool one = E <= 512;
    const int ep = one ? E : (E % 256 == 0 ? 256 : 128);
    if (one && ncb == 1) ncb = 2;  // d_c 32: a padded 64-column slice (fits: e <= 512)
    const size_t lds = static_cast<size_t>(32 * ncb) * (E + 8) * 2;
    const void* fn = nullptr;
#define EGMLA_GATE_CASE(EPV, NCBV, ONE)                                                  \
    if (ep == EPV && ncb == NCBV && one == ONE) fn = reinterpret_cast<const void*>(gate_rows_mfma_kernel<EPV, NCBV, ONE>);
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
    int V = emb_vocab;
    void* args[] = {&ids_c, &emb_c, &w_c, &out_c, &n, const_cast<int*>(&E), const_cast<int*>(&DC), &V,
                    const_cast<int*>(&S)};
    if (hipLaunchKernel(fn, dim3(grid), dim3(64 * kGateWaves), args, lds, stream) != hipSuccess)
      return EG_MLA_ERR_HIP;
  } else {
    if (n > 0x7fffffff) return EG_MLA_ERR_UNSUPPORTED;
    const size_t lds = static_cast<size_t>(E) * sizeof(float);
    dim3 grid(static_cast<unsigned>(n), (DC + kGateThreads - 1) / kGateThreads);
    if (bf) {
      if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(gate_rows_valu_kernel<true>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds)) != hipSuccess)
        return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(gate_rows_valu_kernel<true>, grid, dim3(kGateThreads), lds, stream, ids, emb, w_ue, out,
                         E, DC, emb_vocab);
    } else {
      if (lds > 65536 && hipFuncSetAttribute(reinterpret_cast<const void*>(gate_rows_valu_kernel<false>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize,
                                             static_cast<int>(lds)) != hipSuccess)
        return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(gate_rows_valu_kernel<false>, grid, dim3(kGateThreads), lds, stream, ids, emb, w_ue, out,
                         E, DC, emb_vocab);
    }
  }
  return hipGetLastError() == hipSuccess ? EG_MLA_OK : EG_MLA_ERR_HIP;
}
