// Gate rows from the token embedding on gfx950 (Sec. 3.1 Eq. (3)-(4)):
//   out[i, :] = W^UE Emb[ids[i], :]        (e = emb_dim in, d_c out, fp32 sums)
// Over every vocabulary id this is the offline fold G = Emb W^UE^T of the
// table-lookup variant (Sec. 5.2) that the decode takes as its gate table;
// over the ids of a step's context it is the unfolded model's own gate
// computation.
//
// MFMA kernel (bf16, e a multiple of 32, d_c a multiple of 16): a work-group
// of 4 waves stages a slice of CB <= 128 rows of W^UE (output columns) in LDS
// (rows padded by 16 bytes) and keeps it for all of its row blocks.  A wave
// takes 16 output rows at a time: their embedding rows are gathered straight
// into registers as the B operand of v_mfma_f32_16x16x32_bf16 (lane: row
// lane%16, 8 consecutive embedding components), the A operand is the W^UE
// slice read from LDS (lane: output column lane%16, the same 8 components),
// so the accumulator holds out^T[column][row] and each lane stores 4
// consecutive columns of one row.  Other shapes and fp32 storage take the
// VALU kernel (one thread per output element, the embedding row in LDS).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr int kGateThreads = 256;
constexpr int kGateMaxCB = 128;          // output columns per work-group slice
constexpr int kGateLdsBudget = 147456;   // bytes of W^UE slice in LDS, at most
constexpr int kGateKSeg = 16;            // 32-component chunks of embedding held per pass (512 components)

__global__ __launch_bounds__(kGateThreads) void gate_rows_mfma_kernel(const int32_t* __restrict__ ids,
                                                                       const uint16_t* __restrict__ emb,
                                                                       const uint16_t* __restrict__ w_ue,
                                                                       uint16_t* __restrict__ out, int64_t n,
                                                                       int E, int DC, int CB, int V) {
  extern __shared__ __attribute__((aligned(16))) uint16_t wl[];  // [CB][E + 8]
  const int RS = E + 8;
  const int c0 = blockIdx.y * CB;
  const int nc = min(CB, DC - c0);  // multiple of 16
  const int tid = threadIdx.x, lane = tid & 63, r16 = lane & 15, g = lane >> 4;
  const int w = tid >> 6;

  // stage W^UE rows c0 .. c0 + nc - 1 (16 bytes per thread per step)
  const int pieces = nc * (E / 8);
  for (int p = tid; p < pieces; p += kGateThreads) {
    const int r = p / (E / 8), k8 = (p % (E / 8)) * 8;
    *reinterpret_cast<u32x4_t*>(wl + r * RS + k8) =
        *reinterpret_cast<const u32x4_t*>(w_ue + static_cast<int64_t>(c0 + r) * E + k8);
  }
  __syncthreads();

  const int ncb = nc / 16;
  const int64_t nrb = (n + 15) / 16;
  for (int64_t rb = static_cast<int64_t>(blockIdx.x) * 4 + w; rb < nrb; rb += static_cast<int64_t>(gridDim.x) * 4) {
    const int64_t row = min(rb * 16 + r16, n - 1);  // past the end: repeats the last row (not stored)
    const int id = clamp_id(ids[row], V);
    const uint16_t* erow = emb + static_cast<int64_t>(id) * E + 8 * g;
    f32x4_t acc[kGateMaxCB / 16];
#pragma unroll
    for (int cb = 0; cb < kGateMaxCB / 16; ++cb) acc[cb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < E; k0 += 32 * kGateKSeg) {
      const int nk = min(kGateKSeg, (E - k0) / 32);  // uniform
      bf16x8_t bq[kGateKSeg];
#pragma unroll
      for (int kc = 0; kc < kGateKSeg; ++kc)
        if (kc < nk) bq[kc] = *reinterpret_cast<const bf16x8_t*>(erow + k0 + 32 * kc);
#pragma unroll
      for (int cb = 0; cb < kGateMaxCB / 16; ++cb) {
        if (cb < ncb) {
          const uint16_t* arow = wl + (cb * 16 + r16) * RS + k0 + 8 * g;
#pragma unroll
          for (int kc = 0; kc < kGateKSeg; ++kc)
            if (kc < nk)
              acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*reinterpret_cast<const bf16x8_t*>(arow + 32 * kc),
                                                                bq[kc], acc[cb], 0, 0, 0);
        }
      }
    }
    // lane holds out^T[column cb*16 + 4g + q][row r16]
    const int64_t orow = rb * 16 + r16;
    if (orow < n) {
#pragma unroll
      for (int cb = 0; cb < kGateMaxCB / 16; ++cb)
        if (cb < ncb)
          *reinterpret_cast<u32x2_t*>(out + orow * DC + c0 + cb * 16 + 4 * g) =
              u32x2_t{pack_bf16x2(acc[cb][0], acc[cb][1]), pack_bf16x2(acc[cb][2], acc[cb][3])};
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
  const int cb = std::min({DC, kGateMaxCB, 16 * (kGateLdsBudget / (16 * (E + 8) * 2))});
  const bool mfma = bf && E % 32 == 0 && DC % 16 == 0 && cb >= 16 && reinterpret_cast<uintptr_t>(emb) % 16 == 0 &&
                    reinterpret_cast<uintptr_t>(w_ue) % 16 == 0 && reinterpret_cast<uintptr_t>(out) % 8 == 0;
  if (mfma) {
    const int slices = (DC + cb - 1) / cb;
    const int64_t nrb = (n + 15) / 16;
    // one work-group per compute unit over all slices (the W^UE slice fills
    // most of the LDS), each keeping its slice for many row blocks
    const int64_t want = std::max<int64_t>(1, 256 / slices);
    const int rows_wg = static_cast<int>(std::min<int64_t>((nrb + 3) / 4, want));
    const size_t lds = static_cast<size_t>(cb) * (E + 8) * 2;
    if (lds > 65536 &&
        hipFuncSetAttribute(reinterpret_cast<const void*>(gate_rows_mfma_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds)) != hipSuccess)
      return EG_MLA_ERR_HIP;
    hipLaunchKernelGGL(gate_rows_mfma_kernel, dim3(rows_wg, slices), dim3(kGateThreads), lds, stream, ids,
                       static_cast<const uint16_t*>(emb), static_cast<const uint16_t*>(w_ue),
                       static_cast<uint16_t*>(out), n, E, DC, cb, emb_vocab);
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
