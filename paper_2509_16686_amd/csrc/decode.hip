// EG-MLA decode on gfx950: absorbed-MLA attention over a latent KV cache with
// the token-specific embedding gate applied to each cached latent.
//
// Per call (all on the caller's stream):
//   1. absorb        q_lat[b,h] = W_UK[h]^T q^C[b,h]  (fp32), copied next to q^R
//   2. split kernel  one work-group per (sequence, context split, head group):
//                    stream cached rows, gate them by G[token id], scores,
//                    online softmax (log2 domain), latent-space value sum
//                    -> partial (max, sum, o_lat) per head
//   3. combine       log-sum-exp merge of the splits, o_lat / l, then W_UV[h]
//
// The math is App. C Eq. (C.11)-(C.13) in absorbed form with the gate of
// Sec. 3.1 Eq. (3)-(5) applied in the latent space (c~ = c * G[id]).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdlib>
#include <cfloat>
#include <cmath>
#include <mutex>

#include "device_common.h"
#include "eg_mla.h"
#include "host_plan.h"

namespace egmla {

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// 1. absorption: qfull[b,h,:] = [W_UK[h]^T q^C[b,h] | q^R[b,h]]   (fp32)
// grid (H, ceil(DC / 64), ceil(B / 16)), 256 threads = 64 latent columns x
// 4 slices of the head dim.  Each W_UK row segment is read once per 16
// sequences with 128-byte coalesced loads; the 4 slices are summed in LDS.
// ---------------------------------------------------------------------------
constexpr int kAbsorbRows = 16;
constexpr int kAbsorbCols = 64;

template <bool BF16>
__global__ __launch_bounds__(256) void absorb_kernel(const void* __restrict__ q, const void* __restrict__ w_uk,
                                                     float* __restrict__ qfull, int B, int H, int DH, int DC,
                                                     int DR) {
  extern __shared__ float smem[];  // q rows [kAbsorbRows][DH], partial sums [4][kAbsorbRows][kAbsorbCols]
  float* q_s = smem;
  float* red = smem + kAbsorbRows * DH;
  const int h = blockIdx.x;
  const int c0 = blockIdx.y * kAbsorbCols;
  const int b0 = blockIdx.z * kAbsorbRows;
  const int nb = min(kAbsorbRows, B - b0);
  const int DQin = DH + DR;
  const int DQ = DC + DR;
  const int tid = threadIdx.x;
  for (int i = tid; i < kAbsorbRows * DH; i += 256) {
    const int bb = i / DH, k = i % DH;
    q_s[i] = bb < nb ? ld<BF16>(q, (static_cast<int64_t>(b0 + bb) * H + h) * DQin + k) : 0.f;
  }
  __syncthreads();
  const int cl = tid & (kAbsorbCols - 1);
  const int kq = tid / kAbsorbCols;  // 0..3
  const int c = c0 + cl;
  const int kper = (DH + 3) / 4;
  const int k_lo = kq * kper, k_hi = min(DH, k_lo + kper);
  float acc[kAbsorbRows];
#pragma unroll
  for (int bb = 0; bb < kAbsorbRows; ++bb) acc[bb] = 0.f;
  if (c < DC) {
    const int64_t wbase = static_cast<int64_t>(h) * DH * DC + c;
#pragma unroll 4
    for (int k = k_lo; k < k_hi; ++k) {
      const float wv = ld<BF16>(w_uk, wbase + static_cast<int64_t>(k) * DC);
#pragma unroll
      for (int bb = 0; bb < kAbsorbRows; ++bb) acc[bb] = fmaf(wv, q_s[bb * DH + k], acc[bb]);
    }
  }
#pragma unroll
  for (int bb = 0; bb < kAbsorbRows; ++bb) red[(kq * kAbsorbRows + bb) * kAbsorbCols + cl] = acc[bb];
  __syncthreads();
  for (int i = tid; i < kAbsorbRows * kAbsorbCols; i += 256) {
    const int bb = i / kAbsorbCols, cc = i % kAbsorbCols;
    if (bb < nb && c0 + cc < DC) {
      float v = 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) v += red[(j * kAbsorbRows + bb) * kAbsorbCols + cc];
      qfull[(static_cast<int64_t>(b0 + bb) * H + h) * DQ + c0 + cc] = v;
    }
  }
  if (blockIdx.y == 0) {
    for (int i = tid; i < nb * DR; i += 256) {
      const int bb = i / DR, r = i % DR;
      qfull[(static_cast<int64_t>(b0 + bb) * H + h) * DQ + DC + r] = ld<BF16>(q, (static_cast<int64_t>(b0 + bb) * H + h) * DQin + DH + r);
    }
  }
}

// Split-K bookkeeping shared by the split kernels.
struct SplitArgs {
  const float* qfull;         // [B, H, DQ] fp32; wide kernel: 16-bit [B, H, DQ] = [q_lat fp16 | q^R bf16]
  const void* cache;          // [num_slots, DQ]
  const int32_t* ids;         // [num_slots]
  const void* gate;           // [V, DC]
  const int32_t* seq_lens;    // [B]
  const int32_t* page_table;  // [B, max_pages] or null
  float* part_ml;             // [rows, H, 2]   rows: B * s_max, or the balanced schedule's rows
  float* part_o;              // [rows, H, DC]
  const int64_t* sched_hdr;   // balanced schedule (wide kernel): total tokens, work-groups
  const int2* wg_start;       // balanced schedule: (sequence, offset) where each work-group starts
  int64_t num_slots;
  int B, H, DC, DR, P, max_pages, V, cap, split, s_max, groups, hpg;
  float scale_log2;           // softmax scale * log2(e)
  // Absorption inside the d_c 128 split kernel (null qin: a kernel of its own ran before)
  const uint16_t* qin;        // query [B, H, DH + DR] (bf16)
  const uint16_t* w_uk;       // W_UK [H, DH, DC] (bf16)
  unsigned long long* qflags; // [B, groups, s_max]: stamp of the call whose absorbed heads a split has stored
  unsigned long long stamp;   // this call's stamp (never 0, never repeated within the process)
  int DH;
  int spin_limit;             // polls of the stamps before a work-group absorbs every head itself
};

// ---------------------------------------------------------------------------
// 2a. VALU split kernel: fp32 arithmetic, any shape, fp32 or bf16 storage.
// One work-group (256 threads) per (sequence, split, head block of hpg heads).
// LDS: q [hpg][DQ], gated tile [32][DQ+1], probabilities [hpg][32].
// ---------------------------------------------------------------------------
constexpr int kValuThreads = 256;
constexpr int kValuAcc = 32;  // latent accumulators per thread: hpg * DC <= 8192

template <bool BF16>
__global__ __launch_bounds__(kValuThreads) void split_valu_kernel(SplitArgs a) {
  extern __shared__ float smem[];
  const int DQ = a.DC + a.DR;
  const int TS = DQ + 1;  // padded tile row
  const int nblocks = gridDim.x;
  const int item = xcd_logical_block(blockIdx.x, nblocks);
  const int hb = item % a.groups;
  const int s = (item / a.groups) % a.s_max;
  const int b = item / (a.groups * a.s_max);
  const int L = clamp_len(a.seq_lens[b], a.cap);
  const int t0 = s * a.split;
  if (t0 >= L) return;
  const int t1 = min(t0 + a.split, L);
  const int h0 = hb * a.hpg;
  const int nh = min(a.hpg, a.H - h0);

  float* q_s = smem;                      // [hpg][DQ]
  float* tile = q_s + a.hpg * DQ;         // [32][TS]
  float* prob = tile + kTile * TS;        // [hpg][32]
  float* alpha_s = prob + a.hpg * kTile;  // [hpg]
  int64_t* slot_s = reinterpret_cast<int64_t*>(alpha_s + a.hpg + (a.hpg & 1));  // [32]
  int* id_s = reinterpret_cast<int*>(slot_s + kTile);                           // [32]

  const int tid = threadIdx.x;
  for (int i = tid; i < nh * DQ; i += kValuThreads) q_s[i] = a.qfull[(static_cast<int64_t>(b) * a.H + h0) * DQ + i];

  float acc[kValuAcc];
#pragma unroll
  for (int k = 0; k < kValuAcc; ++k) acc[k] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;  // owned by thread tid < nh
  const int npairs = nh * a.DC;

  for (int tt = t0; tt < t1; tt += kTile) {
    const int nt = min(kTile, t1 - tt);
    __syncthreads();  // previous tile fully consumed
    if (tid < nt) {
      const int64_t sl = cache_slot(a.page_table, b, tt + tid, a.P, a.max_pages, a.num_slots);
      slot_s[tid] = sl;
      id_s[tid] = clamp_id(a.ids[sl], a.V);
    }
    __syncthreads();
    // gated tile: c~ = c * G[id] on the latent part, RoPE key as is
    for (int e = tid; e < nt * DQ; e += kValuThreads) {
      const int t = e / DQ, d = e % DQ;
      float x = ld<BF16>(a.cache, slot_s[t] * DQ + d);
      if (d < a.DC) x *= ld<BF16>(a.gate, static_cast<int64_t>(id_s[t]) * a.DC + d);
      tile[t * TS + d] = x;
    }
    __syncthreads();
    // scores (log2 domain)
    for (int p = tid; p < nh * kTile; p += kValuThreads) {
      const int h = p / kTile, t = p % kTile;
      float sc = -INFINITY;
      if (t < nt) {
        float dot = 0.f;
        const float* qr = q_s + h * DQ;
        const float* tr = tile + t * TS;
        for (int d = 0; d < DQ; ++d) dot = fmaf(qr[d], tr[d], dot);
        sc = dot * a.scale_log2;
      }
      prob[h * kTile + t] = sc;
    }
    __syncthreads();
    // online softmax update, one thread per head
    if (tid < nh) {
      float mt = -INFINITY;
      for (int t = 0; t < nt; ++t) mt = fmaxf(mt, prob[tid * kTile + t]);
      const float m_new = fmaxf(m_run, mt);
      const float alpha = exp2f(m_run - m_new);
      float sum = 0.f;
      for (int t = 0; t < kTile; ++t) {
        const float pv = t < nt ? exp2f(prob[tid * kTile + t] - m_new) : 0.f;
        prob[tid * kTile + t] = pv;
        sum += pv;
      }
      l_run = l_run * alpha + sum;
      m_run = m_new;
      alpha_s[tid] = alpha;
    }
    __syncthreads();
    // latent-space value accumulation
#pragma unroll
    for (int k = 0; k < kValuAcc; ++k) {
      const int idx = tid + k * kValuThreads;
      if (idx < npairs) {
        const int h = idx / a.DC, d = idx % a.DC;
        float o = acc[k] * alpha_s[h];
        const float* pr = prob + h * kTile;
        for (int t = 0; t < nt; ++t) o = fmaf(pr[t], tile[t * TS + d], o);
        acc[k] = o;
      }
    }
  }
  const int64_t pbase = (static_cast<int64_t>(b) * a.s_max + s) * a.H + h0;
  if (tid < nh) {
    a.part_ml[(pbase + tid) * 2 + 0] = m_run;
    a.part_ml[(pbase + tid) * 2 + 1] = l_run;
  }
#pragma unroll
  for (int k = 0; k < kValuAcc; ++k) {
    const int idx = tid + k * kValuThreads;
    if (idx < npairs) a.part_o[pbase * a.DC + idx] = acc[k];
  }
}

// ---------------------------------------------------------------------------
// 2b. MFMA split kernel (bf16 storage, 16 heads per work-group): split_mfma.h
// ---------------------------------------------------------------------------
}  // namespace egmla
#include "split_mfma.h"
#include "split_slice.h"
#include "split_wide.h"
namespace egmla {

// ---------------------------------------------------------------------------
// 3. combine: merge the splits of (b, h) and apply W_UV[h].
// grid (H, B), 256 threads.
// ---------------------------------------------------------------------------
template <bool BF16>
__global__ __launch_bounds__(256) void combine_kernel(const float* __restrict__ part_ml,
                                                      const float* __restrict__ part_o,
                                                      const void* __restrict__ w_uv,
                                                      const int32_t* __restrict__ seq_lens, void* __restrict__ out,
                                                      int H, int DC, int DV, int cap, int split, int s_max,
                                                      int slices, const int2* __restrict__ seq_rows) {
  // s_max splits of `slices` partials each per sequence, or (balanced
  // schedule) the rows seq_rows[b] lists; a partial without tokens has
  // maximum -inf and contributes nothing
  extern __shared__ float smem[];  // o[DC], wgt[partials of one sequence]
  float* o_s = smem;
  float* wgt = smem + DC;
  const int h = blockIdx.x, b = blockIdx.y;
  const int L = clamp_len(seq_lens[b], cap);
  const int64_t obase = (static_cast<int64_t>(b) * H + h) * DV;
  const int ns = L == 0 ? 0 : seq_rows ? seq_rows[b].y : min((L + split - 1) / split, s_max) * slices;
  if (ns == 0) {
    for (int v = threadIdx.x; v < DV; v += blockDim.x) st<BF16>(out, obase + v, 0.f);
    return;
  }
  const int64_t row0 = seq_rows ? seq_rows[b].x : static_cast<int64_t>(b) * s_max * slices;
  // split weights exp2(m_s - M) / sum_s l_s exp2(m_s - M), computed by wave 0
  if (threadIdx.x < 64) {
    float M = -INFINITY;
    for (int sidx = threadIdx.x; sidx < ns; sidx += 64)
      M = fmaxf(M, part_ml[((row0 + sidx) * H + h) * 2]);
    M = wave_max(M);
    float Ls = 0.f;
    for (int sidx = threadIdx.x; sidx < ns; sidx += 64) {
      const int64_t k = ((row0 + sidx) * H + h) * 2;
      const float e = exp2f(part_ml[k] - M);
      wgt[sidx] = e;
      Ls += part_ml[k + 1] * e;
    }
    Ls = wave_sum(Ls);
    const float inv = 1.f / Ls;
    for (int sidx = threadIdx.x; sidx < ns; sidx += 64) wgt[sidx] *= inv;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < DC; c += blockDim.x) {
    float acc = 0.f;
    for (int sidx = 0; sidx < ns; ++sidx)
      acc = fmaf(wgt[sidx], part_o[((row0 + sidx) * H + h) * DC + c], acc);
    o_s[c] = acc;
  }
  __syncthreads();
  const int64_t wbase = static_cast<int64_t>(h) * DV * DC;
  for (int v = threadIdx.x; v < DV; v += blockDim.x) {
    float acc = 0.f;
    const int64_t rb = wbase + static_cast<int64_t>(v) * DC;
    for (int c = 0; c < DC; c += 4) {
      const float4 wv = ld4<BF16>(w_uv, rb + c);
      acc = fmaf(wv.x, o_s[c], acc);
      acc = fmaf(wv.y, o_s[c + 1], acc);
      acc = fmaf(wv.z, o_s[c + 2], acc);
      acc = fmaf(wv.w, o_s[c + 3], acc);
    }
    st<BF16>(out, obase + v, acc);
  }
}

}  // namespace egmla
#include "aux_mfma.h"
namespace egmla {

// ---------------------------------------------------------------------------
// host launch helpers
// ---------------------------------------------------------------------------
namespace {

template <typename K>
hipError_t set_lds(K kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             static_cast<int>(bytes));
}

// Id-sliced kernel: waves per work-group and units in flight per wave.
constexpr int kSliceWaves = 4;
#ifndef EGMLA_SLICE_DEPTH
#define EGMLA_SLICE_DEPTH 2
#endif
constexpr int kSliceDepth = EGMLA_SLICE_DEPTH;

template <int DC>
hipError_t launch_combine_dc(dim3 grid, hipStream_t stream, const float* pm, const float* po, const uint16_t* wv,
                             const int32_t* seq_lens, uint16_t* ov, int B, int H, int cap, int split, int s_max,
                             int slices, const int2* seq_rows, int spw) {
  // Small work-groups when every sequence's partials fit one merge batch and
  // the grid stays within two work-groups per compute unit (measured faster
  // there; many partials per sequence, or many work-groups, favour the
  // 16-wave kernel).
  const int64_t small_wg = static_cast<int64_t>(H) * ((B + kComb4Seq - 1) / kComb4Seq);
  if (!seq_rows && static_cast<int64_t>(s_max) * slices <= 8 && small_wg <= 512) {
    hipLaunchKernelGGL((combine4_kernel<DC, 128>), dim3(H, (B + kComb4Seq - 1) / kComb4Seq), dim3(256), 0, stream,
                       pm, po, wv, seq_lens, ov, B, H, cap, split, s_max, slices);
    return hipGetLastError();
  }
  const size_t lds = combine_lds_bytes(DC);
  if constexpr (DC == 512) {
    // the head-split kernel (balanced schedule) writes fp16 rows normalised by their sums
    if (seq_rows) {
      hipError_t e = set_lds(combine_wide_kernel, combine_wide_lds_bytes());
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL(combine_wide_kernel, dim3(H, (B + kCombWideSeq - 1) / kCombWideSeq),
                         dim3(kCombWideWaves * 64), combine_wide_lds_bytes(), stream, pm,
                         reinterpret_cast<const uint16_t*>(po), wv, seq_rows, ov, B, H);
      return hipGetLastError();
    }
  }
  hipError_t e = set_lds(combine_mfma_kernel<DC, 128>, lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((combine_mfma_kernel<DC, 128>), grid, dim3(kCombWaves * 64), lds, stream, pm, po, wv, seq_lens,
                     ov, B, H, cap, split, s_max, slices, seq_rows, spw);
  return hipGetLastError();
}

hipError_t launch_combine_mfma(int dc, dim3 grid, hipStream_t stream, const float* pm, const float* po,
                               const uint16_t* wv, const int32_t* seq_lens, uint16_t* ov, int B, int H, int cap,
                               int split, int s_max, int slices, const int2* seq_rows, int spw) {
  if (dc == 128)
    return launch_combine_dc<128>(grid, stream, pm, po, wv, seq_lens, ov, B, H, cap, split, s_max, slices, seq_rows,
                                  spw);
  if (dc == 320)
    return launch_combine_dc<320>(grid, stream, pm, po, wv, seq_lens, ov, B, H, cap, split, s_max, slices, seq_rows,
                                  spw);
  return launch_combine_dc<512>(grid, stream, pm, po, wv, seq_lens, ov, B, H, cap, split, s_max, slices, seq_rows,
                                spw);
}

}  // namespace

// Compute units of the current device (cached per device).
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

namespace {

// The MFMA split kernels launch with hipExtLaunchKernelGGL so that optional
// timing events are stamped by the dispatch itself (kernel start and end).
template <int DC, int DR>
hipError_t launch_slice(const SplitArgs& a, int slices, int nblocks, hipStream_t stream, hipEvent_t ev0,
                        hipEvent_t ev1) {
  if (slices == kIdSlices)
    hipExtLaunchKernelGGL((split_slice_kernel<DC, DR, kSliceWaves, kSliceDepth, kIdSlices>), dim3(nblocks * slices),
                          dim3(kSliceWaves * 64), 0, stream, ev0, ev1, 0, a);
  else if (a.qin)
    hipExtLaunchKernelGGL((split_slice_kernel<DC, DR, kSliceWaves, kSliceDepth, 1, true>), dim3(nblocks),
                          dim3(kSliceWaves * 64), 0, stream, ev0, ev1, 0, a);
  else
    hipExtLaunchKernelGGL((split_slice_kernel<DC, DR, kSliceWaves, kSliceDepth, 1>), dim3(nblocks),
                          dim3(kSliceWaves * 64), 0, stream, ev0, ev1, 0, a);
  return hipGetLastError();
}

// Stamp of a decode call whose split kernel absorbs the query: distinct for
// every call of the process and never 0, so that no stamp left in a
// workspace by an earlier call (or found in fresh memory, but for a chance of
// 2^-64 per stamp) matches.  The first value is drawn from the clock and the
// address space layout.
unsigned long long next_stamp() {
  static std::atomic<unsigned long long> counter{
      (static_cast<unsigned long long>(std::chrono::steady_clock::now().time_since_epoch().count()) * 0x9E3779B97F4A7C15ull) ^
      reinterpret_cast<uintptr_t>(&counter)};
  unsigned long long v;
  do v = counter.fetch_add(1, std::memory_order_relaxed) + 1; while (v == 0);
  return v;
}

// Polls of the absorption stamps before a work-group absorbs the query itself
// (a few milliseconds); EGMLA_SPIN_LIMIT overrides it (0: always absorb locally).
int absorb_spin_limit() {
  const char* e = std::getenv("EGMLA_SPIN_LIMIT");
  if (e && *e) return std::max(0, std::atoi(e));
  return 1 << 16;
}

// Balanced head-split kernel: `ranges` token ranges x a.groups blocks of 64 heads.
// Wide kernel: units in flight per score wave.
#ifndef EGMLA_WIDE_DEPTH
#define EGMLA_WIDE_DEPTH 2
#endif
constexpr int kWideDepth = EGMLA_WIDE_DEPTH;

hipError_t launch_wide(const SplitArgs& a, int ranges, hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  hipExtLaunchKernelGGL((split_wide_kernel<kWideDepth>), dim3(ranges * a.groups), dim3(WideCfg::NT), 0,
                        stream, ev0, ev1, 0, a);
  return hipGetLastError();
}

// Token ranges of the balanced schedule: one work-group per compute unit over
// all head blocks, a multiple of 8 (the head blocks of a range share an XCD).
int wide_groups(int head_groups) {
  const int g = std::min(kWideMaxGroups, device_cus() / std::max(1, head_groups));
  return std::max(8, g / 8 * 8);
}

template <int DC, int DR>
hipError_t launch_mfma(const SplitArgs& a, int nblocks, hipStream_t stream, hipEvent_t ev0, hipEvent_t ev1) {
  hipExtLaunchKernelGGL((split_mfma_kernel<DC, DR>), dim3(nblocks), dim3(DsplitCfg<DC, DR>::NW * 64), 0, stream, ev0,
                        ev1, 0, a);
  return hipGetLastError();
}

hipError_t launch_split(const eg_mla_dims& d, const DecodePlan& p, const SplitArgs& a, hipStream_t stream,
                        hipEvent_t ev0, hipEvent_t ev1) {
  const int64_t nblocks64 = static_cast<int64_t>(a.B) * a.s_max * a.groups;
  if (nblocks64 > 0x7fffffff) return hipErrorInvalidValue;
  const int nblocks = static_cast<int>(nblocks64);
  if (p.path == EG_MLA_PATH_MFMA) {
    if (tok_kernel_shape(d)) {
      if (static_cast<int64_t>(nblocks) * p.slices > 0x7fffffff) return hipErrorInvalidValue;
      return launch_slice<128, 64>(a, p.slices, nblocks, stream, ev0, ev1);
    }
    if (heads_kernel_shape(d)) return launch_wide(a, wide_groups(a.groups), stream, ev0, ev1);
    if (d.latent_dim == 320) return launch_mfma<320, 64>(a, nblocks, stream, ev0, ev1);
    if (d.latent_dim == 512) return launch_mfma<512, 64>(a, nblocks, stream, ev0, ev1);
    return hipErrorInvalidValue;
  }
  if (ev0 && hipEventRecord(ev0, stream) != hipSuccess) return hipErrorInvalidValue;
  const int DQ = d.latent_dim + d.rope_dim;
  size_t lds = sizeof(float) * (static_cast<size_t>(a.hpg) * DQ + kTile * (DQ + 1) + a.hpg * kTile + a.hpg + 1) +
               kTile * (sizeof(int64_t) + sizeof(int)) + 16;
  if (d.dtype == EG_MLA_BF16) {
    hipError_t e = set_lds(split_valu_kernel<true>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(split_valu_kernel<true>, dim3(nblocks), dim3(kValuThreads), lds, stream, a);
  } else {
    hipError_t e = set_lds(split_valu_kernel<false>, lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(split_valu_kernel<false>, dim3(nblocks), dim3(kValuThreads), lds, stream, a);
  }
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && ev1) e = hipEventRecord(ev1, stream);
  return e;
}

}  // namespace
}  // namespace egmla

namespace egmla {
namespace {

// Enqueues one decode call whose arguments validate_decode has accepted, with
// its workspace at `workspace` laid out by the plan p.
eg_mla_status run_decode(const eg_mla_dims& d, const DecodePlan& p, int32_t batch, const void* q,
                         const void* latent_cache, const int32_t* token_id_cache, const void* gate_table,
                         const void* w_uk, const void* w_uv, const int32_t* seq_lens, const int32_t* page_table,
                         int32_t max_pages_per_seq, int64_t num_slots, void* workspace, void* out, void* stream_,
                         const eg_mla_plan* plan) {
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  const bool bf = d.dtype == EG_MLA_BF16;
  (void)hipGetLastError();  // clear a stale error so the checks below are ours

  unsigned char* ws = static_cast<unsigned char*>(workspace);
  float* qfull = reinterpret_cast<float*>(ws + p.off_q);
  float* part_ml = reinterpret_cast<float*>(ws + p.off_ml);
  float* part_o = reinterpret_cast<float*>(ws + p.off_o);

  int64_t* sched_hdr = nullptr;
  int2* wg_start = nullptr;
  int2* seq_rows = nullptr;
  if (p.balanced) {
    // 0. balanced schedule of the head-split kernel (token ranges per work-group)
    // (computed by the absorption launch below)
    sched_hdr = reinterpret_cast<int64_t*>(ws + p.off_sched);
    wg_start = reinterpret_cast<int2*>(ws + p.off_sched + 16);
    seq_rows = reinterpret_cast<int2*>(ws + p.off_sched + 16 + kWideMaxGroups * 8);
  }
  const WideSchedArgs sched{seq_lens, p.capacity, p.balanced ? wide_groups(p.head_groups) : 0, sched_hdr, wg_start,
                            seq_rows};
  // 1. absorption (or inside the split kernel)
  if (!p.fused_absorb) {
    dim3 grid(d.num_heads, (d.latent_dim + kAbsorbCols - 1) / kAbsorbCols, (batch + kAbsorbRows - 1) / kAbsorbRows);
    const size_t lds = sizeof(float) * (kAbsorbRows * d.head_dim + 4 * kAbsorbRows * kAbsorbCols);
    if (bf && d.head_dim == 128) {
      // A W_UK of a few MB is read once per block of sequences: group blocks so
      // it is read about once; a small one is cheap to re-read, and one block
      // per work-group spreads the work over more compute units.
      const size_t wuk_bytes = static_cast<size_t>(d.num_heads) * d.head_dim * d.latent_dim * 2;
      const bool grouped = p.balanced || wuk_bytes >= (size_t{4} << 20);
      const int rows = kAbsRows * (grouped ? kAbsBlocks : 1);
      const int row_blocks = (batch + rows - 1) / rows;
      // a small grid takes narrower column slices: more work-groups, each
      // with less of W_UK to load (measured faster for B32 H16, slower for B256)
      const bool narrow = !grouped && d.num_heads * row_blocks < kAbsMinWorkGroups;
      const int cols = narrow ? kAbsColsNarrow : kAbsCols;
      dim3 ga(d.num_heads, row_blocks, (d.latent_dim + cols - 1) / cols);
      const uint16_t* q16 = static_cast<const uint16_t*>(q);
      const uint16_t* wuk16 = static_cast<const uint16_t*>(w_uk);
      if (p.balanced)  // the wide kernel takes the query as fp16 rows (q^R in bf16); one more column: its schedule
        hipLaunchKernelGGL((absorb_mfma_kernel<128, kAbsBlocks, kAbsCols, true>), dim3(ga.x + 1, ga.y, ga.z),
                           dim3(256), 0, stream, q16, wuk16, qfull, batch, d.num_heads, d.latent_dim, d.rope_dim,
                           sched);
      else if (grouped)
        hipLaunchKernelGGL((absorb_mfma_kernel<128, kAbsBlocks, kAbsCols>), ga, dim3(256), 0, stream, q16, wuk16,
                           qfull, batch, d.num_heads, d.latent_dim, d.rope_dim, sched);
      else if (narrow)
        hipLaunchKernelGGL((absorb_mfma_kernel<128, 1, kAbsColsNarrow>), ga, dim3(256), 0, stream, q16, wuk16, qfull,
                           batch, d.num_heads, d.latent_dim, d.rope_dim, sched);
      else
        hipLaunchKernelGGL((absorb_mfma_kernel<128, 1, kAbsCols>), ga, dim3(256), 0, stream, q16, wuk16, qfull, batch,
                           d.num_heads, d.latent_dim, d.rope_dim, sched);
    } else if (bf) {
      if (set_lds(absorb_kernel<true>, lds) != hipSuccess) return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(absorb_kernel<true>, grid, dim3(256), lds, stream, q, w_uk, qfull, batch, d.num_heads,
                         d.head_dim, d.latent_dim, d.rope_dim);
    } else {
      if (set_lds(absorb_kernel<false>, lds) != hipSuccess) return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(absorb_kernel<false>, grid, dim3(256), lds, stream, q, w_uk, qfull, batch, d.num_heads,
                         d.head_dim, d.latent_dim, d.rope_dim);
    }
    if (hipGetLastError() != hipSuccess) return EG_MLA_ERR_HIP;
  }
  // 2. split kernel (skipped when the cache has no capacity: every length clamps to 0)
  if (p.capacity > 0) {
    SplitArgs a;
    a.qfull = qfull;
    a.cache = latent_cache;
    a.ids = token_id_cache;
    a.gate = gate_table;
    a.seq_lens = seq_lens;
    a.page_table = page_table;
    a.part_ml = part_ml;
    a.part_o = part_o;
    a.sched_hdr = sched_hdr;
    a.wg_start = wg_start;
    a.num_slots = num_slots;
    a.B = batch;
    a.H = d.num_heads;
    a.DC = d.latent_dim;
    a.DR = d.rope_dim;
    a.P = d.page_size;
    a.max_pages = max_pages_per_seq;
    a.V = d.vocab_size;
    a.cap = p.capacity;
    a.split = p.split_tokens;
    a.s_max = p.s_max;
    a.groups = p.head_groups;
    a.hpg = p.heads_per_group;
    a.scale_log2 = softmax_scale(d) * kLog2e;
    a.qin = nullptr;
    a.w_uk = nullptr;
    a.qflags = nullptr;
    a.stamp = 0;
    a.DH = d.head_dim;
    a.spin_limit = 0;
    if (p.fused_absorb) {
      a.qin = static_cast<const uint16_t*>(q);
      a.w_uk = static_cast<const uint16_t*>(w_uk);
      a.qflags = reinterpret_cast<unsigned long long*>(ws + p.off_flags);
      a.stamp = next_stamp();
      a.spin_limit = absorb_spin_limit();
    }
    hipEvent_t ev0 = plan ? static_cast<hipEvent_t>(plan->split_start_event) : nullptr;
    hipEvent_t ev1 = plan ? static_cast<hipEvent_t>(plan->split_stop_event) : nullptr;
    if (launch_split(d, p, a, stream, ev0, ev1) != hipSuccess) return EG_MLA_ERR_HIP;
  }
  // 3. combine + W_UV
  {
    dim3 grid(d.num_heads, batch);
    const size_t lds = sizeof(float) * (d.latent_dim + (p.balanced ? static_cast<size_t>(kWideMaxGroups)
                                                                    : static_cast<size_t>(p.s_max) * p.slices));
    if (lds > 160 * 1024) return EG_MLA_ERR_UNSUPPORTED;
    const bool mfma_comb = bf && d.v_head_dim == 128 &&
                           (d.latent_dim == 128 || d.latent_dim == 320 || d.latent_dim == 512);
    if (mfma_comb) {
      // sequences per merge work-group: 16, or fewer while that leaves under
      // 64 work-groups (B4 H16 with 64 splits per sequence: 7.1 us with 16)
      int spw = kCombSeq;
      while (spw > 1 && static_cast<int64_t>(d.num_heads) * ((batch + spw - 1) / spw) < 64) spw /= 2;
      dim3 g2(d.num_heads, (batch + spw - 1) / spw);
      const float* pm = part_ml;
      const float* po = part_o;
      const uint16_t* wv = static_cast<const uint16_t*>(w_uv);
      uint16_t* ov = static_cast<uint16_t*>(out);
      if (launch_combine_mfma(d.latent_dim, g2, stream, pm, po, wv, seq_lens, ov, batch, d.num_heads, p.capacity,
                              p.split_tokens, p.s_max, p.slices, seq_rows, spw) != hipSuccess)
        return EG_MLA_ERR_HIP;
    } else if (bf) {
      if (set_lds(combine_kernel<true>, lds) != hipSuccess) return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(combine_kernel<true>, grid, dim3(256), lds, stream, part_ml, part_o, w_uv, seq_lens, out,
                         d.num_heads, d.latent_dim, d.v_head_dim, p.capacity, p.split_tokens, p.s_max, p.slices,
                         seq_rows);
    } else {
      if (set_lds(combine_kernel<false>, lds) != hipSuccess) return EG_MLA_ERR_HIP;
      hipLaunchKernelGGL(combine_kernel<false>, grid, dim3(256), lds, stream, part_ml, part_o, w_uv, seq_lens, out,
                         d.num_heads, d.latent_dim, d.v_head_dim, p.capacity, p.split_tokens, p.s_max, p.slices,
                         seq_rows);
    }
    if (hipGetLastError() != hipSuccess) return EG_MLA_ERR_HIP;
  }
  return EG_MLA_OK;
}

// Scratch of the allocation-free decode: one array per device, at file
// scope.  Host code never passes `scratch` itself to a kernel (in host code it
// names a host-side stand-in); it takes the device address that
// hipGetSymbolAddress returns on each device, once, with that device current.
constexpr int kScratchDevices = 64;
__device__ __align__(256) unsigned char scratch[EG_MLA_NOALLOC_SCRATCH_BYTES];
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kScratchDevices] = {nullptr};

// Device address of this device's scratch array, looked up on its first use
// (nullptr if the device index is out of range or the lookup fails).
void* device_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace
}  // namespace egmla

using namespace egmla;

extern "C" eg_mla_status eg_mla_decode_planned(const eg_mla_dims* dims, int32_t batch, const void* q,
                                               const void* latent_cache, const int32_t* token_id_cache,
                                               const void* gate_table, const void* w_uk, const void* w_uv,
                                               const int32_t* seq_lens, const int32_t* page_table,
                                               int32_t max_pages_per_seq, int64_t num_slots, void* workspace,
                                               size_t workspace_bytes, void* out, void* stream,
                                               const eg_mla_plan* plan) {
  DecodePlan p;
  eg_mla_status st = validate_decode(dims, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv,
                                     seq_lens, max_pages_per_seq, num_slots, page_table, workspace,
                                     workspace_bytes, out, plan, &p);
  if (st != EG_MLA_OK || batch == 0) return st;
  return run_decode(*dims, p, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens, page_table,
                    max_pages_per_seq, num_slots, workspace, out, stream, plan);
}

extern "C" eg_mla_status eg_mla_decode_noalloc(const eg_mla_dims* dims, int32_t batch, const void* q,
                                               const void* latent_cache, const int32_t* token_id_cache,
                                               const void* gate_table, const void* w_uk, const void* w_uv,
                                               const int32_t* seq_lens, const int32_t* page_table,
                                               int32_t max_pages_per_seq, int64_t num_slots, void* out,
                                               void* stream) {
  // the plan's workspace must fit the scratch array: checked before any device call
  DecodePlan p;
  eg_mla_status st = check_dims(dims);
  if (st != EG_MLA_OK) return st;
  if (batch < 0 || max_pages_per_seq < 0) return EG_MLA_ERR_INVALID_ARG;
  st = make_decode_plan(*dims, batch, max_pages_per_seq, nullptr, &p);
  if (st != EG_MLA_OK) return st;
  if (p.bytes > EG_MLA_NOALLOC_SCRATCH_BYTES) return EG_MLA_ERR_WORKSPACE;
  if (batch == 0) return validate_decode(dims, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv,
                                         seq_lens, max_pages_per_seq, num_slots, page_table, nullptr, 0, out,
                                         nullptr, &p);
  void* ws = device_scratch();
  if (!ws) return EG_MLA_ERR_HIP;
  st = validate_decode(dims, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens,
                       max_pages_per_seq, num_slots, page_table, ws, EG_MLA_NOALLOC_SCRATCH_BYTES, out, nullptr, &p);
  if (st != EG_MLA_OK) return st;
  return run_decode(*dims, p, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens, page_table,
                    max_pages_per_seq, num_slots, ws, out, stream, nullptr);
}

extern "C" eg_mla_status eg_mla_decode(const eg_mla_dims* dims, int32_t batch, const void* q,
                                       const void* latent_cache, const int32_t* token_id_cache,
                                       const void* gate_table, const void* w_uk, const void* w_uv,
                                       const int32_t* seq_lens, const int32_t* page_table,
                                       int32_t max_pages_per_seq, int64_t num_slots, void* workspace,
                                       size_t workspace_bytes, void* out, void* stream) {
  return eg_mla_decode_planned(dims, batch, q, latent_cache, token_id_cache, gate_table, w_uk, w_uv, seq_lens,
                               page_table, max_pages_per_seq, num_slots, workspace, workspace_bytes, out, stream,
                               nullptr);
}
