// Device helpers shared by the EG-MLA HIP kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace egmla {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

// Storage-typed scalar access.
template <bool BF16>
__device__ __forceinline__ float ld(const void* p, int64_t i) {
  if constexpr (BF16) return bf16_to_f32(static_cast<const uint16_t*>(p)[i]);
  else return static_cast<const float*>(p)[i];
}
template <bool BF16>
__device__ __forceinline__ void st(void* p, int64_t i, float v) {
  if constexpr (BF16) static_cast<uint16_t*>(p)[i] = f32_to_bf16(v);
  else static_cast<float*>(p)[i] = v;
}

// Four consecutive storage elements starting at element i (i % 4 == 0).
template <bool BF16>
__device__ __forceinline__ float4 ld4(const void* p, int64_t i) {
  if constexpr (BF16) {
    u32x2_t w = *reinterpret_cast<const u32x2_t*>(static_cast<const uint16_t*>(p) + i);
    return make_float4(bf16_lo(w.x), bf16_hi(w.x), bf16_lo(w.y), bf16_hi(w.y));
  } else {
    return *reinterpret_cast<const float4*>(static_cast<const float*>(p) + i);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Orders this wave's LDS accesses around a point where lanes exchange data
// through LDS (the wave's own region; no other wave involved).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Work-group id -> logical work item such that consecutive logical items run
// on the same XCD.  The dispatcher hands work-groups to the 8 XCDs of an
// MI355X round-robin (id % 8), so item k of XCD x is work-group x + 8k.
__device__ __forceinline__ int xcd_logical_block(int bid, int nblocks) {
  constexpr int kXcd = 8;
  const int xcd = bid % kXcd;
  const int local = bid / kXcd;
  const int per = nblocks / kXcd;
  const int rem = nblocks % kXcd;
  return xcd * per + min(xcd, rem) + local;
}

// Cache row of token j of sequence b (paged or contiguous), clamped into the cache.
__device__ __forceinline__ int64_t cache_slot(const int32_t* __restrict__ page_table, int b, int j, int P,
                                              int max_pages, int64_t num_slots) {
  int64_t s;
  if (page_table) {
    int page = page_table[static_cast<int64_t>(b) * max_pages + j / P];
    const int64_t npages = num_slots / P;
    page = page < 0 ? 0 : page;
    s = (static_cast<int64_t>(page) < npages ? static_cast<int64_t>(page) : npages - 1) * P + j % P;
  } else {
    s = static_cast<int64_t>(b) * max_pages * P + j;
  }
  s = s < 0 ? 0 : s;
  return s < num_slots ? s : num_slots - 1;
}

__device__ __forceinline__ int clamp_id(int id, int V) { return id < 0 ? 0 : (id >= V ? V - 1 : id); }

__device__ __forceinline__ int clamp_len(int L, int cap) { return L < 0 ? 0 : (L > cap ? cap : L); }

}  // namespace egmla
