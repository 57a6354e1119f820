// Device helpers shared by the EG-MLA HIP kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace egmla {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4_t;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4_t;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2_t;
typedef __attribute__((ext_vector_type(4))) short s16x4_t;  // operand of the 16x16x16 bf16 MFMA

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(static_cast<uint32_t>(b) << 16); }

// fp32 -> bf16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(uint16_t, h);
}
// Two fp32 -> packed bf16 pair (lo in bits 0..15), one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
  typedef __attribute__((ext_vector_type(2))) float f32x2_t;
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

typedef __attribute__((ext_vector_type(8))) _Float16 f16x8_t;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4_t;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2_t;

// Two fp32 -> packed fp16 pair (lo in bits 0..15), round to nearest even.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, f16x2_t{static_cast<_Float16>(lo), static_cast<_Float16>(hi)});
}

// 8 bf16 values (16 bytes) to 8 fp16 values: exact for magnitudes between
// 2^-14 and 65504 (a bf16 significand has 8 bits, an fp16 one 11).
__device__ __forceinline__ u32x4_t bf16x8_to_f16x8(u32x4_t v) {
  u32x4_t r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack_f16x2(bf16_lo(v[e]), bf16_hi(v[e]));
  return r;
}

// Gated latent of one 16-byte chunk: word e of the result packs
// bf16(lat.lo * gate.lo) and bf16(lat.hi * gate.hi) of word e.  Each product is
// v_dot2_f32_bf16 of the latent word with the gate word's other half zeroed: a
// product of two bf16 values fits fp32 exactly, and adding the zero product
// and the zero accumulator is exact; v_cvt_pk_bf16_f32 then rounds once.  The
// sequence is one asm block because the compiler's hazard checks cannot see
// into it: a value written by a DOT instruction must not be read by another
// VALU instruction for 3 wait states, so all eight products come first and the
// last conversion, 3 instructions after the last product, gets 2 more; and a
// VALU result must not feed an MFMA operand for 2 wait states, so the block
// ends with 2 (each s_nop 1).
__device__ __forceinline__ u32x4_t gate_chunk(u32x4_t lat, u32x4_t gate) {
  u32x4_t out;
  float t0, t1, t2, t3, t4, t5, t6, t7;
  asm("v_dot2_f32_bf16 %[t0], %[a0], %[l0], 0\n\t"
      "v_dot2_f32_bf16 %[t1], %[a0], %[h0], 0\n\t"
      "v_dot2_f32_bf16 %[t2], %[a1], %[l1], 0\n\t"
      "v_dot2_f32_bf16 %[t3], %[a1], %[h1], 0\n\t"
      "v_dot2_f32_bf16 %[t4], %[a2], %[l2], 0\n\t"
      "v_dot2_f32_bf16 %[t5], %[a2], %[h2], 0\n\t"
      "v_dot2_f32_bf16 %[t6], %[a3], %[l3], 0\n\t"
      "v_dot2_f32_bf16 %[t7], %[a3], %[h3], 0\n\t"
      "v_cvt_pk_bf16_f32 %[o0], %[t0], %[t1]\n\t"
      "v_cvt_pk_bf16_f32 %[o1], %[t2], %[t3]\n\t"
      "v_cvt_pk_bf16_f32 %[o2], %[t4], %[t5]\n\t"
      "s_nop 1\n\t"
      "v_cvt_pk_bf16_f32 %[o3], %[t6], %[t7]\n\t"
      "s_nop 1"
      : [o0] "=&v"(out[0]), [o1] "=&v"(out[1]), [o2] "=&v"(out[2]), [o3] "=&v"(out[3]), [t0] "=&v"(t0),
        [t1] "=&v"(t1), [t2] "=&v"(t2), [t3] "=&v"(t3), [t4] "=&v"(t4), [t5] "=&v"(t5), [t6] "=&v"(t6),
        [t7] "=&v"(t7)
      : [a0] "v"(lat[0]), [a1] "v"(lat[1]), [a2] "v"(lat[2]), [a3] "v"(lat[3]), [l0] "v"(gate[0] & 0xffffu),
        [l1] "v"(gate[1] & 0xffffu), [l2] "v"(gate[2] & 0xffffu), [l3] "v"(gate[3] & 0xffffu),
        [h0] "v"(gate[0] & 0xffff0000u), [h1] "v"(gate[1] & 0xffff0000u), [h2] "v"(gate[2] & 0xffff0000u),
        [h3] "v"(gate[3] & 0xffff0000u));
  return out;
}

// Gated latent of one 16-byte chunk as bf16 hi + lo: hi is gate_chunk's
// result and lo packs bf16(t - hi) of each exact fp32 product t.  A product of
// two bf16 values has at most 16 significant bits and hi keeps the top 8
// (rounded), so the remainder fits a bf16 exactly: hi + lo == lat * gate.  The
// products are read here after gate_chunk's block has ended, which leaves
// them more than the 3 wait states a DOT result needs.
__device__ __forceinline__ void gate_chunk_hilo(u32x4_t lat, u32x4_t gate, u32x4_t& hi, u32x4_t& lo) {
  float t[8];
  asm("v_dot2_f32_bf16 %[t0], %[a0], %[l0], 0\n\t"
      "v_dot2_f32_bf16 %[t1], %[a0], %[h0], 0\n\t"
      "v_dot2_f32_bf16 %[t2], %[a1], %[l1], 0\n\t"
      "v_dot2_f32_bf16 %[t3], %[a1], %[h1], 0\n\t"
      "v_dot2_f32_bf16 %[t4], %[a2], %[l2], 0\n\t"
      "v_dot2_f32_bf16 %[t5], %[a2], %[h2], 0\n\t"
      "v_dot2_f32_bf16 %[t6], %[a3], %[l3], 0\n\t"
      "v_dot2_f32_bf16 %[t7], %[a3], %[h3], 0\n\t"
      "v_cvt_pk_bf16_f32 %[o0], %[t0], %[t1]\n\t"
      "v_cvt_pk_bf16_f32 %[o1], %[t2], %[t3]\n\t"
      "v_cvt_pk_bf16_f32 %[o2], %[t4], %[t5]\n\t"
      "s_nop 1\n\t"
      "v_cvt_pk_bf16_f32 %[o3], %[t6], %[t7]\n\t"
      "s_nop 1"
      : [o0] "=&v"(hi[0]), [o1] "=&v"(hi[1]), [o2] "=&v"(hi[2]), [o3] "=&v"(hi[3]), [t0] "=&v"(t[0]),
        [t1] "=&v"(t[1]), [t2] "=&v"(t[2]), [t3] "=&v"(t[3]), [t4] "=&v"(t[4]), [t5] "=&v"(t[5]), [t6] "=&v"(t[6]),
        [t7] "=&v"(t[7])
      : [a0] "v"(lat[0]), [a1] "v"(lat[1]), [a2] "v"(lat[2]), [a3] "v"(lat[3]), [l0] "v"(gate[0] & 0xffffu),
        [l1] "v"(gate[1] & 0xffffu), [l2] "v"(gate[2] & 0xffffu), [l3] "v"(gate[3] & 0xffffu),
        [h0] "v"(gate[0] & 0xffff0000u), [h1] "v"(gate[1] & 0xffff0000u), [h2] "v"(gate[2] & 0xffff0000u),
        [h3] "v"(gate[3] & 0xffff0000u));
#pragma unroll
  for (int e = 0; e < 4; ++e) lo[e] = pack_bf16x2(t[2 * e] - bf16_lo(hi[e]), t[2 * e + 1] - bf16_hi(hi[e]));
}

// Gated latent of one 16-byte chunk in fp16: the eight exact fp32 products
// (formed as in gate_chunk), each rounded once to fp16.  The block ends with
// 3 wait states (s_nop 2), so that the conversions after it may read the DOT
// results.
__device__ __forceinline__ u32x4_t gate_chunk_f16(u32x4_t lat, u32x4_t gate) {
  float t[8];
  asm("v_dot2_f32_bf16 %[t0], %[a0], %[l0], 0\n\t"
      "v_dot2_f32_bf16 %[t1], %[a0], %[h0], 0\n\t"
      "v_dot2_f32_bf16 %[t2], %[a1], %[l1], 0\n\t"
      "v_dot2_f32_bf16 %[t3], %[a1], %[h1], 0\n\t"
      "v_dot2_f32_bf16 %[t4], %[a2], %[l2], 0\n\t"
      "v_dot2_f32_bf16 %[t5], %[a2], %[h2], 0\n\t"
      "v_dot2_f32_bf16 %[t6], %[a3], %[l3], 0\n\t"
      "v_dot2_f32_bf16 %[t7], %[a3], %[h3], 0\n\t"
      "s_nop 2"
      : [t0] "=&v"(t[0]), [t1] "=&v"(t[1]), [t2] "=&v"(t[2]), [t3] "=&v"(t[3]), [t4] "=&v"(t[4]),
        [t5] "=&v"(t[5]), [t6] "=&v"(t[6]), [t7] "=&v"(t[7])
      : [a0] "v"(lat[0]), [a1] "v"(lat[1]), [a2] "v"(lat[2]), [a3] "v"(lat[3]), [l0] "v"(gate[0] & 0xffffu),
        [l1] "v"(gate[1] & 0xffffu), [l2] "v"(gate[2] & 0xffffu), [l3] "v"(gate[3] & 0xffffu),
        [h0] "v"(gate[0] & 0xffff0000u), [h1] "v"(gate[1] & 0xffff0000u), [h2] "v"(gate[2] & 0xffff0000u),
        [h3] "v"(gate[3] & 0xffff0000u));
  return u32x4_t{pack_f16x2(t[0], t[1]), pack_f16x2(t[2], t[3]), pack_f16x2(t[4], t[5]), pack_f16x2(t[6], t[7])};
}

// Largest growth (log2 units) of a head's running maximum that an online
// softmax absorbs without rescaling its accumulators: probabilities relative
// to the stale maximum stay below 2^8, far from fp32 overflow.
constexpr float kLazyRescale = 8.0f;

// Maximum over the four lanes i, i ^ 16, i ^ 32, i ^ 48 (VALU lane swaps).
__device__ __forceinline__ float max_over_row_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = fmaxf(__uint_as_float(s32[0]), __uint_as_float(s32[1]));
  const uint32_t v = __float_as_uint(x);
  const auto s16 = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return fmaxf(__uint_as_float(s16[0]), __uint_as_float(s16[1]));
}

// Sum over the four lanes i, i ^ 16, i ^ 32, i ^ 48 (VALU lane swaps), added
// in the same order in every lane.
__device__ __forceinline__ float sum_over_row_groups(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  x = __uint_as_float(s32[0]) + __uint_as_float(s32[1]);
  const uint32_t v = __float_as_uint(x);
  const auto s16 = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  return __uint_as_float(s16[0]) + __uint_as_float(s16[1]);
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

// Cache row of token j given its page-table entry, clamped into the cache.
__device__ __forceinline__ int64_t paged_slot(int page, int j, int P, int64_t num_slots) {
  const int64_t npages = num_slots / P;
  page = page < 0 ? 0 : page;
  int64_t s = (static_cast<int64_t>(page) < npages ? static_cast<int64_t>(page) : npages - 1) * P + j % P;
  s = s < 0 ? 0 : s;
  return s < num_slots ? s : num_slots - 1;
}

// Cache row of token j of sequence b in a contiguous cache, clamped into the cache.
__device__ __forceinline__ int64_t contiguous_slot(int b, int j, int P, int max_pages, int64_t num_slots) {
  int64_t s = static_cast<int64_t>(b) * max_pages * P + j;
  s = s < 0 ? 0 : s;
  return s < num_slots ? s : num_slots - 1;
}

// Cache row of token j of sequence b (paged or contiguous), clamped into the cache.
__device__ __forceinline__ int64_t cache_slot(const int32_t* __restrict__ page_table, int b, int j, int P,
                                              int max_pages, int64_t num_slots) {
  if (page_table) return paged_slot(page_table[static_cast<int64_t>(b) * max_pages + j / P], j, P, num_slots);
  return contiguous_slot(b, j, P, max_pages, num_slots);
}

__device__ __forceinline__ int clamp_id(int id, int V) { return id < 0 ? 0 : (id >= V ? V - 1 : id); }

__device__ __forceinline__ int clamp_len(int L, int cap) { return L < 0 ? 0 : (L > cap ? cap : L); }

}  // namespace egmla
