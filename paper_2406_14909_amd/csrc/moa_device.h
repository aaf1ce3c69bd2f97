// Device helpers for the gfx950 (CDNA4) kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "moa_internal.h"

namespace moa {

typedef __bf16 bf16;
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kNegBig = -1.0e30f;   // finite "minus infinity" for running maxima

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// 16-byte vector of T: 8 bf16 or 4 fp32, with conversion to/from float.
template <typename T> struct Vec16;

template <> struct Vec16<bf16> {
  static constexpr int N = 8;
  bf16x8 v;
  __device__ __forceinline__ float get(int i) const { return static_cast<float>(v[i]); }
  __device__ __forceinline__ void set(int i, float x) { v[i] = static_cast<bf16>(x); }
};

template <> struct Vec16<float> {
  static constexpr int N = 4;
  f32x4 v;
  __device__ __forceinline__ float get(int i) const { return v[i]; }
  __device__ __forceinline__ void set(int i, float x) { v[i] = x; }
};

template <typename T>
__device__ __forceinline__ Vec16<T> load16(const T* p) {
  Vec16<T> r;
  r.v = *reinterpret_cast<const decltype(r.v)*>(p);
  return r;
}

// The same load with the non-temporal hint, for data read once per call
// (the decode caches): a read stream marked this way runs at about 7.1 TB/s on
// MI355X against 6.3 TB/s for plain loads, and does not displace lines that
// other work reuses.
template <typename T>
__device__ __forceinline__ Vec16<T> load16_stream(const T* p) {
  Vec16<T> r;
  r.v = __builtin_nontemporal_load(reinterpret_cast<const decltype(r.v)*>(p));
  return r;
}

template <typename T>
__device__ __forceinline__ Vec16<T> zero16() {
  Vec16<T> r;
#pragma unroll
  for (int i = 0; i < Vec16<T>::N; ++i) r.set(i, 0.0f);
  return r;
}

// Raw buffer descriptor (4 dwords, wave-uniform) over [base, base + bytes),
// gfx9-family format; loads at offsets past `bytes` return zeros.
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 make_desc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{static_cast<int32_t>(a & 0xffffffffu), static_cast<int32_t>((a >> 32) & 0xffffu),
               static_cast<int32_t>(bytes), 0x00020000};
}

// Asynchronous 16-byte-per-lane copy from a buffer straight into LDS
// (buffer_load_dwordx4 ... lds): lane i's bytes land at lds_base + 16 * i.
// It is issued as an opaque statement, so the compiler neither counts it as an
// LDS write nor waits for it before unrelated LDS reads; the caller orders it
// with s_waitcnt vmcnt and a work-group barrier before the data is read.
// The LDS address goes in as an M0 operand, so the compiler itself sets M0
// before the statement and keeps any use of its own intact.
// The compiler inserts no hazard wait states around inline asm, so the
// statement carries its own: on this GPU family a vector-memory instruction
// must come at least 5 wait states after a vector-ALU write of an SGPR it
// reads (the compiler may rebuild the descriptor with v_readlane right
// before), and an LDS DMA at least 1 after a scalar write of M0.  s_nop 4 is
// those 5 wait states.
__device__ __forceinline__ void dma16_async(i32x4 desc, uint32_t voffset, void* lds_base) {
#if defined(__HIP_DEVICE_COMPILE__)
  typedef __attribute__((address_space(3))) char lds_char;
  const uint32_t lds = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_char*)lds_base));
  asm volatile("s_nop 4\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "{m0}"(lds), "v"(voffset), "s"(desc)
               : "memory");
#else
  (void)desc;
  (void)voffset;
  (void)lds_base;
#endif
}

// DPP lane permutation of a float (no LDS round trip).
template <int ctrl>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), ctrl, 0xF, 0xF, false));
}

// Sum over aligned groups of `width` lanes (width a power of two <= 64); every
// lane of a group receives the group's sum.  Within 16 lanes the reduction uses
// DPP: quad_perm [1,0,3,2] and [2,3,0,1] give quad sums, then row_half_mirror
// and row_mirror exchange whole quads and half-rows (valid because the values
// are already uniform across each quad / half-row at that point).
template <int width>
__device__ __forceinline__ float group_sum(float x) {
  static_assert(width >= 1 && width <= 64 && (width & (width - 1)) == 0, "width");
  if constexpr (width >= 2) x += dpp<0xB1>(x);
  if constexpr (width >= 4) x += dpp<0x4E>(x);
  if constexpr (width >= 8) x += dpp<0x141>(x);
  if constexpr (width >= 16) x += dpp<0x140>(x);
  if constexpr (width >= 32) x += __shfl_xor(x, 16, 64);
  if constexpr (width >= 64) x += __shfl_xor(x, 32, 64);
  return x;
}

// Nothing is scheduled across this point: it keeps a written interleave of
// matrix products and vector work in the order written.
__device__ __forceinline__ void sched_fence() {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_sched_barrier(0);
#endif
}

// Exchange with lane l ^ D (D = 32: the other half of the wave; D = 16: the
// other row of the same pair of 16-lane rows): lane l gets its own value and
// that of lane l ^ D in one fixed order (lower lane first), so a symmetric
// combination of the pair is bit-identical in both lanes.  One
// v_permlane32_swap / v_permlane16_swap (a vector-ALU exchange) replaces an
// LDS permute, whose wait would also wait for every LDS read issued before
// it.  Checked on gfx950: with both operands holding x, v_permlane32_swap
// leaves [x_0..31, x_0..31] in the first and [x_32..63, x_32..63] in the
// second; v_permlane16_swap leaves the even row of each row pair in the
// first and the odd row in the second.  Written as assembly with its own wait
// states around it; the compiler builtin for the 32-lane swap returned its
// second result wrong.
struct LanePair {
  float lo, hi;
};
template <int D>
__device__ __forceinline__ LanePair lane_pair(float x) {
  static_assert(D == 16 || D == 32, "lane distance");
#if defined(__HIP_DEVICE_COMPILE__)
  unsigned a = __builtin_bit_cast(unsigned, x), b = a;
  if constexpr (D == 32) asm("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
  else asm("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
  return {__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)};
#else
  return {x, x};
#endif
}
template <int D>
__device__ __forceinline__ float max_xor(float x) {
  const LanePair p = lane_pair<D>(x);
  return fmaxf(p.lo, p.hi);
}
template <int D>
__device__ __forceinline__ float sum_xor(float x) {
  const LanePair p = lane_pair<D>(x);
  return p.lo + p.hi;
}

// Sum over the 64 lanes, complete in lane 63 only: row sums within each
// row of 16 lanes, then row_bcast:15 adds row 0 into row 1 and row 2 into
// row 3, and row_bcast:31 adds lane 31 (rows 0 and 1) into rows 2 and 3.
template <int ctrl, int row_mask>
__device__ __forceinline__ float dpp_rows(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), ctrl, row_mask, 0xF, true));
}
__device__ __forceinline__ float wave_sum_lane63(float x) {
  x = group_sum<16>(x);
  x += dpp_rows<0x142, 0xA>(x);
  x += dpp_rows<0x143, 0xC>(x);
  return x;
}

}  // namespace moa
