// Device-side helpers shared by the attention kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>

namespace kvt {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) __bf16 lds_bf16;

constexpr float kLn2 = 0.693147180559945309f;

// s_waitcnt immediate that waits until at most n vector-memory operations
// are outstanding (lgkm and exp counts left unconstrained); vmcnt is split
// over bits 3:0 and 15:14.
constexpr int vmcnt_imm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }
constexpr float kLog2e = 1.4426950408889634f;

// XOR swizzle of the 16-byte chunks of one key row in LDS (64 banks of 4 B,
// so 256 B per bank cycle).  D = 128 (16 chunks per 256-B row):
// s = (key&3)<<2 | (key>>2)&3 is a bijection on key%16, so the K-operand
// reads (16 lanes, 16 consecutive keys, one chunk column) hit 16 distinct
// bank groups, and the transposed V reads (32 lanes: 4 consecutive keys x 4
// adjacent chunks) do too.  D = 64 (8 chunks per 128-B row, two rows per bank
// cycle): s = ((key>>1)&1)<<2 | (key>>2)&3 gives the same two properties.
template <int D>
__device__ __forceinline__ int swz(int key) {
  if constexpr (D == 128) return ((key & 3) << 2) | ((key >> 2) & 3);
  else return (((key >> 1) & 1) << 2) | ((key >> 2) & 3);
}

// 8 consecutive elements as bf16 (fp32 storage is rounded to nearest even).
__device__ __forceinline__ u32x4 load8(const __bf16* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ u32x4 load8(const float* p) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  u32x4 r;
  r[0] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a[0], a[1]}, bf16x2));
  r[1] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a[2], a[3]}, bf16x2));
  r[2] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){b[0], b[1]}, bf16x2));
  r[3] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){b[2], b[3]}, bf16x2));
  return r;
}

__device__ __forceinline__ void store4(__bf16* p, float a, float b, float c, float d) {
  u32x2 v;
  v[0] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){a, b}, bf16x2));
  v[1] = __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2){c, d}, bf16x2));
  *reinterpret_cast<u32x2*>(p) = v;
}
__device__ __forceinline__ void store4(float* p, float a, float b, float c, float d) {
  *reinterpret_cast<f32x4*>(p) = (f32x4){a, b, c, d};
}
__device__ __forceinline__ void store1(__bf16* p, float a) { *p = (__bf16)a; }
__device__ __forceinline__ void store1(float* p, float a) { *p = a; }

// Own value and the partner lane's (l ^ 32) value, via v_permlane32_swap:
// with vdst = vsrc = x the swap leaves {x_lo, x_lo} in vdst and {x_hi, x_hi}
// in vsrc, so every lane sees both halves' values in the two results.  The
// two results are copied into scalars before the bit cast: a bit cast applied
// directly to an element of the returned vector reads element 0 for both.
__device__ __forceinline__ void pair_values(float x, float& a, float& b) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned p0 = p[0];
  const unsigned p1 = p[1];
  a = __builtin_bit_cast(float, p0);
  b = __builtin_bit_cast(float, p1);
}
__device__ __forceinline__ float pair_max(float x) {
  float a, b;
  pair_values(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float pair_sum(float x) {
  float a, b;
  pair_values(x, a, b);
  return a + b;
}

// Index of the sequence whose units contain `unit`: the last s < nseq with
// begin[s] <= unit (begin ascending, begin[0] = 0), by binary search over
// wave-uniform kernel arguments (at most 8 steps for 256 sequences).
__device__ __forceinline__ int find_seq(const int32_t* begin, int nseq, int unit) {
  int lo = 0, hi = nseq - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (begin[mid] <= unit) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

}  // namespace dev
}  // namespace kvt
