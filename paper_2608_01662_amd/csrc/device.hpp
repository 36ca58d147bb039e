// Device helpers shared by the LSA kernels (gfx950 / CDNA4 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lsa {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(2))) float f32x2;
typedef __attribute__((ext_vector_type(4))) short s16x4;

#define LSA_LDS(p) ((__attribute__((address_space(3))) void*)(p))

constexpr int kWave = 64;

// ---------------------------------------------------------------- matrix cores
// v_mfma_f32_32x32x16_bf16. Operand layouts (checked on gfx950):
//   A[i][k]: lane l holds i = l%32, k = 8*(l/32) + 0..7
//   B[k][j]: lane l holds j = l%32, k = 8*(l/32) + 0..7
//   D[i][j]: lane l, register r holds i = 8*(r/4) + 4*(l/32) + r%4, j = l%32
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
// v_mfma_f32_16x16x32_bf16:
//   A[i][k]: lane l holds i = l%16, k = 8*(l/16) + 0..7
//   B[k][j]: lane l holds j = l%16, k = 8*(l/16) + 0..7
//   D[i][j]: lane l, register r holds i = 4*(l/16) + r, j = l%16
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// v_mfma_scale_f32_32x32x64_f8f6f4 with both operands OCP e4m3 and unit block scales (E8M0 127):
//   A[i][k]: lane l holds i = l%32, k = 32*(l/32) + 0..31 (byte t of its 8 dwords is k offset t)
//   B[k][j]: lane l holds j = l%32, k = 32*(l/32) + 0..31
//   D: as v_mfma_f32_32x32x16_bf16 (checked on gfx950 with an in-bounds probe)
typedef __attribute__((ext_vector_type(8))) int i32x8;
__device__ __forceinline__ f32x16 mfma32_fp8(i32x8 a, i32x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 127, 0, 127);
}
__device__ __forceinline__ i32x8 join_fp8x32(u32x4 lo, u32x4 hi) {
  return i32x8{(int)lo.x, (int)lo.y, (int)lo.z, (int)lo.w, (int)hi.x, (int)hi.y, (int)hi.z, (int)hi.w};
}

// ---------------------------------------------------------------- number formats
// Four OCP e4m3fn codes (one dword) -> four bf16, exactly: the hardware converter yields fp32
// values with at most 4 significant bits, so keeping their upper halves loses nothing.
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t v) {
  f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(v, false);
  f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(v, true);
  u32x2 r;
  r.x = __builtin_amdgcn_perm(__float_as_uint(lo.y), __float_as_uint(lo.x), 0x07060302u);
  r.y = __builtin_amdgcn_perm(__float_as_uint(hi.y), __float_as_uint(hi.x), 0x07060302u);
  return r;
}
// 8 e4m3fn codes (two dwords) -> one bf16x8 MFMA operand.
__device__ __forceinline__ u32x4 fp8x8_to_bf16x8(uint32_t a, uint32_t b) {
  u32x2 x = fp8x4_to_bf16x4(a), y = fp8x4_to_bf16x4(b);
  return u32x4{x.x, x.y, y.x, y.y};
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(uint32_t(h) << 16); }

// Two fp32 -> two bf16 (round to nearest even) packed in one dword: v_cvt_pk_bf16_f32.
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Order-preserving map of a float score onto an unsigned key: a > b  <=>  key(a) > key(b).
// Key 0 is reserved for "not a candidate" (it is the image of the NaN 0xFFFFFFFF only).
__device__ __forceinline__ uint32_t score_key(float f) {
  uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// ---------------------------------------------------------------- waits and barriers
// Wait until at most N vector-memory operations of this wave are outstanding (direct-to-LDS
// loads included), then join the workgroup barrier. The asm memory clobber keeps the compiler
// from moving memory accesses across it; no cache flush or fence is implied.
template <int N>
__device__ __forceinline__ void vm_wait_barrier() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(N) : "memory");
}
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Workgroup barrier that the compiler cannot move memory accesses across (no wait implied).
__device__ __forceinline__ void barrier_only() { asm volatile("s_barrier" ::: "memory"); }
// All LDS reads of this wave have returned; then barrier (used before a buffer is refilled).
__device__ __forceinline__ void lds_done_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// Full workgroup barrier with LDS visibility (ordinary ds_write -> ds_read hand-off).
__device__ __forceinline__ void block_sync() { __syncthreads(); }

// ---------------------------------------------------------------- direct global -> LDS loads
// LDS byte address of a pointer into __shared__ memory (the low 32 bits of its generic address).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
}

// ---------------------------------------------------------------- wave reductions
__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ int wave_sum(int v) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
// Reductions over the four lanes l, l^16, l^32, l^48 with gfx950's row swaps: after
// v_permlane16_swap(x, x) a lane holds {x[l], x[l^16]} in its two results, after
// v_permlane32_swap the same for l^32. VALU only; since a + b == b + a, all four lanes end with
// bit-identical results.
__device__ __forceinline__ float max4_xor16_32(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float sum4_xor16_32(float x) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(y), __float_as_uint(y), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ uint64_t lanemask_lt() {
  int l = threadIdx.x & 63;
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// ---------------------------------------------------------------- XCD-aware block order
// Workgroups are dealt round-robin to the 8 XCDs (block b runs on XCD b % 8). Remap so that
// each XCD walks one contiguous band of work items: neighbouring items (which share keys or
// window rows) then meet in the same 4 MB L2.
__device__ __forceinline__ int64_t xcd_band(int64_t b, int64_t n) {
  const int64_t per = (n + 7) / 8;
  const int64_t x = b % 8, i = b / 8;
  // items beyond n in the last bands are folded back so every item is visited exactly once
  const int64_t full = n - 8 * (per - 1);  // bands [0, full) have `per` items, the rest per-1
  if (x < full) return x * per + i;
  return full * per + (x - full) * (per - 1) + i;
}

}  // namespace lsa
