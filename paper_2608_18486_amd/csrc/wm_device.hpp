// Device-side building blocks shared by the WhiteMatter kernels (gfx950 only).
//
// Matrix-core convention used everywhere: a 32x32 MFMA tile is fed, per
// "k16 step", with 8 operand elements per lane. Lane l (h = l / 32, r = l % 32)
// supplies A[row r][k slots 8h .. 8h+7] and B[k slots 8h .. 8h+7][col r]. The
// hardware sums over all 16 slots, so any assignment of logical k indices to
// slots is valid as long as A and B use the same one; the kernels rely on this
// to feed P^T straight from the softmax registers.
//   bf16 : one v_mfma_f32_32x32x16_bf16 per k16 step
//   fp32 : eight v_mfma_f32_32x32x2f32 (slot pair {i, 8+i} per instruction)
// Result layout (all 32x32 MFMAs): lane l holds column l % 32 and, in register
// q = 0..15, row 8*(q/4) + 4*(l/32) + (q%4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wm {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) float f32x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegBig = -1.0e30f;

template <typename T> struct Frag;                 // 8 operand elements of one lane
template <> struct Frag<bf16> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x8 type; };
template <typename T> using frag_t = typename Frag<T>::type;

__device__ __forceinline__ f32x16 mma32(f32x16 acc, const bf16x8& a, const bf16x8& b) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mma32(f32x16 acc, const f32x8& a, const f32x8& b) {
#pragma unroll
  for (int i = 0; i < 8; ++i) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[i], b[i], acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return (float)x; }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return (bf16)x; }

// 8 consecutive elements <-> 8 floats (16 B for bf16, 32 B for fp32).
__device__ __forceinline__ void load8(const bf16* p, float* out) {
  bf16x8 v = *(const bf16x8*)p;
#pragma unroll
  for (int i = 0; i < 8; ++i) out[i] = (float)v[i];
}
__device__ __forceinline__ void load8(const float* p, float* out) {
  f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) { out[i] = a[i]; out[4 + i] = b[i]; }
}
__device__ __forceinline__ void store8(bf16* p, const float* in) {
  bf16x8 v;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (bf16)in[i];
  *(bf16x8*)p = v;
}
__device__ __forceinline__ void store8(float* p, const float* in) {
  f32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) { a[i] = in[i]; b[i] = in[4 + i]; }
  *(f32x4*)p = a;
  *(f32x4*)(p + 4) = b;
}
__device__ __forceinline__ void store4(bf16* p, const float* in) {
  bf16x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = (bf16)in[i];
  *(bf16x4*)p = v;
}
__device__ __forceinline__ void store4(float* p, const float* in) {
  f32x4 v;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = in[i];
  *(f32x4*)p = v;
}

// Raw 8-element copies (no conversion), used to move operand tiles.
template <typename T> __device__ __forceinline__ frag_t<T> ld_frag(const T* p) {
  return *(const frag_t<T>*)p;
}
template <typename T> __device__ __forceinline__ void st_frag(T* p, const frag_t<T>& v) {
  *(frag_t<T>*)p = v;
}
template <typename T> __device__ __forceinline__ frag_t<T> zero_frag() {
  frag_t<T> v;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = from_f32<T>(0.f);
  return v;
}

// Buffer loads through a resource descriptor: an offset at or past the
// descriptor's range returns zeros, so guarded tile loads need no branch (and
// the compiler keeps exact wait counts for loads still in flight). Every view
// spans less than 2 GiB (checked on the host); kOffOob is past any such range.
typedef __attribute__((ext_vector_type(4))) int i32x4;
constexpr uint32_t kOffOob = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_view(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ __forceinline__ i32x4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
// One operand fragment (8 elements) at byte offset off.
template <typename T> __device__ __forceinline__ frag_t<T> buf_frag(__amdgpu_buffer_rsrc_t r,
                                                                    uint32_t off);
template <> __device__ __forceinline__ bf16x8 buf_frag<bf16>(__amdgpu_buffer_rsrc_t r,
                                                             uint32_t off) {
  return __builtin_bit_cast(bf16x8, buf_ld16(r, off));
}
template <> __device__ __forceinline__ f32x8 buf_frag<float>(__amdgpu_buffer_rsrc_t r,
                                                             uint32_t off) {
  f32x4 a = __builtin_bit_cast(f32x4, buf_ld16(r, off));
  f32x4 b = __builtin_bit_cast(f32x4, buf_ld16(r, off + 16));
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Copy 16 bytes per lane from a buffer view straight into LDS: lane l's bytes land
// at LDS byte address lds_addr + 16 l (lds_addr is wave-uniform and goes through
// M0). Issued from inline assembly so that the compiler does not add a full
// vmcnt(0) wait in front of every barrier; callers wait with wait_vmcnt.
__device__ __forceinline__ void lds_dma16(uint32_t lds_addr, uint32_t voff,
                                          __amdgpu_buffer_rsrc_t rsrc) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds_addr), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}

// s_waitcnt vmcnt(n) (expcnt and lgkmcnt left alone), n < 16
template <int N> __device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 16, "vmcnt range");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// Workgroups are dispatched round-robin over the chip's 8 XCDs (block i goes to
// XCD i % 8), and each XCD has its own L2. Remap the linear block index so that
// XCD x walks a contiguous share of the tile sequence: tiles that share
// operands (the N tiles of one GEMM row block, the query tiles of one attention
// head) stay on one L2, and every XCD gets an equal slice of a sequence whose
// costs repeat (heavy and light causal tiles alike).
constexpr int kNumXcd = 8;
__device__ __forceinline__ int xcd_tile(int block, int total) {
  const int x = block % kNumXcd, s = block / kNumXcd;
  const int per = total / kNumXcd, rem = total % kNumXcd;
  return x * per + min(x, rem) + s;
}

// Combine a value with the same lane of the other half-wave (lane i with i ^ 32)
// through v_permlane32_swap, without a trip through LDS.
__device__ __forceinline__ float halves_max(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float v) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ctx_len[b] (NULL: 0) clamped into [0, hi]. The host checks that ctx_max plus the
// positions a call's tokens span fits the cache and passes hi = S_cap minus that span, so
// an entry outside its documented range [0, ctx_max] gives that sequence unspecified
// results but never moves an access outside the cache.
__device__ __forceinline__ int ctx_at(const int32_t* ctx_len, int b, int hi) {
  return ctx_len ? min(max(ctx_len[b], 0), hi) : 0;
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

}  // namespace wm
