// LDS fragment reads shared by the attention kernels and their gradients: a block of
// bf16 rows of head dimension DH (2 DH bytes, 16-byte chunks XOR-swizzled per row), read
// either as MFMA operand rows (a lane's 8 consecutive elements of one row) or, through the
// transposing LDS read, as the transposed operand whose k index runs over rows.
#pragma once
#include "wm_device.hpp"

namespace wm {

typedef short i16x4 __attribute__((ext_vector_type(4)));

// Chunk swizzle of slot row `row`.
// Head dim 64 (128-B rows): bit-reversal of (row / 2) mod 8. Rows 2x and 2x+1 share a
// 256-B bank line, and rows 4y, 4y+2 differ in bit 2, which keeps a transposing read's
// 4 chunks apart.
// Head dim 96 (192-B rows): (row / 4) mod 4, applied within aligned groups of 4 chunks.
// Row 4a + b starts at 16-B bank group 12 b mod 16 (one of 0, 4, 8, 12 per b), and the
// swizzle adds a distinct 0..3 per a, so 16 consecutive rows' chunk c, and 4 rows x one
// aligned 4-chunk group, fall in 16 distinct bank groups.
template <int DH> __device__ __forceinline__ int pf_swz(int row) {
  if constexpr (DH == 64) {
    const int x = (row >> 1) & 7;
    return ((x & 1) << 2) | (x & 2) | (x >> 2);
  } else {
    return (row >> 2) & 3;
  }
}

// Byte offsets of one lane's fragment reads inside a half block (32 slot rows) of LDS:
// k[ks] for the K fragment of k16 step ks, v[dt][s] for the s-th transposing read of the
// V^T fragment of value tile dt (the second 16 rows of the half add 16 rows). They do
// not depend on the ring stage, so the stage and half fold into the instructions'
// offset fields.
template <int DH> struct PfLane {
  uint32_t k[DH / 16], v[DH / 32][2];
};
template <int DH> __device__ __forceinline__ PfLane<DH> pf_lane(int lane) {
  constexpr int ROW = 2 * DH;
  const int h = lane >> 5, r = lane & 31, j = lane & 15, grp = lane >> 4;
  PfLane<DH> o;
  const int sw = pf_swz<DH>(r);
#pragma unroll
  for (int ks = 0; ks < DH / 16; ++ks) o.k[ks] = r * ROW + 16 * ((2 * ks + h) ^ sw);
#pragma unroll
  for (int dt = 0; dt < DH / 32; ++dt)
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int row = 4 * h + (j >> 2) + 8 * s;
      const int chunk = 4 * dt + 2 * (grp & 1) + ((j & 3) >> 1);
      o.v[dt][s] = row * ROW + 16 * (chunk ^ pf_swz<DH>(row)) + 8 * (j & 1);
    }
  return o;
}
template <int DH>
__device__ __forceinline__ bf16x8 pf_ldk(const char* sm, const PfLane<DH>& lo, uint32_t kh,
                                         int ks) {
  return *(const bf16x8*)(sm + lo.k[ks] + kh);
}
// V^T fragment (value column 32 dt + r, keys 16 hf + 4h + {0..3, 8..11} of the half)
template <int DH>
__device__ __forceinline__ bf16x8 pf_ldv(const char* sm, const PfLane<DH>& lo, uint32_t vh,
                                         int hf, int dt) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  const uint32_t base = vh + hf * 16 * 2 * DH;
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sm + lo.v[dt][0] + base));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(sm + lo.v[dt][1] + base));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

}  // namespace wm
