// Exact fp32 x bf16 products on the bf16 matrix cores.
//
// A truncating split writes an fp32 value as the sum of three bf16 values
// (each keeps the next 8 of the 24 significant bits), so a product of a bf16
// weight with an fp32 activation is the sum of three exact bf16 x bf16
// products; the matrix core adds them in fp32.  The r-space products of the
// refiner use this with bf16 weights, which keeps fp32 operand precision at
// bf16 matrix-core throughput.
#pragma once

#include "xp_device.h"

namespace xp {

// fp32 -> three bf16 terms with x == hi + mid + lo exactly (truncating split:
// each term keeps the next 8 significant bits of the 24).  With bf16 weights
// every product w * term is exact in fp32, so W x on the bf16 matrix cores
// is W x with fp32 accumulation, as on the fp32 path.
__device__ __forceinline__ void split3(float x, uint32_t& h, uint32_t& m, uint32_t& l) {
  const uint32_t xh = __float_as_uint(x) & 0xFFFF0000u;
  const float r1 = x - __uint_as_float(xh);
  const uint32_t xm = __float_as_uint(r1) & 0xFFFF0000u;
  const float r2 = r1 - __uint_as_float(xm);
  h = xh >> 16;
  m = xm >> 16;
  l = __float_as_uint(r2) >> 16;
}
// Three bf16x8 MFMA operands from 8 fp32 values (two float4).
__device__ __forceinline__ void split3x8(float4 v0, float4 v1, u32x4& bh, u32x4& bm, u32x4& bl) {
  const float x[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
  uint32_t h[8], m[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) split3(x[i], h[i], m[i], l[i]);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bh[i] = h[2 * i] | (h[2 * i + 1] << 16);
    bm[i] = m[2 * i] | (m[2 * i + 1] << 16);
    bl[i] = l[2 * i] | (l[2 * i + 1] << 16);
  }
}
// acc += a . x over one 32-k step, x (8 fp32 per lane) split into three terms;
// `a` is the exact bf16 operand.  The split operand may be either A or B.
__device__ __forceinline__ floatx4 mma_split_b(u32x4 a, float4 x0, float4 x1, floatx4 acc) {
  u32x4 bh, bm, bl;
  split3x8(x0, x1, bh, bm, bl);
  acc = Mfma<uint16_t>::mma(a, bh, acc);
  acc = Mfma<uint16_t>::mma(a, bm, acc);
  acc = Mfma<uint16_t>::mma(a, bl, acc);
  return acc;
}
__device__ __forceinline__ floatx4 mma_split_a(float4 x0, float4 x1, u32x4 b, floatx4 acc) {
  u32x4 ah, am, al;
  split3x8(x0, x1, ah, am, al);
  acc = Mfma<uint16_t>::mma(ah, b, acc);
  acc = Mfma<uint16_t>::mma(am, b, acc);
  acc = Mfma<uint16_t>::mma(al, b, acc);
  return acc;
}

}  // namespace xp
