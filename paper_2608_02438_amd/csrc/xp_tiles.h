// The Read tile: 16 vocabulary rows of W_r against 16 positions of z, r = 256,
// accumulated onto the base logits s.  The vocabulary stream (k_read), the
// sampling rescan and the verification kernels all go through these functions
// in the same order, so every kernel that needs a refined logit l = s + W_r z
// obtains the same fp32 value for it.
#pragma once

#include "xp_device.h"

namespace xp {

template <typename T>
struct ReadTile {
  static constexpr int KU = Mfma<T>::KU;
  static constexpr int NU = 256 / KU;          // load units over k = 0..255
  static constexpr int EPB = 16 / sizeof(T);   // elements per 16-byte load

  // B operand: z rows of positions p0 .. p0+15 (rows >= M read as zero).
  __device__ static __forceinline__ void load_z(const T* __restrict__ Z, int M, int p0, int lane,
                                                u32x4 (&bf)[NU]) {
    const int p = p0 + (lane & 15);
    const T* zr = Z + (size_t)(p < M ? p : 0) * 256 + (lane >> 4) * EPB;
#pragma unroll
    for (int i = 0; i < NU; ++i) bf[i] = (p < M) ? ld16(zr + i * KU) : u32x4{0u, 0u, 0u, 0u};
  }
  // B operand for an arbitrary row list: lane's position reads z row zrow (< 0: zero).
  __device__ static __forceinline__ void load_z_row(const T* __restrict__ Z, int zrow, int lane,
                                                    u32x4 (&bf)[NU]) {
    const T* zr = Z + (size_t)(zrow >= 0 ? zrow : 0) * 256 + (lane >> 4) * EPB;
#pragma unroll
    for (int i = 0; i < NU; ++i) bf[i] = (zrow >= 0) ? ld16(zr + i * KU) : u32x4{0u, 0u, 0u, 0u};
  }
  // A operand: rows 16*tile .. 16*tile+15 of W_r (rows >= V repeat row V-1).
  // Ordinary (temporal) loads: W_r is re-read by every Jacobi pass and stays
  // resident in the last-level cache between passes.
  __device__ static __forceinline__ void load_w(const T* __restrict__ W, int V, int tile, int lane,
                                                u32x4 (&a)[NU]) {
    int row = tile * 16 + (lane & 15);
    row = row < V ? row : V - 1;
    const T* wr = W + (size_t)row * 256 + (lane >> 4) * EPB;
#pragma unroll
    for (int i = 0; i < NU; ++i) a[i] = ld16(wr + i * KU);
  }
  // s operand: the base logits of the lane's four output rows (the MFMA
  // accumulator starts from them, so the chain yields l = s + W_r z directly).
  __device__ static __forceinline__ floatx4 load_s(const float* __restrict__ S, int Ms, int p,
                                                   bool valid, int tile, int lane) {
    if (!valid) return floatx4{0.f, 0.f, 0.f, 0.f};
    return *reinterpret_cast<const floatx4*>(S + s_index(p, tile * 16 + 4 * (lane >> 4), Ms));
  }
  // acc[i] of lane l = init[i] + sum_k W_r[16*tile + 4*(l/16) + i][k] * z[position l%16][k]
  __device__ static __forceinline__ floatx4 chain(const u32x4 (&a)[NU], const u32x4 (&bf)[NU],
                                                  floatx4 acc) {
#pragma unroll
    for (int i = 0; i < NU; ++i) acc = Mfma<T>::mma(a[i], bf[i], acc);
    return acc;
  }
};

}  // namespace xp
