// Device-side helpers shared by the HIP kernels of the refine + verify path.
// gfx950 (CDNA4) only: wave64, MFMA matrix cores, 160 KB LDS per CU.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xp {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kTile = 16;            // vocabulary rows per MFMA tile (and positions per block)

// ---------------------------------------------------------------------------
// bf16 storage <-> fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}
// round to nearest, ties to even (finite inputs)
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Two fp32 values to packed bf16 (a low, b high), rounded to nearest even
// (v_cvt_pk_bf16_f32; the same as f32_to_bf16_rne for finite values)
typedef __bf16 xp_bf16x2 __attribute__((ext_vector_type(2)));
typedef float xp_f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pk_bf16(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(xp_f32x2{a, b}, xp_bf16x2));
}

// SwiGLU of one feature: silu(g) u = g / (1 + e^-g) u
__device__ __forceinline__ float silu_mul(float g, float u) { return g / (1.f + __expf(-g)) * u; }

template <typename T> __device__ __forceinline__ float to_f32(T v);
template <> __device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) { return bf16_to_f32(v); }

// ---------------------------------------------------------------------------
// 64-bit argmax key: order-preserving image of the fp32 value in the high word,
// bitwise-not of the index in the low word.  max(key) = largest value, and for
// equal values the lowest index.  -0 is mapped to +0 first.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t idx) {
  uint32_t u = __float_as_uint(v);
  if (u == 0x80000000u) u = 0u;
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)u << 32) | (uint64_t)(~idx);
}
__device__ __forceinline__ uint32_t key_index(uint64_t k) { return ~(uint32_t)(k & 0xFFFFFFFFull); }
__device__ __forceinline__ float key_value(uint64_t k) {
  uint32_t u = (uint32_t)(k >> 32);
  u = (u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u;
  return __uint_as_float(u);
}
constexpr uint64_t kKeyMin = 0ull;

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor((uint32_t)v, m, kWave);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// The base logits s are stored tile-major: the 16 rows of vocabulary tile t
// for position p are 64 contiguous bytes at float offset 16 (t Ms + p), so a
// tile's rows for consecutive positions are contiguous.  Ms is the position
// count of the refine call that wrote them.
__host__ __device__ __forceinline__ size_t s_index(int p, int row, int Ms) {
  return ((size_t)(row >> 4) * Ms + p) * 16 + (row & 15);
}

// ---------------------------------------------------------------------------
// Exchanges across the 16- and 32-lane halves of the wave on gfx950's lane-swap
// instructions (v_permlane16_swap, v_permlane32_swap) instead of an LDS round
// trip.  With x as both operands the instruction returns, in every lane, the
// values of lanes l and l ^ 16 (l ^ 32), that of the lower half first, so the
// max or sum of the pair equals x combined with its partner's value bit for
// bit (both operations commute).
// ---------------------------------------------------------------------------
__device__ __forceinline__ float fmax_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float fmax_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float fadd_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float fadd_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// ---------------------------------------------------------------------------
// Order a wave's LDS writes before its later LDS reads of other lanes' data.
// A wave's LDS instructions execute in program order, so only the compiler
// must be kept from moving the accesses across this point.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void wave_lds_order() {
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

// 16 bytes per lane from global memory straight into LDS
// (global_load_lds_dwordx4): lane l's data lands at lds + 16 l, lds must be the
// same for the whole wave.  The loads count in the vector-memory counter and
// the compiler does not wait for them: the caller waits explicitly before the
// data is read.
__device__ __forceinline__ void lds_dma16(const void* g, u32x4* lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0);
}
// The same with the non-temporal hint (nt), for data streamed once per use
// (the base logits in the many-position Read), so that the stream leaves the
// reused operands (W_r, z) in the caches: 304 instead of 311 us per Read pass
// at 2048 positions, 70 instead of 81 us at 512.
__device__ __forceinline__ void lds_dma16_nt(const void* g, u32x4* lds) {
  __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 2);
}

// Workgroup barrier that publishes LDS writes only.  __syncthreads() also
// waits for every outstanding global load of the wave (the fence drains the
// whole vector-memory counter); this one waits for the wave's LDS (and
// scalar) operations, so loads issued earlier stay in flight across it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0); vmcnt, expcnt left at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A per-sequence temperature flag, loaded unconditionally (from `dummy`, any
// valid device address, when there are no flags): a load under a branch makes
// the compiler wait for every load issued before it at the join.
__device__ __forceinline__ int load_flag(const uint8_t* flags, int idx, const void* dummy) {
  const uint8_t* p = flags != nullptr ? flags + idx : reinterpret_cast<const uint8_t*>(dummy);
  const int v = *p;
  return flags != nullptr ? v : 0;
}

// ---------------------------------------------------------------------------
// Online softmax statistics (max, sum of exp(x - max)) in fp32.
// ---------------------------------------------------------------------------
struct Stat {
  float m;
  float s;
};
__device__ __forceinline__ Stat stat_empty() { return Stat{-INFINITY, 0.f}; }
__device__ __forceinline__ Stat stat_merge(Stat a, Stat b) {
  if (b.s == 0.f) return a;
  if (a.s == 0.f) return b;
  float m = fmaxf(a.m, b.m);
  return Stat{m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}
// Four values at once (absent ones passed as -inf): one rescale of the running
// sum instead of one per value.
__device__ __forceinline__ Stat stat_add4(Stat a, float x0, float x1, float x2, float x3) {
  const float m = fmaxf(a.m, fmaxf(fmaxf(x0, x1), fmaxf(x2, x3)));
  const float s = a.s * __expf(a.m - m) +
                  ((__expf(x0 - m) + __expf(x1 - m)) + (__expf(x2 - m) + __expf(x3 - m)));
  const bool none = m == -INFINITY;              // nothing present so far
  return Stat{none ? a.m : m, none ? a.s : s};
}

// ---------------------------------------------------------------------------
// Vocabulary partition.  The ntiles = ceil(V/16) tiles are cut into U
// contiguous units, unit u owning tiles [u*ntiles/U, (u+1)*ntiles/U).  Every
// kernel that writes per-unit partials and every kernel that reads them uses
// this one formula.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ int unit_tile_lo(int u, int ntiles, int U) {
  return (int)(((int64_t)u * ntiles) / U);
}

// ---------------------------------------------------------------------------
// MFMA 16x16 tiles.  A operand: 16 vocabulary rows, B operand: 16 positions,
// D: acc[i] of lane l is (row 4*(l/16)+i, position l%16).
//
// A "load unit" is the 16 bytes lane l reads from its row (l%16) at byte
// offset 16*(l/16) of a stretch of 64 bytes, i.e. KU = 32 bf16 or 16 fp32
// k-values per unit.  Operands A and B use the same k for the same lane, so
// any assignment of k to lanes gives the same dot products; this one makes
// four lanes read 64 contiguous bytes of a row per instruction.
// ---------------------------------------------------------------------------
template <typename T> struct Mfma;

template <> struct Mfma<uint16_t> {                 // bf16 inputs
  static constexpr int KU = 32;
  __device__ static __forceinline__ floatx4 mma(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
};

template <> struct Mfma<float> {                    // fp32 inputs: four K=4 steps
  static constexpr int KU = 16;
  __device__ static __forceinline__ floatx4 mma(u32x4 a, u32x4 b, floatx4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

// 16-byte loads.  Weight streams use the non-temporal hint so that a 1.2 GB
// LM head does not evict the smaller operands reused across passes from the
// caches.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ u32x4 ld16_nt(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}

}  // namespace xp
