// Shared device helpers for the gfx950 kernels (wave64, MFMA, LDS).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace amoe {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// number formats
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Order-preserving map of an fp32 logit to an unsigned key (larger logit ->
// larger key).  -0 and +0 map to the same key, so they tie as they compare
// equal; every real logit (including -inf) maps to a key >= 0x007fffff, which
// leaves key 0 free to mark "not eligible".
__device__ __forceinline__ uint32_t logit_key(float z) {
  uint32_t b = __float_as_uint(z);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// ---------------------------------------------------------------------------
// wave-level helpers (64 lanes)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return static_cast<int>(threadIdx.x & (kWave - 1)); }

// Wave index inside the workgroup as a scalar (SGPR) value.  Without this the
// compiler treats threadIdx.x / 64 as a per-lane value, turns loops bounded by
// it into exec-masked branches and places conservative vmcnt waits at their
// joins (which stalls on prefetched loads).
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x / kWave));
}

__device__ __forceinline__ uint64_t lanes_below(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// Wave reductions on DPP row operations (no LDS round trips): pairs, quads,
// half-rows and rows are combined with quad_perm / mirror moves, then rows
// 0+1 and 2+3 with row_bcast:15 and the two halves with row_bcast:31, leaving
// the result in lane 63, which is broadcast.  The order of operations is
// fixed, so sums are reproducible run to run.
namespace dpp {
constexpr int kXor1 = 0xB1;        // quad_perm [1, 0, 3, 2]
constexpr int kXor2 = 0x4E;        // quad_perm [2, 3, 0, 1]
constexpr int kHalfMirror = 0x141; // lane i <-> 7 - i within each 8
constexpr int kMirror = 0x140;     // lane i <-> 15 - i within each row
constexpr int kBcast15 = 0x142;    // lane 15 of row r -> row r + 1
constexpr int kBcast31 = 0x143;    // lane 31 -> rows 2 and 3

// v moved by the DPP control; lanes of rows outside row_mask get `old`
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ uint32_t mov(uint32_t old, uint32_t v) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(static_cast<int>(old), static_cast<int>(v), Ctrl, RowMask, 0xf, false));
}
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ float mov(float old, float v) {
  return __uint_as_float(mov<Ctrl, RowMask>(__float_as_uint(old), __float_as_uint(v)));
}
template <int Ctrl, int RowMask = 0xf>
__device__ __forceinline__ double mov(double old, double v) {
  const uint64_t o = __double_as_longlong(old), x = __double_as_longlong(v);
  const uint32_t lo = mov<Ctrl, RowMask>(static_cast<uint32_t>(o), static_cast<uint32_t>(x));
  const uint32_t hi = mov<Ctrl, RowMask>(static_cast<uint32_t>(o >> 32), static_cast<uint32_t>(x >> 32));
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

__device__ __forceinline__ uint32_t lane63(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), 63));
}
__device__ __forceinline__ float lane63(float v) { return __uint_as_float(lane63(__float_as_uint(v))); }
__device__ __forceinline__ double lane63(double v) {
  const uint64_t x = __double_as_longlong(v);
  const uint64_t lo = lane63(static_cast<uint32_t>(x)), hi = lane63(static_cast<uint32_t>(x >> 32));
  return __longlong_as_double(static_cast<long long>((hi << 32) | lo));
}

// op(a, b) must be commutative; id is its identity
template <class T, class Op>
__device__ __forceinline__ T reduce(T v, T id, Op op) {
  v = op(v, mov<kXor1>(id, v));
  v = op(v, mov<kXor2>(id, v));
  v = op(v, mov<kHalfMirror>(id, v));
  v = op(v, mov<kMirror>(id, v));
  v = op(v, mov<kBcast15, 0xA>(id, v));
  v = op(v, mov<kBcast31, 0xC>(id, v));
  return lane63(v);
}
}  // namespace dpp

__device__ __forceinline__ double wave_sum_f64(double v) {
  return dpp::reduce(v, 0.0, [](double a, double b) { return a + b; });
}

__device__ __forceinline__ float wave_max_f32(float v) {
  return dpp::reduce(v, -INFINITY, [](float a, float b) { return fmaxf(a, b); });
}

__device__ __forceinline__ double wave_max_f64(double v) {
  return dpp::reduce(v, static_cast<double>(-INFINITY), [](double a, double b) { return fmax(a, b); });
}

__device__ __forceinline__ int wave_sum_i32(int v) {
  return static_cast<int>(dpp::reduce(static_cast<uint32_t>(v), 0u, [](uint32_t a, uint32_t b) { return a + b; }));
}

// Inclusive prefix sum over the 64 lanes on DPP moves: Hillis-Steele within
// each row of 16 (shifts 1, 2, 4, 8; lanes without a source add 0), then row
// 15's total into rows 1 and 3 and lane 31's into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan_i32(int v) {
  const uint32_t z = 0u;
  uint32_t x = static_cast<uint32_t>(v);
  x += dpp::mov<0x111>(z, x);  // row_shr:1
  x += dpp::mov<0x112>(z, x);  // row_shr:2
  x += dpp::mov<0x114>(z, x);  // row_shr:4
  x += dpp::mov<0x118>(z, x);  // row_shr:8
  x += dpp::mov<dpp::kBcast15, 0xA>(z, x);
  x += dpp::mov<dpp::kBcast31, 0xC>(z, x);
  return static_cast<int>(x);
}

__device__ __forceinline__ int lane_value(int v, int lane) { return __builtin_amdgcn_readlane(v, lane); }

// Orders LDS traffic between the lanes of one wave (no cross-wave barrier).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------------------
// MFMA wrappers.  Lane L = r + 16*g (r = L % 16, g = L / 16):
//   A operand: row r of the 16-row A tile, K slice g;
//   B operand: column r of the 16-column B tile, same K slice g;
//   C/D: lane L holds rows 4g..4g+3 of column r.
// Any bijection of K onto (g, slot) works as long as A and B use the same one.
// ---------------------------------------------------------------------------
__device__ __forceinline__ floatx4 mfma_bf16_16x16x32(const uint4& a, const uint4& b, floatx4 c) {
  bf16x8 av = __builtin_bit_cast(bf16x8, a);
  bf16x8 bv = __builtin_bit_cast(bf16x8, b);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f32_16x16x4(float a, float b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

}  // namespace amoe
