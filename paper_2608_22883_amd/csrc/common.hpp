// Device helpers shared by the kernels of the FOVEA retrieval + fusion library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fovea {

typedef uint16_t bf16_t;  // bf16 kept as raw bits in memory
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;  // one 16-byte chunk

constexpr int kWave = 64;

// ---------------------------------------------------------------------------------
// scalar conversions
// ---------------------------------------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Round to nearest, ties to even; NaN stays a quiet NaN, overflow rounds to inf.  The
// packed and float-valued forms below use the gfx950 conversion instruction (same
// rounding); the bit-level form is kept for the selection kernel, whose register
// allocation is tighter with it.
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;

__device__ __forceinline__ float bf16_round(float f) {
  return static_cast<float>(static_cast<__bf16>(f));
}

__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Two values rounded to bf16 and packed (lo in the low half), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2_t r;
  r[0] = static_cast<__bf16>(lo);
  r[1] = static_cast<__bf16>(hi);
  return __builtin_bit_cast(uint32_t, r);
}

// Storage element traits: T is float (fp32 storage) or bf16_t (bf16 storage).
template <typename T>
struct Elem;

template <>
struct Elem<float> {
  static constexpr int kPer16B = 4;
  __device__ __forceinline__ static float to_f32(float v) { return v; }
  __device__ __forceinline__ static float from_f32(float v) { return v; }
};

template <>
struct Elem<bf16_t> {
  static constexpr int kPer16B = 8;
  __device__ __forceinline__ static float to_f32(bf16_t v) { return bf16_bits_to_f32(v); }
  __device__ __forceinline__ static bf16_t from_f32(float v) { return f32_to_bf16_bits(v); }
};

template <typename T>
__device__ __forceinline__ float ld_f32(const T* p, int64_t i) {
  return Elem<T>::to_f32(p[i]);
}

template <typename T>
__device__ __forceinline__ void st_f32(T* p, int64_t i, float v) {
  p[i] = Elem<T>::from_f32(v);
}

// 8 consecutive elements (16 bytes of bf16, 32 of fp32) to / from fp32; p 16-byte aligned.
__device__ __forceinline__ void load8(const float* p, float (&x)[8]) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p);
  const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
  x[0] = a[0]; x[1] = a[1]; x[2] = a[2]; x[3] = a[3];
  x[4] = b[0]; x[5] = b[1]; x[6] = b[2]; x[7] = b[3];
}

__device__ __forceinline__ void load8(const bf16_t* p, float (&x)[8]) {
  const u32x4 a = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[2 * e] = __uint_as_float(a[e] << 16);
    x[2 * e + 1] = __uint_as_float(a[e] & 0xffff0000u);
  }
}

__device__ __forceinline__ void store8(float* p, const float (&x)[8]) {
  *reinterpret_cast<f32x4*>(p) = f32x4{x[0], x[1], x[2], x[3]};
  *reinterpret_cast<f32x4*>(p + 4) = f32x4{x[4], x[5], x[6], x[7]};
}

__device__ __forceinline__ void store8(bf16_t* p, const float (&x)[8]) {
  u32x4 a;
#pragma unroll
  for (int e = 0; e < 4; ++e) a[e] = pack_bf16x2(x[2 * e], x[2 * e + 1]);
  *reinterpret_cast<u32x4*>(p) = a;
}

// ---------------------------------------------------------------------------------
// wave / block reductions (wave64)
// ---------------------------------------------------------------------------------

template <typename V>
__device__ __forceinline__ V wave_sum(V v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

// Wave-wide reductions on DPP and the gfx950 row swaps (VALU only, no LDS round trip):
// xor 1 and xor 2 inside quads, half-row and row mirrors, then row pairs and wave
// halves.  Every lane ends with the result; the combination order is fixed, so a
// floating-point sum is deterministic.
__device__ __forceinline__ uint32_t dpp_perm(uint32_t v, int sel) {
  switch (sel) {
    case 0: return __builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0xB1, 0xF, 0xF, false);
    case 1: return __builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x4E, 0xF, 0xF, false);
    case 2: return __builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x141, 0xF, 0xF, false);
    default: return __builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x140, 0xF, 0xF, false);
  }
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) v = max(v, dpp_perm(v, sel));
  const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
  v = max(static_cast<uint32_t>(p[0]), static_cast<uint32_t>(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(v, v, false, false);
  return max(static_cast<uint32_t>(q[0]), static_cast<uint32_t>(q[1]));
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) v += __uint_as_float(dpp_perm(__float_as_uint(v), sel));
  const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(static_cast<uint32_t>(p[0])) + __uint_as_float(static_cast<uint32_t>(p[1]));
  const auto q = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(static_cast<uint32_t>(q[0])) + __uint_as_float(static_cast<uint32_t>(q[1]));
}

__device__ __forceinline__ int wave_sum_i32(int v) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) v += static_cast<int>(dpp_perm(static_cast<uint32_t>(v), sel));
  const auto p = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(v), static_cast<uint32_t>(v), false, false);
  v = static_cast<int>(p[0]) + static_cast<int>(p[1]);
  const auto q = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(v), static_cast<uint32_t>(v), false, false);
  return static_cast<int>(q[0]) + static_cast<int>(q[1]);
}

// Inclusive prefix sum over the 64 lanes (DPP row shifts, then row broadcasts).
// Inclusive prefix sum within each row of 16 lanes (the row-local steps of the wave scan
// below); every lane of the row must be active.
__device__ __forceinline__ int row16_incl_scan_i32(int v) {
  const int x = v;
  v += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, x, 0x113, 0xF, 0xF, false);  // row_shr:3
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xE, false);  // row_shr:4, banks 1-3
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xC, false);  // row_shr:8, banks 2-3
  return v;
}

__device__ __forceinline__ int wave_incl_scan_i32(int v) {
  const int x = v;
  v += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, x, 0x113, 0xF, 0xF, false);  // row_shr:3
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xE, false);  // row_shr:4, banks 1-3
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xC, false);  // row_shr:8, banks 2-3
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xA, 0xF, false);  // row_bcast:15, rows 1, 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xC, 0xF, false);  // row_bcast:31, rows 2, 3
  return v;
}

// Lanes shifted by a DPP row control; lanes without a source (row edge, masked rows or
// banks) read +0.0.
template <int CTRL, int ROW_MASK, int BANK_MASK>
__device__ __forceinline__ double dpp_shift_f64(double v) {
  const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
  const uint32_t lo = __builtin_amdgcn_update_dpp(0u, static_cast<uint32_t>(u), CTRL, ROW_MASK, BANK_MASK, false);
  const uint32_t hi = __builtin_amdgcn_update_dpp(0u, static_cast<uint32_t>(u >> 32), CTRL, ROW_MASK, BANK_MASK, false);
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}

// Inclusive prefix sum over the wave in fp64 (same steps as the integer scan above).
__device__ __forceinline__ double wave_incl_scan_f64(double v) {
  const double x = v;
  v += dpp_shift_f64<0x111, 0xF, 0xF>(x);
  v += dpp_shift_f64<0x112, 0xF, 0xF>(x);
  v += dpp_shift_f64<0x113, 0xF, 0xF>(x);
  v += dpp_shift_f64<0x114, 0xF, 0xE>(v);
  v += dpp_shift_f64<0x118, 0xF, 0xC>(v);
  v += dpp_shift_f64<0x142, 0xA, 0xF>(v);
  v += dpp_shift_f64<0x143, 0xC, 0xF>(v);
  return v;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const uint64_t lo = dpp_perm(static_cast<uint32_t>(u), sel);
    const uint64_t hi = dpp_perm(static_cast<uint32_t>(u >> 32), sel);
    v += __longlong_as_double(static_cast<long long>((hi << 32) | lo));
  }
  {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const auto pl = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(u), static_cast<uint32_t>(u), false, false);
    const auto ph = __builtin_amdgcn_permlane16_swap(static_cast<uint32_t>(u >> 32), static_cast<uint32_t>(u >> 32), false, false);
    v = __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(static_cast<uint32_t>(ph[0])) << 32) | static_cast<uint32_t>(pl[0]))) +
        __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(static_cast<uint32_t>(ph[1])) << 32) | static_cast<uint32_t>(pl[1])));
  }
  {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const auto pl = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(u), static_cast<uint32_t>(u), false, false);
    const auto ph = __builtin_amdgcn_permlane32_swap(static_cast<uint32_t>(u >> 32), static_cast<uint32_t>(u >> 32), false, false);
    v = __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(static_cast<uint32_t>(ph[0])) << 32) | static_cast<uint32_t>(pl[0]))) +
        __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(static_cast<uint32_t>(ph[1])) << 32) | static_cast<uint32_t>(pl[1])));
  }
  return v;
}

// Sum over the 16 lanes that share lane / 16 (one MFMA 16x16 output row group).
__device__ __forceinline__ float sum16(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// ---------------------------------------------------------------------------------
// MFMA wrappers (CDNA4 16x16 tiles, fp32 accumulate)
//   bf16, K = 32: lane l holds A[l % 16][8 (l / 16) + 0..7] and B[8 (l / 16) + 0..7][l % 16]
//   fp32, K = 4 : lane l holds A[l % 16][l / 16]            and B[l / 16][l % 16]
//   output      : lane l holds D[4 (l / 16) + 0..3][l % 16]
// ---------------------------------------------------------------------------------

__device__ __forceinline__ f32x4 mfma_bf16_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// In-place accumulation: the accumulator is pinned to one register tuple (the
// compiler's own allocation of loop-carried accumulators otherwise rotates them and
// inserts copies that drain the matrix pipeline every iteration).  Back-to-back MFMAs
// on the same accumulator are interlocked in hardware; vector reads of the results
// must be preceded by mfma_results_ready().
__device__ __forceinline__ void mfma_bf16_16x16x32_acc(f32x4& c, bf16x8 a, bf16x8 b) {
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

// Wait states between the last in-place MFMA and vector reads of its results (more
// than the longest MFMA's latency); the scheduling barrier keeps the compiler from
// moving the reads above the padding.
__device__ __forceinline__ void mfma_results_ready() {
  asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Bit pattern of a float as an unsigned key whose integer order is the float order
// (-0 is mapped onto +0 first so that the two zeros tie, as they compare equal).
__device__ __forceinline__ uint32_t order_key(float f) {
  // adding +0 turns -0 into +0 (round to nearest), so both zeros share one key
  const uint32_t u = __float_as_uint(f + 0.0f);
  return u ^ (static_cast<uint32_t>(static_cast<int32_t>(u) >> 31) | 0x80000000u);
}

__device__ __forceinline__ float key_to_float(uint32_t k) {
  uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
  return __uint_as_float(u);
}

// Sticky data-error bits (same values as the public header).
constexpr uint32_t kErrNodeOff = 0x1u;
constexpr uint32_t kErrMemOff = 0x2u;
constexpr uint32_t kErrDepth = 0x4u;
constexpr uint32_t kErrTau = 0x8u;

}  // namespace fovea
