// MFMA GEMM mainloop for gfx950: acc[m, n] = sum_k A[m, k] * B[n, k].
//
// A is a row-major activation ([rows, K], K contiguous) reached through a source
// functor, so that a concatenation such as [h ; r] is read in place.  B is a row-major
// weight [N, K] (the nn.Linear layout).  Both operands are staged through LDS in
// 16-byte chunks (8 bf16 or 4 fp32): a k-tile is 8 chunks wide, the next tile is
// fetched into registers while the current one feeds the matrix cores.
//
// Block tile BM x BN with BM = WM*TM*16, BN = WN*TN*16, run by WM*WN wave64s; each
// wave owns a TM x TN grid of 16x16 MFMA accumulators.  Rows past M and columns past
// N are clamped on load (the kernels' epilogues drop them on store).
#pragma once

#include <type_traits>

#include "common.hpp"

namespace fovea {

template <typename T, int WM, int WN, int TM, int TN>
struct GemmCfg {
  static constexpr int NT = WM * WN * kWave;
  static constexpr int BM = WM * TM * 16;
  static constexpr int BN = WN * TN * 16;
  static constexpr int VEC = Elem<T>::kPer16B;  // elements per 16-byte chunk
  static constexpr int BK = 8 * VEC;            // k-tile: 64 bf16 or 32 fp32
  static constexpr int LDK = BK + VEC;          // LDS row pitch, padded by one chunk
  static constexpr int A_CHUNKS = BM * 8 / NT;
  static constexpr int B_CHUNKS = BN * 8 / NT;
  static constexpr int SMEM_BYTES = (BM + BN) * LDK * static_cast<int>(sizeof(T));
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "tile does not split over the threads");
};

// A operand read from one row-major matrix.
template <typename T>
struct ASingle {
  const T* p;
  int64_t ld;
  __device__ __forceinline__ const T* at(int row, int k) const { return p + row * ld + k; }
};

// A operand read from the concatenation [x0 | x1] of two row-major matrices along k;
// k0 (the width of x0) is a multiple of the k-tile.
template <typename T>
struct AConcat {
  const T* p0;
  int64_t ld0;
  const T* p1;
  int64_t ld1;
  int k0;
  __device__ __forceinline__ const T* at(int row, int k) const {
    return k < k0 ? p0 + row * ld0 + k : p1 + row * ld1 + (k - k0);
  }
};

template <typename T, int WM, int WN, int TM, int TN, class ASrc>
__device__ __forceinline__ void gemm_mainloop(f32x4 (&acc)[TM][TN], const ASrc& a, int M,
                                              const T* __restrict__ Bw, int64_t ldb, int N,
                                              int K, int m0, int n0, T* smem) {
  using C = GemmCfg<T, WM, WN, TM, TN>;
  T* As = smem;
  T* Bs = smem + C::BM * C::LDK;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN;
  const int wn = wave % WN;

#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 ra[C::A_CHUNKS];
  u32x4 rb[C::B_CHUNKS];
  const T* Aw = As + (wm * TM * 16 + (lane & 15)) * C::LDK;
  const T* Bwv = Bs + (wn * TN * 16 + (lane & 15)) * C::LDK;
  const int nk = K / C::BK;

  for (int kt = 0; kt <= nk; ++kt) {
    // fetch k-tile kt into registers (global -> VGPR)
    if (kt < nk) {
      const int k0 = kt * C::BK;
#pragma unroll
      for (int j = 0; j < C::A_CHUNKS; ++j) {
        const int c = tid + j * C::NT;
        const int row = min(m0 + (c >> 3), M - 1);
        ra[j] = *reinterpret_cast<const u32x4*>(a.at(row, k0 + (c & 7) * C::VEC));
      }
#pragma unroll
      for (int j = 0; j < C::B_CHUNKS; ++j) {
        const int c = tid + j * C::NT;
        const int row = min(n0 + (c >> 3), N - 1);
        rb[j] = *reinterpret_cast<const u32x4*>(Bw + row * ldb + k0 + (c & 7) * C::VEC);
      }
    }
    // consume k-tile kt - 1 from LDS while tile kt is in flight
    if (kt > 0) {
      if constexpr (std::is_same<T, bf16_t>::value) {
#pragma unroll
        for (int kk = 0; kk < C::BK; kk += 32) {
          bf16x8 af[TM], bf[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i)
            af[i] = *reinterpret_cast<const bf16x8*>(Aw + i * 16 * C::LDK + kk + (lane >> 4) * 8);
#pragma unroll
          for (int j = 0; j < TN; ++j)
            bf[j] = *reinterpret_cast<const bf16x8*>(Bwv + j * 16 * C::LDK + kk + (lane >> 4) * 8);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_bf16_16x16x32(af[i], bf[j], acc[i][j]);
        }
      } else {
#pragma unroll
        for (int kk = 0; kk < C::BK; kk += 4) {
          float af[TM], bf[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) af[i] = Aw[i * 16 * C::LDK + kk + (lane >> 4)];
#pragma unroll
          for (int j = 0; j < TN; ++j) bf[j] = Bwv[j * 16 * C::LDK + kk + (lane >> 4)];
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma_f32_16x16x4(af[i], bf[j], acc[i][j]);
        }
      }
    }
    if (kt == nk) break;
    __syncthreads();  // everyone is done reading tile kt - 1
#pragma unroll
    for (int j = 0; j < C::A_CHUNKS; ++j) {
      const int c = tid + j * C::NT;
      *reinterpret_cast<u32x4*>(As + (c >> 3) * C::LDK + (c & 7) * C::VEC) = ra[j];
    }
#pragma unroll
    for (int j = 0; j < C::B_CHUNKS; ++j) {
      const int c = tid + j * C::NT;
      *reinterpret_cast<u32x4*>(Bs + (c >> 3) * C::LDK + (c & 7) * C::VEC) = rb[j];
    }
    __syncthreads();  // tile kt is in LDS
  }
}

}  // namespace fovea
