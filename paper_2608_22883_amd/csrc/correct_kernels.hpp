// Correction kernels (paper, Method: correction and gate equation and Eq.
// hidden_correction; appendix: two biased linear layers, 512-wide SiLU hidden layer,
// scalar gate broadcast over the hidden size) and the memory-build projection.
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace fovea {

constexpr int kCorrWM = 2, kCorrWN = 2, kCorrTM = 2, kCorrTN = 4;  // 64 x 128 block tile
constexpr int kPartCols = kCorrTN * 16;  // columns reduced into one partial sum (one wave)

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + expf(-x)); }
__device__ __forceinline__ float sigmoid_f(float x) { return 1.0f / (1.0f + expf(-x)); }

// Layer 1 of both nets in one GEMM: [a_c | a_g] = SiLU([h ; r] [W_c1 ; W_g1]^T + [b_c1 ; b_g1]).
// a_c (correction hidden) is stored in the storage dtype for layer 2; the gate hidden
// a_g is consumed here: each wave reduces SiLU(.) * w_g2 over its 64 columns into one
// partial of the gate logit per row (gate_part[row][slot], deterministic order).
template <typename T>
__global__ __launch_bounds__(256) void corr1_kernel(int n, const T* __restrict__ h, int d,
                                                    const T* __restrict__ rT, int d_m,
                                                    const T* __restrict__ W1,
                                                    const float* __restrict__ b1, int d_c,
                                                    const float* __restrict__ w_g2,
                                                    T* __restrict__ a_c,
                                                    float* __restrict__ gate_part) {
  constexpr int WM = kCorrWM, WN = kCorrWN, TM = kCorrTM, TN = kCorrTN;
  using C = GemmCfg<T, WM, WN, TM, TN>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  const int N = 2 * d_c, K = d + d_m;
  f32x4 acc[TM][TN];
  gemm_mainloop<T, WM, WN, TM, TN>(acc, AConcat<T>{h, d, rT, d_m, d}, n, W1, K, N, K, m0, n0,
                                   reinterpret_cast<T*>(smem));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int col_base = n0 + wn * TN * 16;
  if (col_base >= N) return;
  const int n_gp = d_c / kPartCols;
  if (col_base < d_c) {
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = col_base + j * 16 + (lane & 15);
      const float bias = b1[col];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int row = m0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + v;
          if (row < n) st_f32(a_c, static_cast<int64_t>(row) * d_c + col, silu_f(acc[i][j][v] + bias));
        }
    }
  } else {
    float wg[TN], bias[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int col = col_base + j * 16 + (lane & 15);
      bias[j] = b1[col];
      wg[j] = w_g2[col - d_c];
    }
    const int slot = (col_base - d_c) / kPartCols;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < TN; ++j) s = fmaf(silu_f(acc[i][j][v] + bias[j]), wg[j], s);
        s = sum16(s);
        const int row = m0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + v;
        if ((lane & 15) == 0 && row < n) gate_part[static_cast<int64_t>(row) * n_gp + slot] = s;
      }
  }
}

// Layer 2 and the gated residual: c = a_c W_c2^T + b_c2, g = sigmoid(sum(gate_part) + b_g2),
// h' = h + g c.  Without RMSNorm h' is the output; with it, h' goes to h_out and each
// wave writes the partial sum of h'^2 over its 64 columns (rms_part[row][slot]).
template <typename T>
__global__ __launch_bounds__(256) void corr2_kernel(int n, const T* __restrict__ a_c, int d_c,
                                                    const T* __restrict__ Wc2, int d,
                                                    const float* __restrict__ b_c2,
                                                    const float* __restrict__ gate_part,
                                                    float b_g2, const T* __restrict__ h,
                                                    T* __restrict__ h_out,
                                                    float* __restrict__ gate_out,
                                                    float* __restrict__ rms_part, int has_rms) {
  constexpr int WM = kCorrWM, WN = kCorrWN, TM = kCorrTM, TN = kCorrTN;
  using C = GemmCfg<T, WM, WN, TM, TN>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  f32x4 acc[TM][TN];
  gemm_mainloop<T, WM, WN, TM, TN>(acc, ASingle<T>{a_c, d_c}, n, Wc2, d_c, d, d_c, m0, n0,
                                   reinterpret_cast<T*>(smem));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int col_base = n0 + wn * TN * 16;
  if (col_base >= d) return;
  const int n_gp = d_c / kPartCols;
  const int n_rp = d / kPartCols;
  float bias[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) bias[j] = b_c2[col_base + j * 16 + (lane & 15)];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + v;
      const bool live = row < n;
      float g = 0.f;
      if (live) {
        float s = 0.f;
        for (int p = 0; p < n_gp; ++p) s += gate_part[static_cast<int64_t>(row) * n_gp + p];
        g = sigmoid_f(s + b_g2);
      }
      float ss = 0.f;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = col_base + j * 16 + (lane & 15);
        if (live) {
          const int64_t o = static_cast<int64_t>(row) * d + col;
          const float hp = fmaf(g, acc[i][j][v] + bias[j], ld_f32(h, o));
          st_f32(h_out, o, hp);
          ss = fmaf(hp, hp, ss);
        }
      }
      if (has_rms) {
        ss = sum16(ss);
        if ((lane & 15) == 0 && live) rms_part[static_cast<int64_t>(row) * n_rp + col_base / kPartCols] = ss;
      }
      if (gate_out != nullptr && blockIdx.y == 0 && wn == 0 && (lane & 15) == 0 && live) gate_out[row] = g;
    }
}

// RMSNorm of h' in place: h_out = h' / sqrt(mean(h'^2) + eps) * w, one block per row.
template <typename T>
__global__ __launch_bounds__(256) void rms_kernel(int n, int d, const float* __restrict__ rms_part,
                                                  const float* __restrict__ w, float eps,
                                                  T* __restrict__ h_out) {
  __shared__ float s_rstd;
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  if (tid < 64) {
    const int n_rp = d / kPartCols;
    float s = 0.f;
    for (int p = tid; p < n_rp; p += 64) s += rms_part[static_cast<int64_t>(row) * n_rp + p];
    s = wave_sum(s);
    if (tid == 0) s_rstd = 1.0f / sqrtf(s / static_cast<float>(d) + eps);
  }
  __syncthreads();
  const float rstd = s_rstd;
  T* hr = h_out + static_cast<int64_t>(row) * d;
  for (int c = tid; c < d; c += 256) st_f32(hr, c, Elem<T>::to_f32(hr[c]) * rstd * w[c]);
}

// Memory build: [keys | values] = LN(V) [W_K ; W_U]^T with the LayerNorm folded into the
// epilogue exactly as in the query projection (c1 = W' 1, c2 = W b).
template <typename T>
__global__ __launch_bounds__(256) void mem_proj_kernel(int n, const T* __restrict__ V, int d_v,
                                                       const T* __restrict__ Wku, int d_m,
                                                       const float2* __restrict__ stats,
                                                       const float* __restrict__ c1,
                                                       const float* __restrict__ c2,
                                                       T* __restrict__ keys, T* __restrict__ values) {
  constexpr int WM = kCorrWM, WN = kCorrWN, TM = kCorrTM, TN = kCorrTN;
  using C = GemmCfg<T, WM, WN, TM, TN>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  const int N = 2 * d_m;
  f32x4 acc[TM][TN];
  gemm_mainloop<T, WM, WN, TM, TN>(acc, ASingle<T>{V, d_v}, n, Wku, d_v, N, d_v, m0, n0,
                                   reinterpret_cast<T*>(smem));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + v;
      if (row >= n) continue;
      const float2 st = stats[row];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * TN * 16 + j * 16 + (lane & 15);
        if (col >= N) continue;
        const float val = st.y * (acc[i][j][v] - st.x * c1[col]) + c2[col];
        if (col < d_m)
          st_f32(keys, static_cast<int64_t>(row) * d_m + col, val);
        else
          st_f32(values, static_cast<int64_t>(row) * d_m + (col - d_m), val);
      }
    }
}

// ---------------------------------------------------------------------------------
// context packing
// ---------------------------------------------------------------------------------

// out[i][j] = W[i][j] * g[j], rounded once to the storage dtype (the product of two
// bf16 values is exact in fp32).
template <typename T>
__global__ void fold_gain_kernel(const T* __restrict__ W, const T* __restrict__ g, int64_t rows,
                                 int cols, T* __restrict__ out) {
  const int64_t total = rows * cols;
  for (int64_t i = blockIdx.x * static_cast<int64_t>(blockDim.x) + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x)
    st_f32(out, i, Elem<T>::to_f32(W[i]) * Elem<T>::to_f32(g[i % cols]));
}

// out[l][i] = sum_j W[i][j] * (b[j] + (E ? E[l][j] : 0)), or sum_j W[i][j] when b is
// null; fp64 accumulation, one wave per (l, i).
template <typename T>
__global__ void row_dot_kernel(const T* __restrict__ W, int rows, int cols, const T* __restrict__ b,
                               const T* __restrict__ E, int n_l, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6);
  if (item >= rows * n_l) return;
  const int l = item / rows, i = item % rows;
  const T* wr = W + static_cast<int64_t>(i) * cols;
  double s = 0.0;
  for (int j = lane; j < cols; j += 64) {
    double x = 1.0;
    if (b != nullptr) {
      x = static_cast<double>(Elem<T>::to_f32(b[j]));
      if (E != nullptr) x += static_cast<double>(Elem<T>::to_f32(E[static_cast<int64_t>(l) * cols + j]));
    }
    s += static_cast<double>(Elem<T>::to_f32(wr[j])) * x;
  }
  s = wave_sum(s);
  if (lane == 0) out[item] = static_cast<float>(s);
}

template <typename T>
__global__ void to_f32_kernel(const T* __restrict__ in, int n, float* __restrict__ out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    out[i] = Elem<T>::to_f32(in[i]);
}

}  // namespace fovea
