// Correction kernels (paper, Method: correction and gate equation and Eq.
// hidden_correction; appendix: two biased linear layers, 512-wide SiLU hidden layer,
// scalar gate broadcast over the hidden size) and the memory-build projection.
#pragma once

#include "common.hpp"
#include "gemm.hpp"

namespace fovea {

template <typename T>
using Corr1Cfg = GemmCfg<T, 64, 4>;
template <typename T, int BM = 128>
using Corr2Cfg = GemmCfg<T, BM, 2>;
// memory build: 256-row tiles (three 48 KB stages, two thirds of a 128-row tile's operand
// bytes per multiply-add) for bf16 memories of many rows, else 128-row tiles
template <typename T, int BM = 128>
using MemCfg = GemmCfg<T, BM, BM == 256 ? 3 : 4>;
constexpr int kPartCols = 128;  // columns reduced into one partial sum (one block tile)

__host__ __device__ constexpr int n_parts(int cols) { return (cols + kPartCols - 1) / kPartCols; }

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + expf(-x)); }
__device__ __forceinline__ float sigmoid_f(float x) { return 1.0f / (1.0f + expf(-x)); }

// Layer 1 of both nets: [a_c | a_g] = SiLU(P + r W1r^T + [b_c1 ; b_g1]), where P = h W1h^T
// comes from the hidden-state GEMM, so only the r half (K = d_m) is computed here.
// a_c (correction hidden) is stored in the storage dtype for layer 2; the gate hidden
// a_g is consumed here: each block reduces SiLU(.) * w_g2 over its 128 columns into one
// partial of the gate logit per row (gate_part[row][tile column], deterministic order;
// tiles without gate columns write 0).
template <typename T>
struct Corr1Epi {
  int n, d_c, N;
  const float* P;
  const float* b1;
  const float* w_g2;
  T* a_c;
  __device__ __forceinline__ float operator()(int row, int col0, const float (&v)[8]) const {
    if (row >= n || col0 >= N) return 0.f;
    float p[8];
    load8(P + static_cast<int64_t>(row) * N + col0, p);
    return finish(row, col0, v, p);
  }
  // the epilogue for 8 columns whose P is given
  __device__ __forceinline__ float finish(int row, int col0, const float (&v)[8], const float (&p)[8]) const {
    float b[8], pre[8];
    load8(b1 + col0, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) pre[e] = v[e] + p[e] + b[e];
    if (col0 < d_c) {
#pragma unroll
      for (int e = 0; e < 8; ++e) pre[e] = silu_f(pre[e]);
      store8(a_c + static_cast<int64_t>(row) * d_c + col0, pre);
      return 0.f;
    }
    float wg[8];
    load8(w_g2 + (col0 - d_c), wg);
    float acc_g = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc_g = fmaf(silu_f(pre[e]), wg[e], acc_g);
    return acc_g;
  }
};

struct RowPart {  // part[row][tile] = sum (rows past n dropped)
  int n, n_tiles, tile;
  float* part;
  __device__ __forceinline__ void operator()(int row, float sum) const {
    if (part != nullptr && row < n) part[static_cast<int64_t>(row) * n_tiles + tile] = sum;
  }
};

// ks > 1: split-K (grid.y = ks slices, fp32 partials in part), finished by
// corr1_combine_kernel with the same epilogue.
template <typename T>
__global__ __launch_bounds__(256) void corr1_kernel(TileMap tm, const T* __restrict__ rT, int d_m,
                                                    const T* __restrict__ W1r, Corr1Epi<T> epi,
                                                    float* __restrict__ gate_part, int ks,
                                                    float* __restrict__ part) {
  using C = Corr1Cfg<T>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  if (ks > 1) {
    gemm_splitk_partial<C>(rT, d_m, epi.n, W1r, d_m, epi.N, d_m, ks, m0, n0, part, smem);
    return;
  }
  // each thread's P for the epilogue (8 fp32 per epilogue group, rows and columns clamped
  // into the matrix) is loaded before the mainloop, so that its latency hides behind the
  // matrix work
  constexpr int PRE = C::WM * C::SROWS * 16 / C::NT;
  f32x4 ppre[PRE][2];
#pragma unroll
  for (int gi = 0; gi < PRE; ++gi) {
    int row, col0;
    epilogue_group<C>(gi, m0, n0, row, col0);
    const float* pp = epi.P + static_cast<int64_t>(min(row, epi.n - 1)) * epi.N + min(col0, epi.N - 8);
    ppre[gi][0] = *reinterpret_cast<const f32x4*>(pp);
    ppre[gi][1] = *reinterpret_cast<const f32x4*>(pp + 4);
  }
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, rT, d_m, epi.n, W1r, d_m, epi.N, d_m, m0, n0, smem);
  gemm_epilogue<C>(
      acc, smem, m0, n0,
      [&](int row, int col0, const float(&v)[8], int gi) -> float {
        if (row >= epi.n || col0 >= epi.N) return 0.f;
        const float p[8] = {ppre[gi][0][0], ppre[gi][0][1], ppre[gi][0][2], ppre[gi][0][3],
                            ppre[gi][1][0], ppre[gi][1][1], ppre[gi][1][2], ppre[gi][1][3]};
        return epi.finish(row, col0, v, p);
      },
      RowPart{epi.n, n_parts(epi.N), tc, gate_part});
}

template <typename T>
__global__ __launch_bounds__(256) void corr1_combine_kernel(Corr1Epi<T> epi, float* __restrict__ gate_part,
                                                            int ks, const float* __restrict__ part) {
  splitk_combine(epi.n, epi.N, ks, part, epi,
                 RowPart{epi.n, n_parts(epi.N), static_cast<int>(blockIdx.x), gate_part});
}

// Layer 2 and the gated residual: c = a_c W_c2^T + b_c2, g = sigmoid(sum(gate_part) + b_g2),
// h' = h + g c.  Without RMSNorm h' is the output; with it, h' goes to h_out and each
// block writes the partial sum of h'^2 over its 128 columns (rms_part[row][tile column]).
// sg holds the gate of rows m0 .. (staged per block).
template <typename T>
struct Corr2Epi {
  int n, d;
  const float* b_c2;
  const T* h;
  T* h_out;
  const float* sg;
  int m0;
  __device__ __forceinline__ float operator()(int row, int col0, const float (&v)[8]) const {
    if (row >= n || col0 >= d) return 0.f;
    const float g = sg[row - m0];
    const int64_t o = static_cast<int64_t>(row) * d + col0;
    float hv[8], b[8], hp[8];
    load8(h + o, hv);
    load8(b_c2 + col0, b);
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      hp[e] = fmaf(g, v[e] + b[e], hv[e]);
      ss = fmaf(hp[e], hp[e], ss);
    }
    store8(h_out + o, hp);
    return ss;
  }
};

struct Corr2Args {
  int d_c;
  const float* gate_part;
  float b_g2;
  float* gate_out;
  float* rms_part;  // or null without RMSNorm
};

// gate of `rows` rows from m0 into sg (threads < rows); tile-0 blocks also write gate_out
__device__ __forceinline__ void stage_gates(const Corr2Args& ca, int n, int m0, int rows, bool first,
                                            float* sg) {
  if (threadIdx.x < static_cast<unsigned>(rows)) {
    const int n_gp = n_parts(2 * ca.d_c);
    const int row = m0 + threadIdx.x;
    float g = 0.f;
    if (row < n) {
      float sum = 0.f;
      for (int p2 = 0; p2 < n_gp; ++p2) sum += ca.gate_part[static_cast<int64_t>(row) * n_gp + p2];
      g = sigmoid_f(sum + ca.b_g2);
      if (ca.gate_out != nullptr && first) ca.gate_out[row] = g;
    }
    sg[threadIdx.x] = g;
  }
}

template <typename T, int BM = 128>
__global__ __launch_bounds__(256) void corr2_kernel(TileMap tm, const T* __restrict__ a_c,
                                                    const T* __restrict__ Wc2, Corr2Epi<T> epi,
                                                    Corr2Args ca, int ks, float* __restrict__ part) {
  using C = Corr2Cfg<T, BM>;
  static_assert(C::SMEM_BYTES >= C::OUT_BYTES + C::BM * 4, "gate staging");
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  if (ks > 1) {
    gemm_splitk_partial<C>(a_c, ca.d_c, epi.n, Wc2, ca.d_c, epi.d, ca.d_c, ks, m0, n0, part, smem);
    return;
  }
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, a_c, ca.d_c, epi.n, Wc2, ca.d_c, epi.d, ca.d_c, m0, n0, smem);
  // gate of each row of the tile, next to the epilogue's staging area
  float* sg = reinterpret_cast<float*>(smem + C::OUT_BYTES);
  stage_gates(ca, epi.n, m0, C::BM, tc == 0, sg);
  // (the epilogue's first barrier orders these writes before any read)
  epi.sg = sg;
  epi.m0 = m0;
  gemm_epilogue<C>(acc, smem, m0, n0, epi, RowPart{epi.n, n_parts(epi.d), tc, ca.rms_part});
}

template <typename T>
__global__ __launch_bounds__(256) void corr2_combine_kernel(Corr2Epi<T> epi, Corr2Args ca, int ks,
                                                            const float* __restrict__ part) {
  __shared__ float sg[16];
  const int m0 = static_cast<int>(blockIdx.y) * 16;
  stage_gates(ca, epi.n, m0, 16, blockIdx.x == 0, sg);
  __syncthreads();
  epi.sg = sg;
  epi.m0 = m0;
  splitk_combine(epi.n, epi.d, ks, part, epi,
                 RowPart{epi.n, n_parts(epi.d), static_cast<int>(blockIdx.x), ca.rms_part});
}

// Split-K layer 2 and the RMSNorm in one pass, one 256-thread block per row (d at most
// 8192: thread t owns the 8-column groups 8 t + 2048 j, j < 4): the ks partials are added
// in slice order, h' = h + g (c + b_c2) as in Corr2Epi, the sum of squares of h' is
// reduced over the block, and h_out = T(h') / sqrt(mean(h'^2) + eps) * w.
constexpr int kCorr2RmsMaxD = 8 * 256 * 4;

template <typename T>
__global__ __launch_bounds__(256) void corr2_rms_kernel(Corr2Epi<T> epi, Corr2Args ca, int ks,
                                                        const float* __restrict__ part,
                                                        const float* __restrict__ w, float eps) {
  __shared__ float sg[1];
  __shared__ float red[4];
  const int row = blockIdx.x;
  stage_gates(ca, epi.n, row, 1, true, sg);
  __syncthreads();
  const float g = sg[0];
  const int n = epi.n, d = epi.d;
  float hp[4][8];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col0 = 8 * static_cast<int>(threadIdx.x) + 2048 * j;
    if (col0 < d) {
      float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int y0 = 0; y0 < ks; y0 += 4) {
        float t[4][8];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (y0 + u < ks) load8(part + (static_cast<int64_t>(y0 + u) * n + row) * d + col0, t[u]);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (y0 + u < ks)
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += t[u][e];
      }
      float hv[8], b[8];
      load8(epi.h + static_cast<int64_t>(row) * d + col0, hv);
      load8(epi.b_c2 + col0, b);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hp[j][e] = fmaf(g, v[e] + b[e], hv[e]);
        ss = fmaf(hp[j][e], hp[j][e], ss);
      }
    }
  }
  ss = wave_sum_f32(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float rstd = 1.0f / sqrtf(((red[0] + red[1]) + (red[2] + red[3])) / static_cast<float>(d) + eps);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col0 = 8 * static_cast<int>(threadIdx.x) + 2048 * j;
    if (col0 < d) {
      float wv[8], o[8];
      load8(w + col0, wv);
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = Elem<T>::to_f32(Elem<T>::from_f32(hp[j][e])) * rstd * wv[e];
      store8(epi.h_out + static_cast<int64_t>(row) * d + col0, o);
    }
  }
}

// RMSNorm of h' in place: h_out = h' / sqrt(mean(h'^2) + eps) * w, one wave per row,
// 16-byte accesses (8 consecutive columns per lane and step); d is a multiple of 64.
template <typename T>
__global__ __launch_bounds__(256) void rms_kernel(int n, int d, const float* __restrict__ rms_part,
                                                  const float* __restrict__ w, float eps,
                                                  T* __restrict__ h_out) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const int n_rp = n_parts(d);
  float s2 = 0.f;
  for (int p2 = lane; p2 < n_rp; p2 += 64) s2 += rms_part[static_cast<int64_t>(row) * n_rp + p2];
  const float rstd = 1.0f / sqrtf(wave_sum_f32(s2) / static_cast<float>(d) + eps);
  T* hr = h_out + static_cast<int64_t>(row) * d;
  for (int c0 = 8 * lane; c0 < d; c0 += 8 * 64) {
    float v[8], wv[8];
    load8(hr + c0, v);
    load8(w + c0, wv);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = v[e] * rstd * wv[e];
    store8(hr + c0, v);
  }
}

// Memory build: [keys | values] = LN(V) [W_K ; W_U]^T with the LayerNorm folded into the
// epilogue exactly as in the query projection (c1 = W' 1, c2 = W b).
template <typename T, int BM = 128>
__global__ __launch_bounds__(256) void mem_proj_kernel(TileMap tm, int n, const T* __restrict__ V,
                                                       int d_v, const T* __restrict__ Wku, int d_m,
                                                       const float2* __restrict__ stats,
                                                       const float* __restrict__ c1,
                                                       const float* __restrict__ c2,
                                                       T* __restrict__ keys, T* __restrict__ values) {
  using C = MemCfg<T, BM>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  const int N = 2 * d_m;
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, V, d_v, n, Wku, d_v, N, d_v, m0, n0, smem);
  gemm_epilogue<C>(
      acc, smem, m0, n0,
      [&](int row, int col0, const float(&v)[8]) -> float {
        if (row >= n || col0 >= N) return 0.f;
        const float2 st = stats[row];
        float a[8], b[8], val[8];
        load8(c1 + col0, a);
        load8(c2 + col0, b);
#pragma unroll
        for (int e = 0; e < 8; ++e) val[e] = st.y * (v[e] - st.x * a[e]) + b[e];
        if (col0 < d_m)
          store8(keys + static_cast<int64_t>(row) * d_m + col0, val);
        else
          store8(values + static_cast<int64_t>(row) * d_m + (col0 - d_m), val);
        return 0.f;
      },
      NoRowSum{});
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
