// Backward of one draft step (paper, Method, training objective; appendix, draft model
// training: the module is trained end to end, the selected sets are a discrete choice
// and are held fixed).  Given dL/dh_hat it produces dL/dh, dL/dkeys, dL/dvalues and the
// gradients of every per-step weight, in fp32, from the raw (unfolded) fp32 weights.
//
// Forward quantities are recomputed rather than saved by the forward (the forward
// keeps none of them):  xhat = (h - mu) rstd, xe = xhat g_q + b_q + E_dep[l],
// q = xe W_Q^T, alpha = softmax over I_n of q . k_i / sqrt(d_m), r = sum alpha_i u_i,
// y = [h; r], z = y [W_c1; W_g1]^T + [b_c1; b_g1], a = SiLU(z), c = a_c W_c2^T + b_c2,
// g = sigmoid(a_g . w_g2 + b_g2), h' = h + g c.  Then, in order:
//   RMSNorm and gate (per node)      dh' , dc = g dh', dlogit = (dh' . c) g (1 - g),
//                                    dz_g = dlogit w_g2 SiLU'(z_g)
//   layer 2 (GEMM)                   dz_c = (dc W_c2) SiLU'(z_c)
//   layer 1 (GEMM)                   [dh | dr] += dz [W_c1; W_g1]
//   readout and scores (per node)    da_i = dr . u_i, ds_i = alpha_i (da_i - alpha . da),
//                                    dq = sum ds_i k_i / sqrt(d_m),
//                                    du_i += alpha_i dr, dk_i += ds_i q / sqrt(d_m)
//   query (GEMM) and LayerNorm       dxe = dq W_Q, dh += LN backward of dxe g_q
//   weight gradients (GEMMs over the node axis of transposed activations) and
//   bias / gain / E_dep gradients (column sums, deterministic two-stage).
// The memory gradients are accumulated per request in a fixed order (dense rows of
// alpha and ds over the request's memory, then one pass over the request's nodes per
// tile of memory rows), so every output is deterministic.
#pragma once

#include "common.hpp"
#include "correct_kernels.hpp"
#include "gemm.hpp"
#include "retrieve_kernels.hpp"

namespace fovea {

constexpr uint32_t kErrSelection = 0x10u;  // K or an index outside the request's memory
constexpr int kColChunks = 64;             // row chunks of the column sums
constexpr int kColGroups = 8;              // groups (depths) per column-sum pass

__device__ __forceinline__ float dsilu_f(float z) {
  const float s = sigmoid_f(z);
  return s * (1.0f + z * (1.0f - s));
}

// sum over the 256 threads of a block, in every thread (red: 4 floats of LDS)
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum_f32(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// sum_{i < K} w[i] * rows[(m0 + ix[i]) * ld + j + c] for the four columns c < 4 (16-byte loads;
// ld and j multiples of 4), the row loads issued eight at a time so that their latencies overlap
__device__ __forceinline__ f32x4 weighted_rows4(const float* __restrict__ w, const int32_t* __restrict__ ix,
                                                int K, const float* __restrict__ rows, int64_t m0,
                                                int64_t ld, int j) {
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i0 = 0; i0 < K; i0 += 8) {
    f32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u)
      v[u] = i0 + u < K ? *reinterpret_cast<const f32x4*>(rows + (m0 + ix[i0 + u]) * ld + j)
                        : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (i0 + u < K) {
        const float wu = w[i0 + u];
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[c] = fmaf(wu, v[u][c], acc[c]);
      }
  }
  return acc;
}

// out[i] = scale * (x . rows[m0 + ix[i]]) for the entries i = wave, wave + 4, ... < K of
// a 4-wave block (x in LDS, d_m wide): four entries at a time, each lane's loads of all
// four issued together (512 columns per pass).
__device__ __forceinline__ void wave_row_dots(const float* x, const int32_t* __restrict__ ix, int K,
                                              const float* __restrict__ rows, int64_t m0, int d_m,
                                              float scale, float* out, int wave, int lane) {
  for (int i0 = wave; i0 < K; i0 += 16) {
    const float* rp[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) rp[u] = rows + (m0 + ix[min(i0 + 4 * u, K - 1)]) * d_m;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int j0 = 0; j0 < d_m; j0 += 512) {
      float v[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const int j = j0 + lane + 64 * t;
          v[u][t] = j < d_m ? rp[u][j] : 0.f;
        }
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int j = j0 + lane + 64 * t;
        const float xj = j < d_m ? x[j] : 0.f;
#pragma unroll
        for (int u = 0; u < 4; ++u) acc[u] = fmaf(xj, v[u][t], acc[u]);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float sdot = wave_sum_f32(acc[u]);
      if (lane == 0 && i0 + 4 * u < K) out[i0 + 4 * u] = sdot * scale;
    }
  }
}

__global__ __launch_bounds__(256) void fill_f32_kernel(int64_t count, float* __restrict__ p, float v) {
  for (int64_t i = blockIdx.x * 256 + threadIdx.x; i < count; i += static_cast<int64_t>(gridDim.x) * 256)
    p[i] = v;
}

// dst[c * ldd + r] = src[r * lds + c] for r < R, and 0 for R <= r < R_pad (c < C);
// 64 x 64 tiles through LDS.  Grid: (ceil(C / 64), ceil(R_pad / 64)).
__global__ __launch_bounds__(256) void transpose_f32_kernel(int R, int R_pad, int C,
                                                            const float* __restrict__ src,
                                                            int64_t lds, float* __restrict__ dst,
                                                            int64_t ldd) {
  __shared__ float t[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    t[i][tx] = (r < R && c < C) ? src[static_cast<int64_t>(r) * lds + c] : 0.f;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < C && r < R_pad) dst[static_cast<int64_t>(c) * ldd + r] = t[tx][i];
  }
}

// Per node: xhat and xe = xhat g_q + b_q + E_dep[l], and h into y[:, :d] (ld d + d_m).
// Rows of nodes that failed validation are written as zeros.
__global__ __launch_bounds__(256) void bwd_prep_kernel(int n, int d, int d_m,
                                                       const float* __restrict__ h,
                                                       const float2* __restrict__ stats,
                                                       const int32_t* __restrict__ node_req,
                                                       const int32_t* __restrict__ depth, int n_depth,
                                                       const float* __restrict__ g_q,
                                                       const float* __restrict__ b_q,
                                                       const float* __restrict__ E_dep,
                                                       float* __restrict__ xhat,
                                                       float* __restrict__ xe,
                                                       float* __restrict__ y) {
  const int row = blockIdx.x;
  if (row >= n) return;
  const bool ok = node_req[row] >= 0;
  const float2 st = stats[row];
  const int l = min(max(depth[row], 0), n_depth - 1);
  const float* hr = h + static_cast<int64_t>(row) * d;
  const float* er = E_dep + static_cast<int64_t>(l) * d;
  #pragma unroll 8
  for (int j = threadIdx.x; j < d; j += 256) {
    const float x = ok ? (hr[j] - st.x) * st.y : 0.f;
    xhat[static_cast<int64_t>(row) * d + j] = x;
    xe[static_cast<int64_t>(row) * d + j] = ok ? fmaf(x, g_q[j], b_q[j] + er[j]) : 0.f;
    y[static_cast<int64_t>(row) * (d + d_m) + j] = ok ? hr[j] : 0.f;
  }
}

// Per node (one block): validates its K and indices, then recomputes the renormalised
// softmax over the selected entries (alpha [n, k_max]) and the readout r into
// y[:, d:].  ok[n] = 0 marks a node that failed validation (here or in the statistics
// kernel); it contributes nothing to any gradient and its dh row becomes NaN.
__global__ __launch_bounds__(256) void bwd_sel_fwd_kernel(int n, int d, int d_m, int k_max,
                                                          const NodeInfo* __restrict__ info,
                                                          const int32_t* __restrict__ K_in,
                                                          const int32_t* __restrict__ idx,
                                                          const float* __restrict__ q,
                                                          const float* __restrict__ keys,
                                                          const float* __restrict__ values,
                                                          float scale, float* __restrict__ alpha,
                                                          float* __restrict__ y,
                                                          int32_t* __restrict__ ok_out,
                                                          uint32_t* err) {
  extern __shared__ float smem_f[];
  float* sq = smem_f;             // q_n [d_m]
  float* sa = smem_f + d_m;       // scores, then alpha [k_max]
  __shared__ float red[4];
  __shared__ int sbad;
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (row >= n) return;
  const NodeInfo ni = info[row];
  int K = K_in[row];
  if (tid == 0) sbad = 0;
  __syncthreads();
  bool ok = ni.M >= 0;
  if (ok && (K < 0 || K > min(k_max, ni.M))) {
    ok = false;
    if (tid == 0) atomicOr(err, kErrSelection);
  }
  if (ok) {
    for (int i = tid; i < K; i += 256) {
      const int ix = idx[static_cast<int64_t>(row) * k_max + i];
      if (ix < 0 || ix >= ni.M) sbad = 1;
    }
  }
  __syncthreads();
  if (ok && sbad) {
    ok = false;
    if (tid == 0) atomicOr(err, kErrSelection);
  }
  if (tid == 0) ok_out[row] = ok ? 1 : 0;
  if (!ok) K = 0;
  #pragma unroll 8
  for (int j = tid; j < d_m; j += 256) sq[j] = q[static_cast<int64_t>(row) * d_m + j];
  __syncthreads();
  // scores of the selected entries
  wave_row_dots(sq, idx + static_cast<int64_t>(row) * k_max, K, keys, ni.m0, d_m, scale, sa, wave, lane);
  __syncthreads();
  float mx = -INFINITY;
  for (int i = tid; i < K; i += 256) mx = fmaxf(mx, sa[i]);
  mx = wave_max(mx);
  __syncthreads();
  if (lane == 0) red[wave] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float z = 0.f;
  for (int i = tid; i < K; i += 256) z += expf(sa[i] - mx);
  z = block_sum256(z, red);
  for (int i = tid; i < K; i += 256) {
    const float a = expf(sa[i] - mx) / z;
    sa[i] = a;
    alpha[static_cast<int64_t>(row) * k_max + i] = a;
  }
  __syncthreads();
  // r = sum alpha_i u_i, columns over the threads
  const int32_t* ixr = idx + static_cast<int64_t>(row) * k_max;
  for (int j = 4 * tid; j < d_m; j += 1024)
    *reinterpret_cast<f32x4*>(y + static_cast<int64_t>(row) * (d + d_m) + d + j) =
        weighted_rows4(sa, ixr, K, values, ni.m0, d_m, j);
}

// Per node: gate, h' = h + g c, RMSNorm backward, the residual split and the gate's
// backward.  Writes dh (= dh'), dc = g dh', hn = h' rho (for dL/drms_w), dlogit[row] and
// dz[:, d_c:] = dlogit w_g2 SiLU'(z_g).  Nodes with ok = 0 get zero gradients.
__global__ __launch_bounds__(256) void bwd_rms_gate_kernel(int n, int d, int d_c,
                                                           const float* __restrict__ h,
                                                           const float* __restrict__ c,
                                                           const float* __restrict__ z,
                                                           const float* __restrict__ a,
                                                           const float* __restrict__ w_g2, float b_g2,
                                                           const float* __restrict__ rms_w, float eps,
                                                           const float* __restrict__ dh_hat,
                                                           const int32_t* __restrict__ ok_in,
                                                           float* __restrict__ dh,
                                                           float* __restrict__ dc,
                                                           float* __restrict__ hn,
                                                           float* __restrict__ dlogit,
                                                           float* __restrict__ dz) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (row >= n) return;
  const bool ok = ok_in[row] != 0;
  const int64_t ro = static_cast<int64_t>(row) * d;
  const int64_t zo = static_cast<int64_t>(row) * 2 * d_c;
  float t = 0.f;
  #pragma unroll 8
  for (int j = tid; j < d_c; j += 256) t = fmaf(a[zo + d_c + j], w_g2[j], t);
  const float g = sigmoid_f(block_sum256(t, red) + b_g2);
  float rho = 1.f, tw = 0.f;
  if (rms_w != nullptr) {
    float ss = 0.f, sw = 0.f;
    #pragma unroll 8
    for (int j = tid; j < d; j += 256) {
      const float hp = fmaf(g, c[ro + j], h[ro + j]);
      ss = fmaf(hp, hp, ss);
      sw = fmaf(rms_w[j] * dh_hat[ro + j], hp, sw);
    }
    ss = block_sum256(ss, red);
    tw = block_sum256(sw, red);
    rho = 1.0f / sqrtf(ss / static_cast<float>(d) + eps);
  }
  const float k3 = rho * rho * rho * tw / static_cast<float>(d);
  float sdg = 0.f;
  #pragma unroll 8
  for (int j = tid; j < d; j += 256) {
    const float hp = fmaf(g, c[ro + j], h[ro + j]);
    float dhp;
    if (rms_w != nullptr) {
      dhp = rho * rms_w[j] * dh_hat[ro + j] - k3 * hp;
      hn[ro + j] = ok ? hp * rho : 0.f;
    } else {
      dhp = dh_hat[ro + j];
    }
    dhp = ok ? dhp : 0.f;
    dh[ro + j] = dhp;
    dc[ro + j] = g * dhp;
    sdg = fmaf(dhp, c[ro + j], sdg);
  }
  const float dl = block_sum256(sdg, red) * g * (1.0f - g);
  if (tid == 0) dlogit[row] = dl;
  #pragma unroll 8
  for (int j = tid; j < d_c; j += 256) dz[zo + d_c + j] = dl * w_g2[j] * dsilu_f(z[zo + d_c + j]);
}

// Per node: the readout and score backward.  dr [n, d_m]; writes dq [n, d_m] and the
// node's dense rows over its request's memory (m_max wide): wa = alpha_i and
// ws = ds_i / sqrt(d_m) at the selected entries, 0 elsewhere (the selected indices are
// distinct, as the forward produces them).
__global__ __launch_bounds__(256) void bwd_sel_kernel(int n, int d_m, int k_max, int m_max,
                                                      const NodeInfo* __restrict__ info,
                                                      const int32_t* __restrict__ K_in,
                                                      const int32_t* __restrict__ idx,
                                                      const int32_t* __restrict__ ok_in,
                                                      const float* __restrict__ alpha,
                                                      const float* __restrict__ dr,
                                                      const float* __restrict__ keys,
                                                      const float* __restrict__ values,
                                                      float scale, float* __restrict__ dq,
                                                      float* __restrict__ wa,
                                                      float* __restrict__ ws) {
  extern __shared__ float smem_f[];
  float* sdr = smem_f;        // dr_n [d_m]
  float* sds = smem_f + d_m;  // da, then ds [k_max]
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (row >= n) return;
  const int K = ok_in[row] ? K_in[row] : 0;
  const int64_t m0 = info[row].m0;
  const int32_t* ix = idx + static_cast<int64_t>(row) * k_max;
  const float* al = alpha + static_cast<int64_t>(row) * k_max;
  float* war = wa + static_cast<int64_t>(row) * m_max;
  float* wsr = ws + static_cast<int64_t>(row) * m_max;
  for (int i = tid; i < m_max; i += 256) {
    war[i] = 0.f;
    wsr[i] = 0.f;
  }
  #pragma unroll 8
  for (int j = tid; j < d_m; j += 256) sdr[j] = dr[static_cast<int64_t>(row) * d_m + j];
  __syncthreads();
  wave_row_dots(sdr, ix, K, values, m0, d_m, 1.0f, sds, wave, lane);  // da_i = dr . u_i
  __syncthreads();
  float ad = 0.f;
  for (int i = tid; i < K; i += 256) ad = fmaf(al[i], sds[i], ad);
  ad = block_sum256(ad, red);
  for (int i = tid; i < K; i += 256) {
    const float dsi = al[i] * (sds[i] - ad);
    sds[i] = dsi;
    war[ix[i]] = al[i];  // after the zeroing above (block barrier in block_sum256)
    wsr[ix[i]] = dsi * scale;
  }
  __syncthreads();
  for (int j = 4 * tid; j < d_m; j += 1024) {
    const f32x4 v = weighted_rows4(sds, ix, K, keys, m0, d_m, j);
    *reinterpret_cast<f32x4*>(dq + static_cast<int64_t>(row) * d_m + j) =
        f32x4{v[0] * scale, v[1] * scale, v[2] * scale, v[3] * scale};
  }
}

// Memory gradients of one request, one tile of 32 memory rows x 256 columns per block:
//   dvalues[m0 + i] = sum over the request's nodes t of wa[t][i] dr[t]
//   dkeys[m0 + i]   = sum over the request's nodes t of ws[t][i] q[t]
// in node order.  Grid: (ceil(d_m / 256), ceil(m_max / 32), B).
constexpr int kMemRows = 32;

// A request whose memory and node ranges are usable (the memory-gradient kernel writes
// every row of such a request, zeros included)
__device__ __forceinline__ bool mem_request_ok(int64_t m0, int64_t m1, int t0, int t1, int m_max,
                                               int t_max, int n, int64_t n_mem) {
  return 0 <= m0 && m0 <= m1 && m1 <= n_mem && m1 - m0 <= m_max && 0 <= t0 && t0 <= t1 &&
         t1 <= n && t1 - t0 <= t_max;
}

// Zero rows of dkeys and dvalues that no usable request covers (run before
// bwd_mem_grad_kernel, which writes all the others).  16 rows per block, 16 threads per
// row.  The covering request is found by binary search over mem_off; where mem_off is
// not sorted the search may miss a cover, and the zeros written are then overwritten.
__global__ __launch_bounds__(256) void bwd_mem_gaps_kernel(int d_m, int m_max, int t_max, int B,
                                                           const int64_t* __restrict__ mem_off,
                                                           const int32_t* __restrict__ node_off,
                                                           int n, int64_t n_mem,
                                                           float* __restrict__ dkeys,
                                                           float* __restrict__ dvalues) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 16 + (threadIdx.x >> 4);
  if (i >= n_mem) return;
  int lo = 0, hi = B;  // the last b < B with mem_off[b] <= i, else 0
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (mem_off[mid] <= i)
      lo = mid;
    else
      hi = mid;
  }
  const int64_t m0 = mem_off[lo], m1 = mem_off[lo + 1];
  if (mem_request_ok(m0, m1, node_off[lo], node_off[lo + 1], m_max, t_max, n, n_mem) && m0 <= i &&
      i < m1)
    return;
  const f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int j = 4 * (threadIdx.x & 15); j < d_m; j += 64) {
    *reinterpret_cast<f32x4*>(dkeys + i * d_m + j) = z;
    *reinterpret_cast<f32x4*>(dvalues + i * d_m + j) = z;
  }
}

__global__ __launch_bounds__(256) void bwd_mem_grad_kernel(int d_m, int m_max, int t_max,
                                                           const int64_t* __restrict__ mem_off,
                                                           const int32_t* __restrict__ node_off,
                                                           int n, int64_t n_mem,
                                                           const float* __restrict__ wa,
                                                           const float* __restrict__ ws,
                                                           const float* __restrict__ dr,
                                                           const float* __restrict__ q,
                                                           float* __restrict__ dkeys,
                                                           float* __restrict__ dvalues) {
  extern __shared__ float smem_f[];  // [t_max][kMemRows] of wa, then of ws
  float* swa = smem_f;
  float* sws = smem_f + t_max * kMemRows;
  const int b = blockIdx.z, r0 = blockIdx.y * kMemRows;
  const int64_t m0 = mem_off[b], m1 = mem_off[b + 1];
  const int t0 = node_off[b], t1 = node_off[b + 1];
  // offsets were validated per node; a request whose range is unusable is skipped here
  const bool ok = mem_request_ok(m0, m1, t0, t1, m_max, t_max, n, n_mem);
  const int M = ok ? static_cast<int>(m1 - m0) : 0;
  if (r0 >= M) return;
  const int T = t1 - t0;
  // stage the request's rows of wa / ws (eight loads in flight per thread)
  for (int e0 = 0; e0 < T * kMemRows; e0 += 256 * 4) {
    float va[4], vs[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u * 256 + static_cast<int>(threadIdx.x);
      const int t = min(e / kMemRows, T - 1), r = e % kMemRows;
      const int64_t src = static_cast<int64_t>(t0 + t) * m_max + min(r0 + r, m_max - 1);
      va[u] = wa[src];
      vs[u] = ws[src];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int e = e0 + u * 256 + static_cast<int>(threadIdx.x);
      if (e < T * kMemRows) {
        swa[e] = va[u];
        sws[e] = vs[u];
      }
    }
  }
  __syncthreads();
  // wave w owns memory rows r0 + 8 w .. + 7; lane l owns columns j0 .. j0 + 3
  const int wv = threadIdx.x >> 6;
  const int j0 = blockIdx.x * 256 + 4 * (threadIdx.x & 63);
  if (j0 >= d_m) return;
  float au[8][4], ak[8][4];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      au[r][c] = 0.f;
      ak[r][c] = 0.f;
    }
  // the node rows of dr and q come through a 4-deep register prefetch (a request
  // without nodes skips the loop and writes zeros)
  constexpr int PF = 4;
  f32x4 drb[PF], qb[PF];
  if (T > 0) {
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    const int tt = t0 + min(u, T - 1);
    drb[u] = *reinterpret_cast<const f32x4*>(dr + static_cast<int64_t>(tt) * d_m + j0);
    qb[u] = *reinterpret_cast<const f32x4*>(q + static_cast<int64_t>(tt) * d_m + j0);
  }
  for (int tb = 0; tb < T; tb += PF) {
#pragma unroll
  for (int u = 0; u < PF; ++u) {
    const int t = tb + u;
    if (t >= T) break;
    const f32x4 drv = drb[u], qv = qb[u];
    {
      const int tt = t0 + min(t + PF, T - 1);
      drb[u] = *reinterpret_cast<const f32x4*>(dr + static_cast<int64_t>(tt) * d_m + j0);
      qb[u] = *reinterpret_cast<const f32x4*>(q + static_cast<int64_t>(tt) * d_m + j0);
    }
    const f32x4 wa0 = *reinterpret_cast<const f32x4*>(swa + t * kMemRows + 8 * wv);
    const f32x4 wa1 = *reinterpret_cast<const f32x4*>(swa + t * kMemRows + 8 * wv + 4);
    const f32x4 ws0 = *reinterpret_cast<const f32x4*>(sws + t * kMemRows + 8 * wv);
    const f32x4 ws1 = *reinterpret_cast<const f32x4*>(sws + t * kMemRows + 8 * wv + 4);
    const float wa[8] = {wa0[0], wa0[1], wa0[2], wa0[3], wa1[0], wa1[1], wa1[2], wa1[3]};
    const float ws[8] = {ws0[0], ws0[1], ws0[2], ws0[3], ws1[0], ws1[1], ws1[2], ws1[3]};
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        au[r][c] = fmaf(wa[r], drv[c], au[r][c]);
        ak[r][c] = fmaf(ws[r], qv[c], ak[r][c]);
      }
  }
  }
  }
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int i = r0 + 8 * wv + r;
    if (i < M) {
      *reinterpret_cast<f32x4*>(dvalues + (m0 + i) * d_m + j0) = f32x4{au[r][0], au[r][1], au[r][2], au[r][3]};
      *reinterpret_cast<f32x4*>(dkeys + (m0 + i) * d_m + j0) = f32x4{ak[r][0], ak[r][1], ak[r][2], ak[r][3]};
    }
  }
}

// Per node: dh += LayerNorm backward of dxe g_q (xhat, rstd); rows of nodes with
// ok = 0 become NaN (ok_in null: every row is valid).
__global__ __launch_bounds__(256) void bwd_ln_kernel(int n, int d, const float* __restrict__ dxe,
                                                     const float* __restrict__ xhat,
                                                     const float* __restrict__ g_q,
                                                     const float2* __restrict__ stats,
                                                     const int32_t* __restrict__ ok_in,
                                                     float* __restrict__ dh) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (row >= n) return;
  const int64_t ro = static_cast<int64_t>(row) * d;
  float s1 = 0.f, s2 = 0.f;
  #pragma unroll 8
  for (int j = tid; j < d; j += 256) {
    const float t = dxe[ro + j] * g_q[j];
    s1 += t;
    s2 = fmaf(t, xhat[ro + j], s2);
  }
  const float m1 = block_sum256(s1, red) / static_cast<float>(d);
  const float m2 = block_sum256(s2, red) / static_cast<float>(d);
  const float rstd = stats[row].y;
  const bool ok = ok_in == nullptr || ok_in[row] != 0;
  #pragma unroll 8
  for (int j = tid; j < d; j += 256) {
    const float t = dxe[ro + j] * g_q[j];
    dh[ro + j] = ok ? dh[ro + j] + rstd * (t - m1 - xhat[ro + j] * m2) : __builtin_nanf("");
  }
}

// Per row of the memory build's input: xhat = (v - mu) rstd and xn = xhat g + b.
__global__ __launch_bounds__(256) void ln_apply_kernel(int n, int d, const float* __restrict__ x,
                                                       const float2* __restrict__ stats,
                                                       const float* __restrict__ g,
                                                       const float* __restrict__ b,
                                                       float* __restrict__ xhat,
                                                       float* __restrict__ xn) {
  const int row = blockIdx.x;
  if (row >= n) return;
  const float2 st = stats[row];
  const int64_t ro = static_cast<int64_t>(row) * d;
#pragma unroll 8
  for (int j = threadIdx.x; j < d; j += 256) {
    const float v = (x[ro + j] - st.x) * st.y;
    xhat[ro + j] = v;
    xn[ro + j] = fmaf(v, g[j], b[j]);
  }
}

// out[j] = sum_i X[j * ldx + i] (* s[i]) over i < len: one wave per row of a transposed
// (node-minor, zero-padded) array.
__global__ __launch_bounds__(256) void rowsum_kernel(int rows, int len, const float* __restrict__ X,
                                                     int64_t ldx, const float* __restrict__ s,
                                                     float* __restrict__ out) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= rows) return;
  const float* xr = X + static_cast<int64_t>(r) * ldx;
  float acc = 0.f;
  for (int i0 = lane; i0 < len; i0 += 64 * 8) {
    float x[8], w[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + 64 * u;
      x[u] = i < len ? xr[i] : 0.f;
      w[u] = s != nullptr && i < len ? s[i] : 1.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc = fmaf(x[u], w[u], acc);
  }
  acc = wave_sum_f32(acc);
  if (lane == 0) out[r] = acc;
}

// Column sums of several row-major fp32 arrays in one launch.  A job sums over the rows
// i < n of X (16-byte aligned, ldx and cols multiples of 4), each row scaled by rs[i] if
// given, into up to three kinds of outputs:
//   out_x[j]                   = sum_i X[i][j]
//   out_xy[j]                  = sum_i X[i][j] Y[i][j]
//   out_grp[(g0 + g) cols + j] = sum over the rows with grp[i] == g0 + g (g < ng) of X[i][j]
// (a null output is not computed; grp values are clamped to 0 .. n_grp_total - 1).
// Stage 1 writes per-chunk partial sums, stage 2 adds the chunks in a fixed order, so
// every sum is deterministic.
constexpr int kColJobs = 8;
constexpr int kColSlots = 2 + kColGroups;

struct ColJob {
  const float* X;
  int64_t ldx;
  const float* Y;  // nullable (needed for out_xy)
  int64_t ldy;
  const float* rs;       // nullable
  const int32_t* grp;    // nullable (needed for out_grp)
  float* out_x;          // nullable
  float* out_xy;         // nullable
  float* out_grp;        // nullable
  int g0, ng, n_grp_total;
  int cols;
  int64_t part_off;      // floats: this job's partials, [kColChunks][slots][cols]
};

struct ColJobs {
  ColJob job[kColJobs];
  int n_jobs;
};

__device__ __forceinline__ int col_job_slots(const ColJob& jb) {
  return (jb.out_x != nullptr) + (jb.out_xy != nullptr) + (jb.out_grp != nullptr ? jb.ng : 0);
}

// Stage 1: grid (ceil(max cols / 1024), kColChunks, n_jobs); thread t of block x sums the
// columns 4 (256 x + t) .. + 3 over the block's chunk of rows, eight rows in flight.
__global__ __launch_bounds__(256) void colsum_multi_kernel(int n, ColJobs jobs,
                                                           float* __restrict__ part) {
  const ColJob& jb = jobs.job[blockIdx.z];
  const int j = 4 * (blockIdx.x * 256 + threadIdx.x);
  if (j >= jb.cols) return;
  const int per = (n + kColChunks - 1) / kColChunks;
  const int i0 = blockIdx.y * per, i1 = min(n, i0 + per);
  const bool want_x = jb.out_x != nullptr, want_xy = jb.out_xy != nullptr,
             want_g = jb.out_grp != nullptr;
  f32x4 ax = f32x4{0.f, 0.f, 0.f, 0.f}, axy = ax, ag[kColGroups];
#pragma unroll
  for (int g = 0; g < kColGroups; ++g) ag[g] = ax;
  for (int ib = i0; ib < i1; ib += 8) {
    f32x4 x[8], y[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      x[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      y[u] = x[u];
      if (ib + u < i1) {
        x[u] = *reinterpret_cast<const f32x4*>(jb.X + static_cast<int64_t>(ib + u) * jb.ldx + j);
        if (want_xy) y[u] = *reinterpret_cast<const f32x4*>(jb.Y + static_cast<int64_t>(ib + u) * jb.ldy + j);
      }
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (ib + u < i1) {
        const float sc = jb.rs != nullptr ? jb.rs[ib + u] : 1.f;
        f32x4 v;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          v[c] = x[u][c] * sc;
          ax[c] += v[c];
          axy[c] = fmaf(v[c], y[u][c], axy[c]);
        }
        if (want_g) {
          const int g = min(max(jb.grp[ib + u], 0), jb.n_grp_total - 1) - jb.g0;
#pragma unroll
          for (int gg = 0; gg < kColGroups; ++gg) {
            const bool hit = gg == g;
#pragma unroll
            for (int c = 0; c < 4; ++c) ag[gg][c] += hit ? v[c] : 0.f;
          }
        }
      }
    }
  }
  const int slots = col_job_slots(jb);
  float* pp = part + jb.part_off + static_cast<int64_t>(blockIdx.y) * slots * jb.cols + j;
  int sl = 0;
  if (want_x) *reinterpret_cast<f32x4*>(pp + static_cast<int64_t>(sl++) * jb.cols) = ax;
  if (want_xy) *reinterpret_cast<f32x4*>(pp + static_cast<int64_t>(sl++) * jb.cols) = axy;
  if (want_g) {
#pragma unroll
    for (int g = 0; g < kColGroups; ++g)
      if (g < jb.ng) *reinterpret_cast<f32x4*>(pp + static_cast<int64_t>(sl + g) * jb.cols) = ag[g];
  }
}

// Stage 2: grid (ceil(max cols / 256), kColSlots, n_jobs); the chunks' partials of one
// slot added in chunk order.
__global__ __launch_bounds__(256) void colsum_multi_final_kernel(ColJobs jobs,
                                                                 const float* __restrict__ part) {
  const ColJob& jb = jobs.job[blockIdx.z];
  const int j = blockIdx.x * 256 + threadIdx.x;
  const int slots = col_job_slots(jb), sl = blockIdx.y;
  if (j >= jb.cols || sl >= slots) return;
  const float* pp = part + jb.part_off + static_cast<int64_t>(sl) * jb.cols + j;
  const int64_t stride = static_cast<int64_t>(slots) * jb.cols;
  float acc = 0.f;
#pragma unroll 16
  for (int ch = 0; ch < kColChunks; ++ch) acc += pp[ch * stride];
  int k = sl;
  float* out;
  if (jb.out_x != nullptr && k == 0) {
    out = jb.out_x;
  } else {
    k -= jb.out_x != nullptr;
    if (jb.out_xy != nullptr && k == 0) {
      out = jb.out_xy;
    } else {
      k -= jb.out_xy != nullptr;
      out = jb.out_grp + static_cast<int64_t>(jb.g0 + k) * jb.cols;
    }
  }
  out[j] = acc;
}

// fp32 operands as bf16 planes, for GEMMs on the bf16 matrix cores with close to fp32
// accuracy: x = hi + lo + O(2^-16 |x|) with hi = bf16(x), lo = bf16(x - hi), and
//   A B^T = A_hi B_hi^T + A_lo B_hi^T + A_hi B_lo^T + O(2^-16)
// is one bf16 GEMM over a tripled K with A' = [A_hi | A_lo | A_hi] (pattern 0) and
// B' = [B_hi | B_hi | B_lo] (pattern 1).  dst [R, 3 C] row-major.
// Grid: (ceil(C / 1024), R); thread t of block (x, r) converts columns 4 (256 x + t) ..
// + 3 of row r (C a multiple of 4, rows 16-byte aligned).
__global__ __launch_bounds__(256) void split3_kernel(int R, int C, const float* __restrict__ src,
                                                     int64_t lds, bf16_t* __restrict__ dst,
                                                     int pattern) {
  const int r = blockIdx.y;
  const int c = 4 * (blockIdx.x * 256 + static_cast<int>(threadIdx.x));
  if (r >= R || c >= C) return;
  const f32x4 x = *reinterpret_cast<const f32x4*>(src + static_cast<int64_t>(r) * lds + c);
  uint32_t hp[2], lp[2];
#pragma unroll
  for (int e = 0; e < 4; e += 2) {
    const float h0 = bf16_round(x[e]), h1 = bf16_round(x[e + 1]);
    hp[e / 2] = pack_bf16x2(h0, h1);
    lp[e / 2] = pack_bf16x2(x[e] - h0, x[e + 1] - h1);
  }
  const uint2 hv = make_uint2(hp[0], hp[1]), lv = make_uint2(lp[0], lp[1]);
  bf16_t* d = dst + static_cast<int64_t>(r) * 3 * C + c;
  *reinterpret_cast<uint2*>(d) = hv;
  *reinterpret_cast<uint2*>(d + C) = pattern == 0 ? lv : hv;
  *reinterpret_cast<uint2*>(d + 2 * C) = pattern == 0 ? hv : lv;
}

// The planes of src^T: row c of dst (3 W wide, planes W apart) holds column c of src
// [R, C] (ld lds) at positions r_off .. r_off + R_pad - 1 of each plane (rows R .. R_pad - 1
// zero), through 64 x 64 LDS tiles: the node-axis operands of the weight-gradient GEMMs
// and the transposed weights.  Grid: (ceil(C / 64), ceil(R_pad / 64)).  Each thread
// loads 16-byte row pieces and stores 8-byte plane pieces (four source rows): C, R_pad,
// W, r_off and lds multiples of 4, src 16-byte and dst 8-byte aligned.
__global__ __launch_bounds__(256) void transpose_split3_kernel(int R, int R_pad, int C,
                                                               const float* __restrict__ src,
                                                               int64_t lds, bf16_t* __restrict__ dst,
                                                               int W, int r_off, int pattern) {
  __shared__ float t[64][65];
  const int c0 = blockIdx.x * 64, r0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
  // tile row (tid / 16) + 16 p, columns 4 (tid % 16) .. + 3
  const int q = 4 * (tid & 15);
  f32x4 v[4];
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int r = r0 + (tid >> 4) + 16 * p, c = c0 + q;
    v[p] = (r < R && c < C) ? *reinterpret_cast<const f32x4*>(src + static_cast<int64_t>(r) * lds + c)
                            : f32x4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int p = 0; p < 4; ++p)
#pragma unroll
    for (int e = 0; e < 4; ++e) t[(tid >> 4) + 16 * p][q + e] = v[p][e];
  __syncthreads();
  // tile column (tid / 16) + 16 p (a row of dst), tile rows 4 (tid % 16) .. + 3
  const int64_t ldd = 3 * static_cast<int64_t>(W);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int cl = (tid >> 4) + 16 * p, c = c0 + cl, r = r0 + q;
    if (c < C && r < R_pad) {
      float x[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) x[e] = t[q + e][cl];
      uint32_t hp[2], lp[2];
#pragma unroll
      for (int e = 0; e < 4; e += 2) {
        const float h0 = bf16_round(x[e]), h1 = bf16_round(x[e + 1]);
        hp[e / 2] = pack_bf16x2(h0, h1);
        lp[e / 2] = pack_bf16x2(x[e] - h0, x[e + 1] - h1);
      }
      const uint2 hv = make_uint2(hp[0], hp[1]), lv = make_uint2(lp[0], lp[1]);
      bf16_t* d = dst + static_cast<int64_t>(c) * ldd + r_off + r;
      *reinterpret_cast<uint2*>(d) = hv;
      *reinterpret_cast<uint2*>(d + W) = pattern == 0 ? lv : hv;
      *reinterpret_cast<uint2*>(d + 2 * W) = pattern == 0 ? hv : lv;
    }
  }
}

// GEMM C = A B^T (A [M, K], B [N, K], K a multiple of the k-tile, N a multiple of 8) on
// the gemm.hpp core, fp32 or bf16 operands (fp32 accumulation), with the epilogues the
// backward needs.
enum BwdEpi : int {
  kEpiStore = 0,  // out = v (+ bias[col])
  kEpiZ = 1,      // out = v + bias (pre-activation), out2 = SiLU(out)
  kEpiDsilu = 2,  // out = v * SiLU'(aux)
  kEpiSplit = 3,  // col < split: out[col] += v; else out2[col - split] = v
  kEpiRows = 4,   // row < split: out[row] = v; else out2[row - split] = v
};

struct BwdGemm {
  int M, N, K;
  const void* A;  // fp32, or bf16 planes when bf16
  int64_t lda;
  const void* B;
  int64_t ldb;
  bool bf16;
  float* out;
  int64_t ldo;
  const float* bias;   // nullable
  const float* bias2;  // nullable: the bias of the columns from split on (Store, Z)
  float* out2;
  int64_t ldo2;
  const float* aux;
  int64_t ldaux;
  int split;
};

template <typename T, int BM>
using BwdCfg = GemmCfg<T, BM, 4>;

template <int EPI, typename T, int BM>
__global__ __launch_bounds__(256) void bwd_gemm_kernel(TileMap tm, BwdGemm g) {
  using C = BwdCfg<T, BM>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, static_cast<const T*>(g.A), g.lda, g.M, static_cast<const T*>(g.B), g.ldb,
                   g.N, g.K, m0, n0, smem);
  gemm_epilogue<C>(
      acc, smem, m0, n0,
      [&](int row, int col0, const float(&v)[8]) -> float {
        if (row >= g.M || col0 >= g.N) return 0.f;
        float o[8];
        // bias of the column group: bias2 past split when given (8-column groups do not
        // straddle split, a multiple of 8)
        const float* bb = g.bias == nullptr ? nullptr
                          : g.bias2 != nullptr && col0 >= g.split ? g.bias2 + (col0 - g.split)
                                                                   : g.bias + col0;
        if (EPI == kEpiStore || EPI == kEpiZ) {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = v[e] + (bb != nullptr ? bb[e] : 0.f);
          store8(g.out + static_cast<int64_t>(row) * g.ldo + col0, o);
          if (EPI == kEpiZ) {
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = silu_f(o[e]);
            store8(g.out2 + static_cast<int64_t>(row) * g.ldo2 + col0, o);
          }
        } else if (EPI == kEpiDsilu) {
          float zz[8];
          load8(g.aux + static_cast<int64_t>(row) * g.ldaux + col0, zz);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = v[e] * dsilu_f(zz[e]);
          store8(g.out + static_cast<int64_t>(row) * g.ldo + col0, o);
        } else if (EPI == kEpiRows) {
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = v[e];
          if (row < g.split)
            store8(g.out + static_cast<int64_t>(row) * g.ldo + col0, o);
          else
            store8(g.out2 + static_cast<int64_t>(row - g.split) * g.ldo2 + col0, o);
        } else {
          if (col0 < g.split) {
            float* p = g.out + static_cast<int64_t>(row) * g.ldo + col0;
            load8(p, o);
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] += v[e];
            store8(p, o);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = v[e];
            store8(g.out2 + static_cast<int64_t>(row) * g.ldo2 + (col0 - g.split), o);
          }
        }
        return 0.f;
      },
      NoRowSum{});
}

}  // namespace fovea
