// Retrieval kernels: node preparation, query projection, scoring, and the per-node
// cumulative-mass selection with the renormalised gather (paper, Method: query and
// score equation, normalised-score equation, cardinality equation K_r, readout).
#pragma once

#include <climits>

#include "common.hpp"
#include "gemm.hpp"

namespace fovea {

// Limits shared with the host code.
constexpr int kMaxM = 16384;
constexpr int kMaxKmax = 1024;
constexpr int kQSplitBf16 = 3;  // q = hi + mid + lo in bf16 for the score MFMA

// Bounds check of request b's node and memory ranges against the host-side sizes.
struct Extent {
  int64_t m0, m1;
  int t0, t1;
  bool nodes_ok, mem_ok;
};

__device__ __forceinline__ Extent request_extent(int b, const int64_t* mem_off, int64_t n_mem,
                                                 int m_max, const int32_t* node_off,
                                                 int n_nodes, int t_max) {
  Extent e;
  e.t0 = node_off[b];
  e.t1 = node_off[b + 1];
  e.m0 = mem_off[b];
  e.m1 = mem_off[b + 1];
  e.nodes_ok = 0 <= e.t0 && e.t0 <= e.t1 && e.t1 <= n_nodes && e.t1 - e.t0 <= t_max;
  e.mem_ok = 0 <= e.m0 && e.m0 <= e.m1 && e.m1 <= n_mem && e.m1 - e.m0 <= m_max;
  return e;
}

// ---------------------------------------------------------------------------------
// Row statistics of LayerNorm (mean, 1/sqrt(var + eps)), one wave per row.  With
// node_off given it also finds each node's request and validates depth, tau and the
// request's node range; node_req[n] = -1 marks a node whose outputs become NaN.
// ---------------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void row_stats_kernel(int n, const T* __restrict__ x, int d,
                                                        float eps, float2* __restrict__ stats,
                                                        const int32_t* __restrict__ depth,
                                                        int n_depth,
                                                        const int32_t* __restrict__ node_off,
                                                        int B, int t_max,
                                                        const float* __restrict__ tau,
                                                        int32_t* __restrict__ node_req,
                                                        uint32_t* err) {
  constexpr int VEC = Elem<T>::kPer16B;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const T* xr = x + static_cast<int64_t>(row) * d;
  const int nch = d / VEC;
  float s = 0.f;
  for (int c = lane; c < nch; c += kWave) {
    const u32x4 raw = *reinterpret_cast<const u32x4*>(xr + c * VEC);
    const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int j = 0; j < VEC; ++j) s += Elem<T>::to_f32(v[j]);
  }
  const float mu = wave_sum(s) / static_cast<float>(d);
  float ss = 0.f;
  for (int c = lane; c < nch; c += kWave) {
    const u32x4 raw = *reinterpret_cast<const u32x4*>(xr + c * VEC);
    const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      const float t = Elem<T>::to_f32(v[j]) - mu;
      ss = fmaf(t, t, ss);
    }
  }
  const float var = wave_sum(ss) / static_cast<float>(d);
  if (lane == 0) stats[row] = make_float2(mu, 1.0f / sqrtf(var + eps));

  if (node_off != nullptr && lane == 0) {
    // largest b with node_off[b] <= row (a fixed number of steps even if the offsets are bad)
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (node_off[mid] <= row) lo = mid; else hi = mid - 1;
    }
    const int b = lo;
    const int t0 = node_off[b], t1 = node_off[b + 1];
    uint32_t bad = 0;
    if (!(0 <= t0 && t0 <= row && row < t1 && t1 <= n && t1 - t0 <= t_max)) bad |= kErrNodeOff;
    const int dep = depth[row];
    if (dep < 0 || dep >= n_depth) bad |= kErrDepth;
    const float tb = tau[b];
    if (!(tb >= 0.f && tb <= 1.f)) bad |= kErrTau;
    node_req[row] = bad ? -1 : b;
    if (bad) atomicOr(err, bad);
  }
}

// ---------------------------------------------------------------------------------
// Query projection with the LayerNorm folded into the epilogue:
//   q = W_Q (LN(h) + E_dep[l]) = rstd * (W' h - mu * W' 1) + W_Q (b + E_dep[l]),
// W' = W_Q diag(gain) packed at context creation, c1 = W' 1, c2[l] = W_Q (b + E_dep[l]).
// bf16 storage writes q as three bf16 planes hi + mid + lo (exact split of the fp32
// value) for the score MFMA; fp32 storage writes q itself.
// ---------------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void q_proj_kernel(int n, const T* __restrict__ h, int d,
                                                     const T* __restrict__ Wq, int d_m,
                                                     const float2* __restrict__ stats,
                                                     const int32_t* __restrict__ depth,
                                                     const int32_t* __restrict__ node_req,
                                                     int n_depth, const float* __restrict__ c1,
                                                     const float* __restrict__ c2,
                                                     T* __restrict__ q) {
  constexpr int WM = 2, WN = 2, TM = 2, TN = 4;
  using C = GemmCfg<T, WM, WN, TM, TN>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  f32x4 acc[TM][TN];
  gemm_mainloop<T, WM, WN, TM, TN>(acc, ASingle<T>{h, d}, n, Wq, d, d_m, d, m0, n0,
                                   reinterpret_cast<T*>(smem));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int64_t plane = static_cast<int64_t>(n) * d_m;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int row = m0 + wm * TM * 16 + i * 16 + 4 * (lane >> 4) + v;
      if (row >= n) continue;
      const float2 st = stats[row];
      const bool ok = node_req[row] >= 0;
      const int dep = min(max(depth[row], 0), n_depth - 1);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int col = n0 + wn * TN * 16 + j * 16 + (lane & 15);
        if (col >= d_m) continue;
        float val = st.y * (acc[i][j][v] - st.x * c1[col]) + c2[dep * d_m + col];
        if (!ok) val = __builtin_nanf("");
        const int64_t o = static_cast<int64_t>(row) * d_m + col;
        if constexpr (std::is_same<T, bf16_t>::value) {
          const bf16_t hi = f32_to_bf16_bits(val);
          const float r1 = val - bf16_bits_to_f32(hi);
          const bf16_t mid = f32_to_bf16_bits(r1);
          const bf16_t lo = f32_to_bf16_bits(r1 - bf16_bits_to_f32(mid));
          q[o] = hi;
          q[plane + o] = mid;
          q[2 * plane + o] = lo;
        } else {
          q[o] = val;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------
// Scores s = q . k / sqrt(d_m) for every (node, key) of a request.  One block per
// (request, 64-key tile); wave w owns keys [16 w, 16 w + 16) of the tile and loops over
// the request's nodes in chunks of 64.  Keys stream straight from HBM into registers
// (each lane reads 16 consecutive k of one key row: 32 B for bf16), the query chunk is
// staged once per block in LDS.  The k order inside a 64-wide step is permuted the
// same way for both operands: lane group g = lane / 16 feeds k = 16 g + 0..15.
// ---------------------------------------------------------------------------------

template <typename T>
__global__ __launch_bounds__(256) void score_kernel(int B, const int64_t* __restrict__ mem_off,
                                                    int64_t n_mem, int m_max,
                                                    const int32_t* __restrict__ node_off,
                                                    int n_nodes, int t_max,
                                                    const T* __restrict__ keys, int d_m,
                                                    const T* __restrict__ q, float scale,
                                                    float* __restrict__ S) {
  constexpr bool kBf16 = std::is_same<T, bf16_t>::value;
  constexpr int NS = kBf16 ? kQSplitBf16 : 1;  // q planes
  constexpr int VEC = Elem<T>::kPer16B;
  constexpr int LDQ = 64 + VEC;
  constexpr int CH_ROW = 64 / VEC;           // 16-byte chunks per 64-wide q row
  constexpr int CH_TOTAL = NS * 64 * CH_ROW;
  static_assert(CH_TOTAL % 256 == 0, "q staging does not split over the block");
  __shared__ __align__(16) T qs[NS][64][LDQ];

  const int b = blockIdx.x % B;
  const int tile = blockIdx.x / B;
  const Extent e = request_extent(b, mem_off, n_mem, m_max, node_off, n_nodes, t_max);
  if (!e.nodes_ok || !e.mem_ok) return;  // the select kernel reports and fills NaN
  const int M = static_cast<int>(e.m1 - e.m0);
  const int Tn = e.t1 - e.t0;
  const int i0 = tile * 64;
  if (i0 >= M || Tn == 0) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int key = i0 + wave * 16 + (lane & 15);
  const T* krow = keys + (e.m0 + min(key, M - 1)) * d_m + 16 * g;
  const int64_t plane = static_cast<int64_t>(n_nodes) * d_m;

  for (int c0 = 0; c0 < Tn; c0 += 64) {
    const int nblk = min(4, (Tn - c0 + 15) / 16);
    f32x4 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d_m; k0 += 64) {
      // key fragment: 16 consecutive k of this lane's key row
      u32x4 kr[16 / VEC];
#pragma unroll
      for (int u = 0; u < 16 / VEC; ++u)
        kr[u] = *reinterpret_cast<const u32x4*>(krow + k0 + u * VEC);
      // stage q[c0 .. c0+63][k0 .. k0+63] for every plane
#pragma unroll
      for (int j = 0; j < CH_TOTAL / 256; ++j) {
        const int c = tid + 256 * j;
        const int p = c / (64 * CH_ROW);
        const int rr = (c / CH_ROW) % 64;
        const int cc = c % CH_ROW;
        const int src = e.t0 + min(c0 + rr, Tn - 1);
        *reinterpret_cast<u32x4*>(&qs[p][rr][cc * VEC]) = *reinterpret_cast<const u32x4*>(
            q + p * plane + static_cast<int64_t>(src) * d_m + k0 + cc * VEC);
      }
      __syncthreads();
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        if (nb >= nblk) break;
        const T* qrow = &qs[0][nb * 16 + (lane & 15)][16 * g];
        if constexpr (kBf16) {
          const bf16x8 kb0 = *reinterpret_cast<const bf16x8*>(&kr[0]);
          const bf16x8 kb1 = *reinterpret_cast<const bf16x8*>(&kr[1]);
#pragma unroll
          for (int p = 0; p < NS; ++p) {
            const T* qp = qrow + p * 64 * LDQ;
            acc[nb] = mfma_bf16_16x16x32(*reinterpret_cast<const bf16x8*>(qp), kb0, acc[nb]);
            acc[nb] = mfma_bf16_16x16x32(*reinterpret_cast<const bf16x8*>(qp + 8), kb1, acc[nb]);
          }
        } else {
          const float* kf = reinterpret_cast<const float*>(kr);
#pragma unroll
          for (int s = 0; s < 16; ++s) acc[nb] = mfma_f32_16x16x4(qrow[s], kf[s], acc[nb]);
        }
      }
      __syncthreads();
    }
    if (key < M) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        if (nb >= nblk) break;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = c0 + nb * 16 + 4 * g + v;
          if (r < Tn) S[static_cast<int64_t>(e.t0 + r) * m_max + key] = acc[nb][v] * scale;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------
// Per-node selection and gather, one 256-thread block per node:
//   max and Z over the valid scores; exact top-k_max by (score desc, index asc) with an
//   MSB-first radix select on the order-preserving score key (plus, for ties, on the
//   inverted index); bitonic sort of the candidates; prefix masses in fp64; K from the
//   cumulative-mass rule; renormalised weights; weighted gather of value rows.
// ---------------------------------------------------------------------------------

template <typename T>
struct SelectArgs {
  const int64_t* mem_off;
  int64_t n_mem;
  int m_max;
  const int32_t* node_req;
  const float* tau;
  const uint8_t* valid;
  const T* values;
  int d_m;
  const float* S;
  int k_min, k_max;
  T* rT;
  float* r_out;
  int32_t* k_out;
  int32_t* idx_out;
  float* mass_out;
  uint32_t* err;
};

template <int NT>
__device__ __forceinline__ int block_sum_int(int v, int* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) s += red[w];
  return s;
}

template <int NT>
__device__ __forceinline__ double block_sum_f64(double v, double* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) s += red[w];
  return s;
}

template <int NT>
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, uint32_t* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = max(v, static_cast<uint32_t>(__shfl_xor(static_cast<int>(v), o, kWave)));
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  uint32_t m = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) m = max(m, red[w]);
  return m;
}

// Radix step: among elements whose key matches `prefix` on `pmask`, histogram the
// 8-bit digit at `shift` and find the digit holding the krem-th largest element.
// Returns the digit; *above = elements in higher digits, *in_bin = elements in it.
struct RadixPick {
  int digit, above, in_bin;
};

__device__ __forceinline__ RadixPick radix_pick(int* hist, int krem, RadixPick* out) {
  // called by wave 0 after the histogram is complete; lane l owns bins 255-4l .. 252-4l
  const int lane = threadIdx.x & 63;
  int cnt[4], tot = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    cnt[j] = hist[255 - 4 * lane - j];
    tot += cnt[j];
  }
  int incl = tot;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  int run = incl - tot;  // elements in bins above this lane's bins
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (run < krem && run + cnt[j] >= krem) {
      out->digit = 255 - 4 * lane - j;
      out->above = run;
      out->in_bin = cnt[j];
    }
    run += cnt[j];
  }
  return *out;
}

template <typename T>
__global__ __launch_bounds__(256) void select_gather_kernel(SelectArgs<T> a) {
  constexpr int NT = 256;
  extern __shared__ uint32_t skey[];  // [m_max] order keys; 0 marks a masked entry
  __shared__ int hist[256];
  __shared__ unsigned long long cand[kMaxKmax];
  __shared__ double pre[kMaxKmax];
  __shared__ float alpha[kMaxKmax];
  __shared__ int sidx[kMaxKmax];
  __shared__ int ired[NT / 64];
  __shared__ double dred[NT / 64];
  __shared__ uint32_t ured[NT / 64];
  __shared__ RadixPick pick;
  __shared__ int s_count, s_first;

  const int n = blockIdx.x;
  const int tid = threadIdx.x;
  const int b = a.node_req[n];
  int64_t m0 = 0, m1 = 0;
  bool ok = b >= 0;
  if (ok) {
    m0 = a.mem_off[b];
    m1 = a.mem_off[b + 1];
    if (!(0 <= m0 && m0 <= m1 && m1 <= a.n_mem && m1 - m0 <= a.m_max)) {
      ok = false;
      if (tid == 0) atomicOr(a.err, kErrMemOff);
    }
  }
  const int64_t rbase = static_cast<int64_t>(n) * a.d_m;
  if (!ok) {
    const float qnan = __builtin_nanf("");
    for (int c = tid; c < a.d_m; c += NT) {
      st_f32(a.rT, rbase + c, qnan);
      if (a.r_out) a.r_out[rbase + c] = qnan;
    }
    if (a.idx_out)
      for (int t = tid; t < a.k_max; t += NT) a.idx_out[static_cast<int64_t>(n) * a.k_max + t] = -1;
    if (tid == 0) {
      if (a.k_out) a.k_out[n] = 0;
      if (a.mass_out) a.mass_out[n] = qnan;
    }
    return;
  }
  const int M = static_cast<int>(m1 - m0);
  const float* srow = a.S + static_cast<int64_t>(n) * a.m_max;

  // keys, valid count, max
  int cnt = 0;
  uint32_t kmax = 0;
  for (int i = tid; i < M; i += NT) {
    const bool v = a.valid == nullptr || a.valid[m0 + i] != 0;
    const uint32_t k = v ? order_key(srow[i]) : 0u;
    skey[i] = k;
    cnt += v ? 1 : 0;
    kmax = max(kmax, k);
  }
  const int nV = block_sum_int<NT>(cnt, ired);
  kmax = block_max_u32<NT>(kmax, ured);

  int K = 0;
  double mass = 0.0;
  if (nV > 0) {
    const float smax = key_to_float(kmax);
    double z = 0.0;
    for (int i = tid; i < M; i += NT) {
      const uint32_t k = skey[i];
      if (k != 0u) z += static_cast<double>(expf(key_to_float(k) - smax));
    }
    const double Z = block_sum_f64<NT>(z, dred);

    // ---- candidates: the top min(nV, k_max) entries ----
    const int C = min(nV, a.k_max);
    uint32_t thr = 0u, thr_inv = 0u;
    bool all_eq = true;
    if (nV > a.k_max) {
      uint32_t prefix = 0u, pmask = 0u;
      int krem = a.k_max;
      int in_bin = 0;
      for (int shift = 24; shift >= 0; shift -= 8) {
        hist[tid] = 0;
        __syncthreads();
        for (int i = tid; i < M; i += NT) {
          const uint32_t k = skey[i];
          if (k != 0u && (k & pmask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid < 64) radix_pick(hist, krem, &pick);
        __syncthreads();
        prefix |= static_cast<uint32_t>(pick.digit) << shift;
        pmask |= 255u << shift;
        krem -= pick.above;
        in_bin = pick.in_bin;
        __syncthreads();
      }
      thr = prefix;
      if (in_bin > krem) {
        // ties at the threshold score: keep the krem lowest indices (largest 0xFFFF - i)
        all_eq = false;
        uint32_t iprefix = 0u, imask = 0u;
        for (int shift = 8; shift >= 0; shift -= 8) {
          hist[tid] = 0;
          __syncthreads();
          for (int i = tid; i < M; i += NT) {
            const uint32_t inv = 0xFFFFu - static_cast<uint32_t>(i);
            if (skey[i] == thr && (inv & imask) == iprefix) atomicAdd(&hist[(inv >> shift) & 255u], 1);
          }
          __syncthreads();
          if (tid < 64) radix_pick(hist, krem, &pick);
          __syncthreads();
          iprefix |= static_cast<uint32_t>(pick.digit) << shift;
          imask |= 255u << shift;
          krem -= pick.above;
          __syncthreads();
        }
        thr_inv = iprefix;
      }
    }
    if (tid == 0) s_count = 0;
    __syncthreads();
    for (int i = tid; i < M; i += NT) {
      const uint32_t k = skey[i];
      if (k == 0u) continue;
      const bool take = nV <= a.k_max || k > thr ||
                        (k == thr && (all_eq || 0xFFFFu - static_cast<uint32_t>(i) >= thr_inv));
      if (take) {
        const int pos = atomicAdd(&s_count, 1);
        if (pos < kMaxKmax)
          cand[pos] = (static_cast<unsigned long long>(k) << 32) |
                      static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(i));
      }
    }
    __syncthreads();
    // s_count equals C by construction; never let a short count expose stale slots
    const int C_ok = min(C, s_count);
    int P = 1;
    while (P < C) P <<= 1;
    for (int i = C_ok + tid; i < C; i += NT) cand[i] = 0ull;
    for (int i = C + tid; i < P; i += NT) cand[i] = 0ull;
    __syncthreads();
    // bitonic sort, descending
    for (int kk = 2; kk <= P; kk <<= 1) {
      for (int j = kk >> 1; j > 0; j >>= 1) {
        for (int i = tid; i < P; i += NT) {
          const int ixj = i ^ j;
          if (ixj > i) {
            const unsigned long long x = cand[i], y = cand[ixj];
            const bool desc = (i & kk) == 0;
            if (desc ? (x < y) : (x > y)) {
              cand[i] = y;
              cand[ixj] = x;
            }
          }
        }
        __syncthreads();
      }
    }
    // prefix sums of exp(s - max) in rank order, four consecutive ranks per thread
    double e4[4];
    double loc = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = 4 * tid + j;
      e4[j] = t < C ? static_cast<double>(expf(key_to_float(static_cast<uint32_t>(cand[t] >> 32)) - smax))
                    : 0.0;
      loc += e4[j];
      e4[j] = loc;
    }
    // exclusive scan of the thread totals
    {
      const int lane = tid & 63, wave = tid >> 6;
      double incl = loc;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      __syncthreads();
      if (lane == 63) dred[wave] = incl;
      __syncthreads();
      double off = incl - loc;
      for (int w = 0; w < wave; ++w) off += dred[w];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = 4 * tid + j;
        if (t < kMaxKmax) pre[t] = off + e4[j];
      }
    }
    if (tid == 0) s_first = INT_MAX;
    __syncthreads();
    const double tau = static_cast<double>(a.tau[b]);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = 4 * tid + j;
      if (t < C && pre[t] / Z >= tau) atomicMin(&s_first, t);
    }
    __syncthreads();
    const int K_raw = s_first != INT_MAX ? s_first + 1 : (C == nV ? nV : a.k_max + 1);
    K = min(nV, min(a.k_max, max(a.k_min, K_raw)));
    mass = pre[K - 1] / Z;
    const double sumI = pre[K - 1];
    for (int t = tid; t < K; t += NT) {
      const float et = expf(key_to_float(static_cast<uint32_t>(cand[t] >> 32)) - smax);
      alpha[t] = static_cast<float>(static_cast<double>(et) / sumI);
      const uint32_t ix = 0xFFFFFFFFu - static_cast<uint32_t>(cand[t]);
      sidx[t] = static_cast<int>(min(ix, static_cast<uint32_t>(M - 1)));
    }
    __syncthreads();
  }

  // ---- renormalised gather r = sum_t alpha_t u_{idx_t} (fp32, rank order) ----
  constexpr int CV = 4;  // columns per thread per pass
  for (int c = tid * CV; c < a.d_m; c += NT * CV) {
    float acc[CV] = {0.f, 0.f, 0.f, 0.f};
    for (int t = 0; t < K; ++t) {
      const float w = alpha[t];
      const T* u = a.values + (m0 + sidx[t]) * a.d_m + c;
#pragma unroll
      for (int j = 0; j < CV; ++j) acc[j] = fmaf(w, Elem<T>::to_f32(u[j]), acc[j]);
    }
#pragma unroll
    for (int j = 0; j < CV; ++j) {
      st_f32(a.rT, rbase + c + j, acc[j]);
      if (a.r_out) a.r_out[rbase + c + j] = acc[j];
    }
  }
  if (a.idx_out)
    for (int t = tid; t < a.k_max; t += NT)
      a.idx_out[static_cast<int64_t>(n) * a.k_max + t] = t < K ? sidx[t] : -1;
  if (tid == 0) {
    if (a.k_out) a.k_out[n] = K;
    if (a.mass_out) a.mass_out[n] = static_cast<float>(mass);
  }
}

}  // namespace fovea
