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
constexpr int kQSplitBf16 = 2;  // q = hi + lo in bf16 for the score MFMA

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

// Rows of up to 64 * kRowChunks 16-byte chunks are held in registers (one load round
// trip, both LayerNorm passes from registers); longer rows stream in passes.
constexpr int kRowChunks = 16;

// Per-node view of its request, written by the statistics kernel so that the selection
// reads it with one load: the request's memory range and tau.  M < 0 marks a node whose
// offsets, depth, tau or memory range failed validation (the error bits are set).
struct NodeInfo {
  int64_t m0;
  int32_t M;
  float tau;
};

template <typename T>
__global__ __launch_bounds__(256) void row_stats_kernel(int n, const T* __restrict__ x, int d,
                                                        float eps, float2* __restrict__ stats,
                                                        const int32_t* __restrict__ depth,
                                                        int n_depth,
                                                        const int32_t* __restrict__ node_off,
                                                        int B, int t_max,
                                                        const float* __restrict__ tau,
                                                        const int64_t* __restrict__ mem_off,
                                                        int64_t n_mem, int m_max,
                                                        int32_t* __restrict__ node_req,
                                                        NodeInfo* __restrict__ info,
                                                        uint32_t* err) {
  constexpr int VEC = Elem<T>::kPer16B;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= n) return;
  const T* xr = x + static_cast<int64_t>(row) * d;
  const int nch = d / VEC;
  // request lookup operands, loaded together with the row
  int off_v = 0, dep_v = 0;
  float tau_v = 0.f;
  int64_t mem_v = 0;
  if (node_off != nullptr && B < 64) {
    off_v = node_off[min(lane, B)];
    tau_v = tau[min(lane, B - 1)];
    mem_v = mem_off[min(lane, B)];
    dep_v = depth[row];
  }
  float mu, var;
  if (nch <= 64 * kRowChunks) {
    u32x4 raw[kRowChunks];
#pragma unroll
    for (int u = 0; u < kRowChunks; ++u) {
      const int c = lane + 64 * u;
      if (c < nch) raw[u] = *reinterpret_cast<const u32x4*>(xr + c * VEC);
    }
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < kRowChunks; ++u)
      if (lane + 64 * u < nch) {
        const T* v = reinterpret_cast<const T*>(&raw[u]);
#pragma unroll
        for (int j = 0; j < VEC; ++j) s += Elem<T>::to_f32(v[j]);
      }
    mu = wave_sum_f32(s) / static_cast<float>(d);
    float ss = 0.f;
#pragma unroll
    for (int u = 0; u < kRowChunks; ++u)
      if (lane + 64 * u < nch) {
        const T* v = reinterpret_cast<const T*>(&raw[u]);
#pragma unroll
        for (int j = 0; j < VEC; ++j) {
          const float t = Elem<T>::to_f32(v[j]) - mu;
          ss = fmaf(t, t, ss);
        }
      }
    var = wave_sum_f32(ss) / static_cast<float>(d);
  } else {
    float s = 0.f;
    for (int c = lane; c < nch; c += kWave) {
      const u32x4 raw = *reinterpret_cast<const u32x4*>(xr + c * VEC);
      const T* v = reinterpret_cast<const T*>(&raw);
#pragma unroll
      for (int j = 0; j < VEC; ++j) s += Elem<T>::to_f32(v[j]);
    }
    mu = wave_sum_f32(s) / static_cast<float>(d);
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
    var = wave_sum_f32(ss) / static_cast<float>(d);
  }
  if (lane == 0) stats[row] = make_float2(mu, 1.0f / sqrtf(var + eps));

  if (node_off != nullptr) {
    // largest b with node_off[b] <= row (a fixed number of steps even if the offsets
    // are bad); for B < 64 the offsets, tau and depth were loaded with the row, and the
    // search reads them across lanes
    int b, t0, t1, dep;
    float tb;
    int64_t m0, m1;
    if (B < 64) {
      int lo = 0, hi = B - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (__builtin_amdgcn_readlane(off_v, mid) <= row) lo = mid; else hi = mid - 1;
      }
      b = lo;
      t0 = __builtin_amdgcn_readlane(off_v, b);
      t1 = __builtin_amdgcn_readlane(off_v, b + 1);
      tb = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(tau_v), b));
      const uint64_t mu = static_cast<uint64_t>(mem_v);
      m0 = static_cast<int64_t>((static_cast<uint64_t>(__builtin_amdgcn_readlane(static_cast<uint32_t>(mu >> 32), b)) << 32) |
                                __builtin_amdgcn_readlane(static_cast<uint32_t>(mu), b));
      m1 = static_cast<int64_t>((static_cast<uint64_t>(__builtin_amdgcn_readlane(static_cast<uint32_t>(mu >> 32), b + 1)) << 32) |
                                __builtin_amdgcn_readlane(static_cast<uint32_t>(mu), b + 1));
      dep = dep_v;
    } else {
      int lo = 0, hi = B - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (node_off[mid] <= row) lo = mid; else hi = mid - 1;
      }
      b = lo;
      t0 = node_off[b];
      t1 = node_off[b + 1];
      tb = tau[b];
      m0 = mem_off[b];
      m1 = mem_off[b + 1];
      dep = depth[row];
    }
    if (lane == 0) {
      uint32_t bad = 0;
      if (!(0 <= t0 && t0 <= row && row < t1 && t1 <= n && t1 - t0 <= t_max)) bad |= kErrNodeOff;
      if (dep < 0 || dep >= n_depth) bad |= kErrDepth;
      if (!(tb >= 0.f && tb <= 1.f)) bad |= kErrTau;
      node_req[row] = bad ? -1 : b;
      // the memory range is checked only for nodes that map to a request
      const bool mem_ok = 0 <= m0 && m0 <= m1 && m1 <= n_mem && m1 - m0 <= m_max;
      if (!bad && !mem_ok) bad |= kErrMemOff;
      NodeInfo ni;
      ni.m0 = mem_ok ? m0 : 0;
      ni.M = bad ? -1 : static_cast<int32_t>(m1 - m0);
      ni.tau = tb;
      info[row] = ni;
      if (bad) atomicOr(err, bad);
    }
  }
}

// Request of node `row` and its validation, by one thread (the same checks as the
// statistics kernel): node_req[row] = b, or -1 for a node whose offsets, depth or tau are
// bad; info[row] as in NodeInfo; the error bits are set.  Returns node_req[row] >= 0.
struct NodeMapArgs {
  const int32_t* node_off;
  int B, t_max, n;
  const int32_t* depth;
  int n_depth;
  const float* tau;
  const int64_t* mem_off;
  int64_t n_mem;
  int m_max;
  int32_t* node_req;
  NodeInfo* info;
  uint32_t* err;
};

__device__ __forceinline__ bool map_node(const NodeMapArgs& m, int row, bool write) {
  int lo = 0, hi = m.B - 1;  // largest b with node_off[b] <= row (fixed step count)
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (m.node_off[mid] <= row) lo = mid; else hi = mid - 1;
  }
  const int b = lo;
  const int t0 = m.node_off[b], t1 = m.node_off[b + 1], dep = m.depth[row];
  const float tb = m.tau[b];
  const int64_t m0 = m.mem_off[b], m1 = m.mem_off[b + 1];
  uint32_t bad = 0;
  if (!(0 <= t0 && t0 <= row && row < t1 && t1 <= m.n && t1 - t0 <= m.t_max)) bad |= kErrNodeOff;
  if (dep < 0 || dep >= m.n_depth) bad |= kErrDepth;
  if (!(tb >= 0.f && tb <= 1.f)) bad |= kErrTau;
  const bool ok = bad == 0;
  if (write) {
    m.node_req[row] = ok ? b : -1;
    const bool mem_ok = 0 <= m0 && m0 <= m1 && m1 <= m.n_mem && m1 - m0 <= m.m_max;
    if (ok && !mem_ok) bad |= kErrMemOff;
    NodeInfo ni;
    ni.m0 = mem_ok ? m0 : 0;
    ni.M = bad ? -1 : static_cast<int32_t>(m1 - m0);
    ni.tau = tb;
    m.info[row] = ni;
    if (bad) atomicOr(m.err, bad);
  }
  return ok;
}

// LayerNorm statistics of the split-K query GEMM: the block of column tile tc over K slice
// y (columns k0 .. k0 + Kc) writes, for the rows m0 + tc, m0 + tc + cb, .. of its row tile,
// the slice's mean and sum of squared deviations from it (two passes over the slice,
// which the GEMM has just brought into L2) to part[y][row]; the combine merges the slices.
// The blocks of slice 0 also map and validate those rows (map_node).
template <typename T>
__device__ __forceinline__ void slice_row_stats(const T* __restrict__ h, int d, int n, int m0, int rows,
                                                int tc, int cb, int k0, int Kc, int y,
                                                float2* __restrict__ part, const NodeMapArgs& nm) {
  // 8 consecutive elements per lane and step (Kc is a multiple of 64)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rend = min(m0 + rows, n);
  for (int r = m0 + tc + cb * wave; r < rend; r += cb * 4) {
    const T* hr = h + static_cast<int64_t>(r) * d + k0;
    float s = 0.f;
    for (int c = 8 * lane; c < Kc; c += 8 * 64) {
      float x[8];
      load8(hr + c, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) s += x[e];
    }
    const float mean = wave_sum_f32(s) / static_cast<float>(Kc);
    float ss = 0.f;
    for (int c = 8 * lane; c < Kc; c += 8 * 64) {
      float x[8];
      load8(hr + c, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float t = x[e] - mean;
        ss = fmaf(t, t, ss);
      }
    }
    const float m2 = wave_sum_f32(ss);
    if (lane == 0) {
      part[static_cast<int64_t>(y) * n + r] = make_float2(mean, m2);
      if (y == 0) map_node(nm, r, true);  // the slice-0 blocks map and validate the rows
    }
  }
}

// ---------------------------------------------------------------------------------
// Query projection with the LayerNorm folded into the epilogue:
//   q = W_Q (LN(h) + E_dep[l]) = rstd * (W' h - mu * W' 1) + W_Q (b + E_dep[l]),
// W' = W_Q diag(gain) packed at context creation, c1 = W' 1, c2[l] = W_Q (b + E_dep[l]).
// bf16 storage writes q as two bf16 planes, hi = bf16(q) and lo = bf16(q - hi), for the
// score MFMA (|q - hi - lo| <= 2^-16 |q|); fp32 storage writes q itself.
// ---------------------------------------------------------------------------------

template <typename T, int BM = 128>
using HqCfg = GemmCfg<T, BM, 4>;

// One GEMM over the hidden states for everything that depends on h alone:
// columns [0, d_m) are the query projection (LayerNorm folded as described above),
// columns [d_m, d_m + n_p) are h W1h^T, the h half of the correction and gate nets'
// first layer, kept in fp32 for the layer-1 kernel (P, [n, n_p]).
template <typename T>
struct HqEpi {
  int n, d_m, N, n_depth;
  int64_t n_p;
  const float2* stats;     // (mean, rstd) of row - srow0
  const int32_t* depth;
  const int32_t* node_req;
  const int* ok_s = nullptr;  // if set: row - srow0 valid (else node_req[row] >= 0)
  int srow0 = 0;
  const float* c1;
  const float* c2;
  T* q;
  float* P;
  __device__ __forceinline__ float operator()(int row, int col0, const float (&v)[8]) const {
    if (row >= n || col0 >= N) return 0.f;
    if (col0 >= d_m) {
      store8(P + static_cast<int64_t>(row) * n_p + (col0 - d_m), v);
      return 0.f;
    }
    const int64_t plane = static_cast<int64_t>(n) * d_m;
    const float2 st = stats[row - srow0];
    const bool ok = ok_s != nullptr ? ok_s[row - srow0] != 0 : node_req[row] >= 0;
    const int dep = min(max(depth[row], 0), n_depth - 1);
    float a[8], b[8], val[8];
    load8(c1 + col0, a);
    load8(c2 + static_cast<int64_t>(dep) * d_m + col0, b);
#pragma unroll
    for (int e = 0; e < 8; ++e) val[e] = ok ? st.y * (v[e] - st.x * a[e]) + b[e] : __builtin_nanf("");
    const int64_t o = static_cast<int64_t>(row) * d_m + col0;
    if constexpr (std::is_same<T, bf16_t>::value) {
      float hi[8], lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        hi[e] = bf16_round(val[e]);
        lo[e] = val[e] - hi[e];
      }
      store8(q + o, hi);
      store8(q + plane + o, lo);
    } else {
      store8(q + o, val);
    }
    return 0.f;
  }
};

// ks > 1: split-K (grid.y = ks slices, fp32 partials in part), finished by
// hq_combine_kernel with the same epilogue.
// With ks > 1 and stat_part set, the LayerNorm statistics come from the slices
// (slice_row_stats, after each block's partial product) and the combine merges them;
// no separate statistics launch.
template <typename T, int BM = 128>
__global__ __launch_bounds__(256) void hq_kernel(TileMap tm, int n, const T* __restrict__ h, int d,
                                                 const T* __restrict__ Whq, HqEpi<T> epi, int ks,
                                                 float* __restrict__ part,
                                                 float2* __restrict__ stat_part = nullptr,
                                                 NodeMapArgs nm = NodeMapArgs{}) {
  using C = HqCfg<T, BM>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  if (ks > 1) {
    gemm_splitk_partial<C>(h, d, n, Whq, d, epi.N, d, ks, m0, n0, part, smem);
    if (stat_part != nullptr) {
      const int Kc = d / ks;
      slice_row_stats(h, d, n, m0, C::BM, tc, tm.cb, static_cast<int>(blockIdx.y) * Kc, Kc,
                      static_cast<int>(blockIdx.y), stat_part, nm);
    }
    return;
  }
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, h, d, n, Whq, d, epi.N, d, m0, n0, smem);
  gemm_epilogue<C>(acc, smem, m0, n0, epi, NoRowSum{});
}

// stat_part set: the block's 16 rows get their LayerNorm statistics by merging the ks
// slices' (mean, M2) in slice order (Chan's pairwise update, equal slice widths) and their
// validity from node_req (written by the slice-0 partial blocks).  Every thread first
// adds its 8 columns' partials (as
// splitk_combine does), so that those loads and the statistics' loads are in flight
// together; then the barrier; then the epilogue.
constexpr int kHqMaxKs = 32;  // the query GEMM's k slices are at most d / 128 <= 32 here

template <typename T>
__global__ __launch_bounds__(256) void hq_combine_kernel(HqEpi<T> epi, int ks,
                                                         const float* __restrict__ part,
                                                         const float2* __restrict__ stat_part,
                                                         int d, float eps) {
  if (stat_part == nullptr) {
    splitk_combine(epi.n, epi.N, ks, part, epi, NoRowSum{});
    return;
  }
  __shared__ float2 s_st[16];
  __shared__ int s_ok[16];
  const int r0 = static_cast<int>(blockIdx.y) * 16;
  const int row = r0 + static_cast<int>(threadIdx.x >> 4);
  const int col0 = static_cast<int>(blockIdx.x) * 128 + static_cast<int>(threadIdx.x & 15) * 8;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (row < epi.n && col0 < epi.N) {
    for (int y0 = 0; y0 < ks; y0 += 8) {
      float t[8][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (y0 + u < ks) load8(part + (static_cast<int64_t>(y0 + u) * epi.n + row) * epi.N + col0, t[u]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (y0 + u < ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += t[u][e];
    }
  }
  if (threadIdx.x < 16) {
    const int srow = r0 + static_cast<int>(threadIdx.x);
    float2 st = make_float2(0.f, 1.f);
    int ok = 0;
    if (srow < epi.n) {
      float2 p[kHqMaxKs];
#pragma unroll
      for (int y = 0; y < kHqMaxKs; ++y)
        if (y < ks) p[y] = stat_part[static_cast<int64_t>(y) * epi.n + srow];
      ok = epi.node_req[srow] >= 0 ? 1 : 0;
      const float w = static_cast<float>(d / ks);
      float mean = 0.f, m2 = 0.f, cnt = 0.f;
#pragma unroll
      for (int y = 0; y < kHqMaxKs; ++y)
        if (y < ks) {
          const float c2 = cnt + w;
          const float delta = p[y].x - mean;
          mean += delta * (w / c2);
          m2 += p[y].y + delta * delta * (cnt * w / c2);
          cnt = c2;
        }
      st = make_float2(mean, 1.0f / sqrtf(m2 / static_cast<float>(d) + eps));
    }
    s_st[threadIdx.x] = st;
    s_ok[threadIdx.x] = ok;
  }
  __syncthreads();
  epi.stats = s_st;
  epi.ok_s = s_ok;
  epi.srow0 = r0;
  epi(row, col0, v);  // rows and columns past the matrix are dropped by the functor
}

// ---------------------------------------------------------------------------------
// Work-item mapping that keeps the blocks of one request on one XCD: blocks are
// dispatched round-robin over the 8 XCDs (block i on XCD i % 8), so item
// x * per_xcd + j is given to block 8 j + x.  Returns -1 for padding blocks.
// ---------------------------------------------------------------------------------

constexpr int kXcds = 8;

__device__ __forceinline__ int xcd_item(int total) {
  const int per_xcd = (total + kXcds - 1) / kXcds;
  const int item = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
  return item < total ? item : -1;
}

inline int xcd_grid(int total) { return kXcds * ((total + kXcds - 1) / kXcds); }

// ---------------------------------------------------------------------------------
// Scores s = q . k / sqrt(d_m), bf16 storage.  One block per (request, tile of 16 KB
// keys, chunk of 64 nodes), four waves; wave w owns node block w (16 nodes) of the
// chunk and all keys of the tile (KB 16x16 MFMA accumulators).  The k dimension is walked in
// 64-wide chunks:
//   * keys: the block stages each chunk ([16 KB keys][64 k]) into one of two LDS slots;
//     every thread keeps the next DK chunks in flight in registers, so HBM latency
//     hides behind DK chunks of matrix work;
//   * q: each wave reads its own 16 rows of the two bf16 planes (hi, lo) straight from
//     L2 into A-fragment registers, also DK chunks ahead;
//   * k order inside a chunk is permuted identically for both operands: lane group
//     g = lane / 16 feeds k = 16 g + 0..7 to the first MFMA and 16 g + 8..15 to the
//     second;
//   * the KB accumulator chains are interleaved so consecutive MFMAs are independent.
// The chunk count NKC is a template parameter: every loop unrolls and every load is
// unconditional (rows past the request are clamped and dropped at the store), which
// keeps the wait counters exact so the prefetch queue is never drained.
// ---------------------------------------------------------------------------------

namespace score_cfg {
constexpr int KC = 64;    // k per chunk
constexpr int LDK = KC + 8;
constexpr int DK = 6;     // key prefetch depth (chunks)
constexpr int NS = kQSplitBf16;
template <int KB>
struct Tile {
  static constexpr int KT = 16 * KB;                    // keys per block
  static constexpr int KCH = (KT * 8 + 255) / 256;      // 16-byte staging loads per thread
  static constexpr int ROWS = KCH * 32;                 // LDS rows (padding rows unused)
};
}  // namespace score_cfg

template <int NKC, int KB>
__global__ __launch_bounds__(256, (KB >= 5 || NKC >= 20) ? 1 : 2) void score_bf16_kernel(
    int B, const int64_t* __restrict__ mem_off, int64_t n_mem, int m_max,
    const int32_t* __restrict__ node_off, int n_nodes, int t_max, const bf16_t* __restrict__ keys,
    int d_m, const bf16_t* __restrict__ q, float scale, float* __restrict__ S, int parts,
    int spread) {
  using namespace score_cfg;
  using TL = Tile<KB>;
  __shared__ __align__(16) bf16_t ks[2][TL::ROWS][LDK];
  const int tiles = (m_max + TL::KT - 1) / TL::KT;
  const int nch = (t_max + 63) / 64;  // 64-node chunks; a block takes one
  // parts > 1: the block contracts k slice `part` (NKC chunks) of d_m = parts NKC KC and
  // writes partial scores to S + part n_nodes m_max (the selection adds them in order)
  // spread = 0: a request's blocks share an XCD (and its q in L2); spread = 1: items go
  // round-robin over the XCDs, which balances requests of very different sizes
  const int total = B * tiles * nch * parts;
  const int item0 = spread ? (static_cast<int>(blockIdx.x) < total ? static_cast<int>(blockIdx.x) : -1)
                           : xcd_item(total);
  if (item0 < 0) return;
  const int part = item0 % parts, item = item0 / parts;
  const int b = item / (tiles * nch);
  const int tile = (item / nch) % tiles;
  const int cn = (item % nch) * 64;
  const int kofs0 = part * NKC * KC;
  const Extent e = request_extent(b, mem_off, n_mem, m_max, node_off, n_nodes, t_max);
  if (!e.nodes_ok || !e.mem_ok) return;  // the select kernel reports and fills NaN
  const int M = static_cast<int>(e.m1 - e.m0);
  const int Tn = e.t1 - e.t0;
  const int i0 = tile * TL::KT;
  if (i0 >= M || cn >= Tn) return;

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4;
  const int64_t plane = static_cast<int64_t>(n_nodes) * d_m;
  const bf16_t* kg[TL::KCH];
  u32x4* kd0[TL::KCH];
  u32x4* kd1[TL::KCH];
#pragma unroll
  for (int u = 0; u < TL::KCH; ++u) {
    const int qi = tid + 256 * u;               // 16-byte chunk of the [rows][64] tile
    const int row = qi >> 3, kofs = (qi & 7) * 8;
    kg[u] = keys + (e.m0 + min(i0 + row, M - 1)) * d_m + kofs0 + kofs;
    kd0[u] = reinterpret_cast<u32x4*>(&ks[0][row][kofs]);
    kd1[u] = reinterpret_cast<u32x4*>(&ks[1][row][kofs]);
  }
  const bf16_t* kb0 = &ks[0][lane & 15][16 * g];
  const bf16_t* kb1 = &ks[1][lane & 15][16 * g];

  {
    const int qrow = e.t0 + min(cn + 16 * w + (lane & 15), Tn - 1);
    const bf16_t* qg = q + static_cast<int64_t>(qrow) * d_m + kofs0 + 16 * g;
    u32x4 kr[DK][TL::KCH];
    u32x4 qr[DK][NS][2];
    f32x4 acc[KB];
#pragma unroll
    for (int i = 0; i < KB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Loads retire in issue order (one counter for all vector memory), so they are
    // issued in the order they are consumed: key chunk j + 1 is staged just before q
    // chunk j is used, hence the issue order K0, K1, Q0, K2, Q1, ...  Scheduling
    // barriers keep the compiler from hoisting later key loads above earlier q loads.
#pragma unroll
    for (int u = 0; u < TL::KCH; ++u) kr[0][u] = *reinterpret_cast<const u32x4*>(kg[u]);
#pragma unroll
    for (int c = 1; c <= DK; ++c) {
      if (c < DK && c < NKC)
#pragma unroll
        for (int u = 0; u < TL::KCH; ++u) kr[c][u] = *reinterpret_cast<const u32x4*>(kg[u] + c * KC);
      if (c == DK) {
        // chunk 0 leaves its register slot for chunk DK
#pragma unroll
        for (int u = 0; u < TL::KCH; ++u) *kd0[u] = kr[0][u];
        if (DK < NKC)
#pragma unroll
          for (int u = 0; u < TL::KCH; ++u) kr[0][u] = *reinterpret_cast<const u32x4*>(kg[u] + DK * KC);
      }
      if (c - 1 < NKC)
#pragma unroll
        for (int p = 0; p < NS; ++p) {
          qr[c - 1][p][0] = *reinterpret_cast<const u32x4*>(qg + p * plane + (c - 1) * KC);
          qr[c - 1][p][1] = *reinterpret_cast<const u32x4*>(qg + p * plane + (c - 1) * KC + 8);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < NKC; ++c) {
      if (c + 1 < NKC) {
#pragma unroll
        for (int u = 0; u < TL::KCH; ++u) *(((c + 1) & 1) ? kd1[u] : kd0[u]) = kr[(c + 1) % DK][u];
        if (c + 1 + DK < NKC)
#pragma unroll
          for (int u = 0; u < TL::KCH; ++u)
            kr[(c + 1) % DK][u] = *reinterpret_cast<const u32x4*>(kg[u] + (c + 1 + DK) * KC);
      }
      __builtin_amdgcn_sched_barrier(0);
      const bf16_t* kb = (c & 1) ? kb1 : kb0;
      bf16x8 bfr[KB][2];
#pragma unroll
      for (int kblk = 0; kblk < KB; ++kblk) {
        bfr[kblk][0] = *reinterpret_cast<const bf16x8*>(kb + kblk * 16 * LDK);
        bfr[kblk][1] = *reinterpret_cast<const bf16x8*>(kb + kblk * 16 * LDK + 8);
      }
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int p = 0; p < NS; ++p)
#pragma unroll
          for (int kblk = 0; kblk < KB; ++kblk)
            acc[kblk] = mfma_bf16_16x16x32(*reinterpret_cast<const bf16x8*>(&qr[c % DK][p][h]),
                                           bfr[kblk][h], acc[kblk]);
      __builtin_amdgcn_sched_barrier(0);
      if (c + DK < NKC)
#pragma unroll
        for (int p = 0; p < NS; ++p) {
          qr[c % DK][p][0] = *reinterpret_cast<const u32x4*>(qg + p * plane + (c + DK) * KC);
          qr[c % DK][p][1] = *reinterpret_cast<const u32x4*>(qg + p * plane + (c + DK) * KC + 8);
        }
      __syncthreads();
    }
    if (cn + 16 * w < Tn) {
      float* Sp = S + static_cast<int64_t>(part) * n_nodes * m_max;
#pragma unroll
      for (int kblk = 0; kblk < KB; ++kblk) {
        const int key = i0 + kblk * 16 + (lane & 15);
        if (key >= M) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = cn + 16 * w + 4 * g + v;
          if (r < Tn) Sp[static_cast<int64_t>(e.t0 + r) * m_max + key] = acc[kblk][v] * scale;
        }
      }
    }
  }
}

// Fallback for chunk counts without a fixed instantiation: same tiling (64 keys per
// block), no register prefetch; each 64-k chunk is loaded, staged and consumed in turn.
__global__ __launch_bounds__(256) void score_bf16_any_kernel(
    int B, const int64_t* __restrict__ mem_off, int64_t n_mem, int m_max,
    const int32_t* __restrict__ node_off, int n_nodes, int t_max, const bf16_t* __restrict__ keys,
    int d_m, const bf16_t* __restrict__ q, float scale, float* __restrict__ S, int /*parts: 1*/,
    int /*spread*/) {
  using namespace score_cfg;
  constexpr int KT = 64;
  __shared__ __align__(16) bf16_t ks[KT][LDK];
  const int tiles = (m_max + KT - 1) / KT;
  const int item = xcd_item(B * tiles);
  if (item < 0) return;
  const int b = item / tiles;
  const int tile = item % tiles;
  const Extent e = request_extent(b, mem_off, n_mem, m_max, node_off, n_nodes, t_max);
  if (!e.nodes_ok || !e.mem_ok) return;
  const int M = static_cast<int>(e.m1 - e.m0);
  const int Tn = e.t1 - e.t0;
  const int i0 = tile * KT;
  if (i0 >= M || Tn == 0) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4;
  const int64_t plane = static_cast<int64_t>(n_nodes) * d_m;
  const int srow = tid >> 2, sk = (tid & 3) * 16;
  const bf16_t* kg = keys + (e.m0 + min(i0 + srow, M - 1)) * d_m + sk;
  for (int cn = 0; cn < Tn; cn += 64) {
    const int qrow = e.t0 + min(cn + 16 * w + (lane & 15), Tn - 1);
    const bf16_t* qg = q + static_cast<int64_t>(qrow) * d_m + 16 * g;
    f32x4 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d_m; k0 += KC) {
      reinterpret_cast<u32x4*>(&ks[srow][sk])[0] = *reinterpret_cast<const u32x4*>(kg + k0);
      reinterpret_cast<u32x4*>(&ks[srow][sk])[1] = *reinterpret_cast<const u32x4*>(kg + k0 + 8);
      u32x4 qa[NS][2];
#pragma unroll
      for (int p = 0; p < NS; ++p) {
        qa[p][0] = *reinterpret_cast<const u32x4*>(qg + p * plane + k0);
        qa[p][1] = *reinterpret_cast<const u32x4*>(qg + p * plane + k0 + 8);
      }
      __syncthreads();
      const bf16_t* kb = &ks[lane & 15][16 * g];
#pragma unroll
      for (int kblk = 0; kblk < 4; ++kblk)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int p = 0; p < NS; ++p)
            acc[kblk] = mfma_bf16_16x16x32(*reinterpret_cast<const bf16x8*>(&qa[p][h]),
                                           *reinterpret_cast<const bf16x8*>(kb + kblk * 16 * LDK + 8 * h),
                                           acc[kblk]);
      __syncthreads();
    }
    if (cn + 16 * w < Tn) {
#pragma unroll
      for (int kblk = 0; kblk < 4; ++kblk) {
        const int key = i0 + kblk * 16 + (lane & 15);
        if (key >= M) continue;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int r = cn + 16 * w + 4 * g + v;
          if (r < Tn) S[static_cast<int64_t>(e.t0 + r) * m_max + key] = acc[kblk][v] * scale;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------
// Scores for fp32 storage (a simple version: one block per (request, 64-key tile),
// wave w owns keys [16 w, 16 w + 16), fp32 MFMA, q staged per 64-k chunk in LDS).
// ---------------------------------------------------------------------------------

__global__ __launch_bounds__(256) void score_f32_kernel(int B, const int64_t* __restrict__ mem_off,
                                                        int64_t n_mem, int m_max,
                                                        const int32_t* __restrict__ node_off,
                                                        int n_nodes, int t_max,
                                                        const float* __restrict__ keys, int d_m,
                                                        const float* __restrict__ q, float scale,
                                                        float* __restrict__ S) {
  constexpr int LDQ = 64 + 4;
  __shared__ __align__(16) float qs[64][LDQ];
  const int tiles = (m_max + 63) / 64;
  const int item = xcd_item(B * tiles);
  if (item < 0) return;
  const int b = item / tiles;
  const int tile = item % tiles;
  const Extent e = request_extent(b, mem_off, n_mem, m_max, node_off, n_nodes, t_max);
  if (!e.nodes_ok || !e.mem_ok) return;
  const int M = static_cast<int>(e.m1 - e.m0);
  const int Tn = e.t1 - e.t0;
  const int i0 = tile * 64;
  if (i0 >= M || Tn == 0) return;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4;
  const int key = i0 + wave * 16 + (lane & 15);
  const float* krow = keys + (e.m0 + min(key, M - 1)) * d_m + 16 * g;

  for (int c0 = 0; c0 < Tn; c0 += 64) {
    const int nblk = min(4, (Tn - c0 + 15) / 16);
    f32x4 acc[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d_m; k0 += 64) {
      float kf[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) kf[u] = krow[k0 + u];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int c = tid + 256 * j;  // 64 rows x 16 chunks of 4 floats
        const int rr = c >> 4, cc = (c & 15) * 4;
        const int src = e.t0 + min(c0 + rr, Tn - 1);
        *reinterpret_cast<u32x4*>(&qs[rr][cc]) =
            *reinterpret_cast<const u32x4*>(q + static_cast<int64_t>(src) * d_m + k0 + cc);
      }
      __syncthreads();
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        if (nb >= nblk) break;
        const float* qrow = &qs[nb * 16 + (lane & 15)][16 * g];
#pragma unroll
        for (int s2 = 0; s2 < 16; ++s2) acc[nb] = mfma_f32_16x16x4(qrow[s2], kf[s2], acc[nb]);
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
//   inverted index); candidates ranked by counting; prefix masses in fp64; K from the
//   cumulative-mass rule; renormalised weights; weighted gather of value rows.
// ---------------------------------------------------------------------------------

constexpr int kScoreMaxParts = 4;  // k slices of the score GEMM (partial score arrays)

template <typename T>
struct SelectArgs {
  const int64_t* mem_off;
  int64_t n_mem;
  int m_max;
  const int32_t* node_req;
  const NodeInfo* info;
  const float* tau;
  const uint8_t* valid;
  const T* values;
  int d_m;
  const float* S;
  int s_parts;        // partial score arrays to add (in order), s_stride floats apart
  int64_t s_stride;
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

// keys read per load round in the block-wide selection's scans over its LDS keys, for
// memories of more than kSelScanB * 256 entries (shorter ones scan one key at a time)
constexpr int kSelScanB = 8;

// Dynamic LDS of select_gather_kernel: the order keys (or the gather's partial sums,
// 3 x 64 lanes x VEC floats, whichever is larger; 8-byte aligned end), then the candidate
// keys (8 B), prefix masses (8 B), weights (4 B) and indices (4 B) of kcap slots.
__host__ __device__ inline int select_kcap(int k_max) { return (k_max + 3) & ~3; }
__host__ __device__ inline int select_key_bytes(int m_max, int vec) {
  const int b = m_max * 4 > 3 * 64 * vec * 4 ? m_max * 4 : 3 * 64 * vec * 4;
  return (b + 7) & ~7;
}
__host__ __device__ inline int select_gather_smem(int m_max, int k_max, int vec) {
  return select_key_bytes(m_max, vec) + select_kcap(k_max) * 24;
}

// exp(s - smax) of an order key as 2^((s - smax) log2 e) on the hardware exp2 (relative
// error a few 1e-7, far inside the score rounding band); the normaliser, the prefix masses
// and the weights all take it from here, so the prefixes never exceed the normaliser by a
// differing rounding.
__device__ __forceinline__ float key_mass(uint32_t k, float smax) {
  return __builtin_amdgcn_exp2f((key_to_float(k) - smax) * 1.4426950408889634f);
}

// Sorts the C distinct keys of list descending in place: the rank of a key is the number
// of keys above it, counted in one broadcast pass over the list (thread tid ranks the
// keys at tid + NT q, q < Q).
template <int Q, int NT>
__device__ __forceinline__ void rank_sort_desc(unsigned long long* list, int C, int tid) {
  unsigned long long mine[Q];
  int rk[Q];
#pragma unroll
  for (int q = 0; q < Q; ++q) {
    const int t = tid + NT * q;
    mine[q] = t < C ? list[t] : 0ull;
    rk[q] = 0;
  }
  for (int j = 0; j < C; ++j) {
    const unsigned long long y = list[j];
#pragma unroll
    for (int q = 0; q < Q; ++q) rk[q] += y > mine[q] ? 1 : 0;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < Q; ++q)
    if (tid + NT * q < C) list[rk[q]] = mine[q];
  __syncthreads();
}

template <typename T>
__global__ __launch_bounds__(256) void select_gather_kernel(SelectArgs<T> a) {
  constexpr int NT = 256;
  // dynamic LDS (select_gather_smem): the order keys [m_max] (0 marks a masked entry;
  // later the gather's partial sums), then the candidate arrays sized for k_max, so that
  // two blocks share a compute unit even at 16384 keys
  extern __shared__ __align__(16) unsigned char sel_smem[];
  uint32_t* skey = reinterpret_cast<uint32_t*>(sel_smem);
  const int kcap = select_kcap(a.k_max);
  unsigned long long* cand =
      reinterpret_cast<unsigned long long*>(sel_smem + select_key_bytes(a.m_max, Elem<T>::kPer16B));
  double* pre = reinterpret_cast<double*>(cand + kcap);
  float* alpha = reinterpret_cast<float*>(pre + kcap);
  int* sidx = reinterpret_cast<int*>(alpha + kcap);
  __shared__ int hist[256];
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
  // U entries per thread and step, every load issued before the first use (16 for long
  // memories, whose rows take many steps; 4 otherwise)
  auto load_keys = [&](auto U_) {
    constexpr int U = decltype(U_)::value;
    for (int i0 = tid; i0 < M; i0 += U * NT) {
      float sc[U], ps[U][kScoreMaxParts - 1];
      bool v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * NT;
        const bool in = i < M;
        sc[u] = in ? srow[i] : 0.f;
#pragma unroll
        for (int p = 1; p < kScoreMaxParts; ++p)
          ps[u][p - 1] = in && p < a.s_parts ? srow[p * a.s_stride + i] : 0.f;
        v[u] = in && (a.valid == nullptr || a.valid[m0 + i] != 0);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * NT;
        if (i < M) {
#pragma unroll
          for (int p = 1; p < kScoreMaxParts; ++p)
            if (p < a.s_parts) sc[u] += ps[u][p - 1];
          const uint32_t k = v[u] ? order_key(sc[u]) : 0u;
          skey[i] = k;
          cnt += v[u] ? 1 : 0;
          kmax = max(kmax, k);
        }
      }
    }
  };
  if (M > 16 * NT)
    load_keys(std::integral_constant<int, 16>());
  else
    load_keys(std::integral_constant<int, 4>());
  const int nV = block_sum_int<NT>(cnt, ired);
  kmax = block_max_u32<NT>(kmax, ured);

  int K = 0;
  double mass = 0.0;
  if (nV > 0) {
    const float smax = key_to_float(kmax);
    double z = 0.0;
    for (int i = tid; i < M; i += NT) {
      const uint32_t k = skey[i];
      if (k != 0u) z += static_cast<double>(key_mass(k, smax));
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
        // a thread's keys mostly share a digit: one atomic per run of equal digits; the
        // keys are read SB at a time (all reads issued before the first use)
        int cur = -1, run = 0;
        auto hist_scan = [&](auto SB_) {
          constexpr int SB = decltype(SB_)::value;
          for (int i0 = tid; i0 < M; i0 += SB * NT) {
            uint32_t kk[SB];
#pragma unroll
            for (int u = 0; u < SB; ++u) kk[u] = i0 + u * NT < M ? skey[i0 + u * NT] : 0u;
#pragma unroll
            for (int u = 0; u < SB; ++u) {
              const uint32_t k = kk[u];
              if (k != 0u && (k & pmask) == prefix) {
                const int dg = static_cast<int>((k >> shift) & 255u);
                if (dg != cur) {
                  if (run > 0) atomicAdd(&hist[cur], run);
                  cur = dg;
                  run = 0;
                }
                ++run;
              }
            }
          }
        };
        if (M > kSelScanB * NT)
          hist_scan(std::integral_constant<int, kSelScanB>());
        else
          hist_scan(std::integral_constant<int, 1>());
        if (run > 0) atomicAdd(&hist[cur], run);
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
    // the candidates appended in any order (the ranking below orders them); long memories:
    // per wave one atomic per step for all its lanes' picks, keys read SB at a time
    auto compact = [&](auto SB_) {
      constexpr int SB = decltype(SB_)::value;
      for (int i0 = tid - (tid & 63); i0 < M; i0 += SB * NT) {
        uint32_t kk[SB];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
          const int i = i0 + (tid & 63) + u * NT;
          kk[u] = i < M ? skey[i] : 0u;
        }
#pragma unroll
        for (int u = 0; u < SB; ++u) {
          const int i = i0 + (tid & 63) + u * NT;
          const uint32_t k = kk[u];
          const bool take = k != 0u && (nV <= a.k_max || k > thr ||
                                        (k == thr && (all_eq || 0xFFFFu - static_cast<uint32_t>(i) >= thr_inv)));
          const unsigned long long bal = __ballot(take);
          if (bal == 0ull) continue;  // wave-uniform
          int base = 0;
          if ((tid & 63) == __ffsll(static_cast<long long>(bal)) - 1) base = atomicAdd(&s_count, __popcll(bal));
          base = __shfl(base, __ffsll(static_cast<long long>(bal)) - 1, kWave);
          if (take) {
            const int pos = base + __popcll(bal & ((1ull << (tid & 63)) - 1ull));
            if (pos < kcap)
              cand[pos] = (static_cast<unsigned long long>(k) << 32) |
                          static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(i));
          }
        }
      }
    };
    if (M > kSelScanB * NT) {
      compact(std::integral_constant<int, kSelScanB>());
    } else {
      for (int i = tid; i < M; i += NT) {
        const uint32_t k = skey[i];
        if (k == 0u) continue;
        const bool take = nV <= a.k_max || k > thr ||
                          (k == thr && (all_eq || 0xFFFFu - static_cast<uint32_t>(i) >= thr_inv));
        if (take) {
          const int pos = atomicAdd(&s_count, 1);
          if (pos < kcap)
            cand[pos] = (static_cast<unsigned long long>(k) << 32) |
                        static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(i));
        }
      }
    }
    __syncthreads();
    // s_count equals C by construction; never let a short count expose stale slots
    const int C_ok = min(C, s_count);
    // (distinct values below every real key, which has a nonzero high word)
    for (int i = C_ok + tid; i < C; i += NT) cand[i] = static_cast<unsigned long long>(C - i);
    __syncthreads();
    // descending order by counting (the keys are distinct: each holds its entry index)
    if (C <= NT)
      rank_sort_desc<1, NT>(cand, C, tid);
    else
      rank_sort_desc<kMaxKmax / NT, NT>(cand, C, tid);
    // prefix sums of exp(s - max) in rank order, four consecutive ranks per thread
    double e4[4];
    double loc = 0.0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int t = 4 * tid + j;
      e4[j] = t < C ? static_cast<double>(key_mass(static_cast<uint32_t>(cand[t] >> 32), smax))
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
        if (t < kcap) pre[t] = off + e4[j];
      }
    }
    if (tid == 0) s_first = INT_MAX;
    __syncthreads();
    // the first rank whose prefix reaches tau Z: the prefixes only grow with the rank, so
    // a wave's first qualifying rank sits in its lowest qualifying lane (one atomic per wave)
    const double tau = static_cast<double>(a.tau[b]);
    {
      int first = INT_MAX;
#pragma unroll
      for (int j = 3; j >= 0; --j) {
        const int t = 4 * tid + j;
        if (t < C && pre[t] / Z >= tau) first = t;
      }
      const unsigned long long hit = __ballot(first != INT_MAX);
      if (hit != 0ull && (tid & 63) == __ffsll(static_cast<long long>(hit)) - 1) atomicMin(&s_first, first);
    }
    __syncthreads();
    const int K_raw = s_first != INT_MAX ? s_first + 1 : (C == nV ? nV : a.k_max + 1);
    K = min(nV, min(a.k_max, max(a.k_min, K_raw)));
    mass = pre[K - 1] / Z;
    const double sumI = pre[K - 1];
    for (int t = tid; t < K; t += NT) {
      const float et = key_mass(static_cast<uint32_t>(cand[t] >> 32), smax);
      alpha[t] = static_cast<float>(static_cast<double>(et) / sumI);
      const uint32_t ix = 0xFFFFFFFFu - static_cast<uint32_t>(cand[t]);
      sidx[t] = static_cast<int>(min(ix, static_cast<uint32_t>(M - 1)));
    }
    __syncthreads();
  }

  // ---- renormalised gather r = sum_t alpha_t u_{idx_t} ----
  // This block covers the 16-byte chunks [c_lo, c_hi) of the row (its column slice);
  // lane l takes chunk c_lo + l + 64 j in pass j, wave w the ranks w, w + 4, .. in
  // batches of GR rows whose loads all issue before the first multiply-add; the four
  // partial sums are added by wave 0 in a fixed order through LDS.
  {
    constexpr int VEC = Elem<T>::kPer16B;
    constexpr int GR = 8;
    const int cpr = a.d_m / VEC;
    const int ns = gridDim.y;
    const int c_lo = static_cast<int>(static_cast<int64_t>(cpr) * blockIdx.y / ns);
    const int c_hi = static_cast<int>(static_cast<int64_t>(cpr) * (blockIdx.y + 1) / ns);
    const int lane = tid & 63, w = tid >> 6;
    const int mine = K > w ? (K - w + 3) / 4 : 0;
    float* red = reinterpret_cast<float*>(skey);  // the keys are no longer needed
    for (int cb = c_lo; cb < c_hi; cb += 64) {
      const int c = min(cb + lane, c_hi - 1);
      float acc[VEC];
#pragma unroll
      for (int x = 0; x < VEC; ++x) acc[x] = 0.f;
      // batches of 2 GR rows while that many remain, then of up to GR
      auto batch = [&](auto G_, int q0, int nr) {
        constexpr int G = decltype(G_)::value;
        u32x4 raw[G];
#pragma unroll
        for (int r = 0; r < G; ++r) {
          const int t = w + 4 * (q0 + min(r, nr - 1));
          raw[r] = *reinterpret_cast<const u32x4*>(a.values + (m0 + sidx[t]) * a.d_m + c * VEC);
        }
#pragma unroll
        for (int r = 0; r < G; ++r) {
          if (r < nr) {
            const float wt = alpha[w + 4 * (q0 + r)];
            const T* v = reinterpret_cast<const T*>(&raw[r]);
#pragma unroll
            for (int x = 0; x < VEC; ++x) acc[x] = fmaf(wt, Elem<T>::to_f32(v[x]), acc[x]);
          }
        }
      };
      for (int q0 = 0; q0 < mine;) {
        if (mine - q0 >= 2 * GR) {
          batch(std::integral_constant<int, 2 * GR>(), q0, 2 * GR);
          q0 += 2 * GR;
        } else {
          const int nr = min(GR, mine - q0);
          batch(std::integral_constant<int, GR>(), q0, nr);
          q0 += nr;
        }
      }
      if (w > 0)
#pragma unroll
        for (int x = 0; x < VEC; ++x) red[((w - 1) * 64 + lane) * VEC + x] = acc[x];
      __syncthreads();
      if (w == 0 && cb + lane < c_hi) {
#pragma unroll
        for (int q = 0; q < 3; ++q)
#pragma unroll
          for (int x = 0; x < VEC; ++x) acc[x] += red[(q * 64 + lane) * VEC + x];
        const int64_t o = rbase + static_cast<int64_t>(c) * VEC;
#pragma unroll
        for (int x = 0; x < VEC; ++x) {
          st_f32(a.rT, o + x, acc[x]);
          if (a.r_out) a.r_out[o + x] = acc[x];
        }
      }
      __syncthreads();
    }
  }
  if (blockIdx.y != 0) return;  // one block of the node writes the selection outputs
  if (a.idx_out)
    for (int t = tid; t < a.k_max; t += NT)
      a.idx_out[static_cast<int64_t>(n) * a.k_max + t] = t < K ? sidx[t] : -1;
  if (tid == 0) {
    if (a.k_out) a.k_out[n] = K;
    if (a.mass_out) a.mass_out[n] = static_cast<float>(mass);
  }
}


// ---------------------------------------------------------------------------------
// Per-node selection by one wave, for memories of at most 64 * NPL entries and
// k_max <= 256.  Each lane holds NPL order keys (entry lane + 64 j).  The k_max-th
// largest key is found bit by bit (at most 32 steps of ballot counts); ties at it are
// cut by a second bit search over the entry index so the lowest indices win.
// Candidates are compacted with ballot prefix counts, sorted descending by
// (key, -index) in registers (<= 64) or in LDS (<= 256), then prefix masses in fp64,
// K and the renormalised weights.
// ---------------------------------------------------------------------------------

constexpr int kWaveSelKmax = 256;

template <typename T>
__device__ __forceinline__ void write_invalid_node(const SelectArgs<T>& a, int n, int tid, int nt) {
  const float qnan = __builtin_nanf("");
  const int64_t rbase = static_cast<int64_t>(n) * a.d_m;
  for (int c = tid; c < a.d_m; c += nt) {
    st_f32(a.rT, rbase + c, qnan);
    if (a.r_out) a.r_out[rbase + c] = qnan;
  }
  if (a.idx_out)
    for (int t = tid; t < a.k_max; t += nt) a.idx_out[static_cast<int64_t>(n) * a.k_max + t] = -1;
  if (tid == 0) {
    if (a.k_out) a.k_out[n] = 0;
    if (a.mass_out) a.mass_out[n] = qnan;
  }
}

__device__ __forceinline__ int ballot_count(bool p) { return __popcll(__ballot(p)); }

// Number of lanes and slots j with key slot j >= t.  The NPL ballots are taken first
// (each in its own scalar register pair) and counted afterwards, so that the compares
// issue back to back instead of each waiting for the previous count to read the one
// condition register.
template <int NPL>
__device__ __forceinline__ int count_ge(const uint32_t (&kv)[NPL], uint32_t t) {
  unsigned long long b[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) b[j] = __builtin_amdgcn_ballot_w64(kv[j] >= t);
  int c = 0;
#pragma unroll
  for (int j = 0; j < NPL; ++j) c += __popcll(b[j]);
  return c;
}

__device__ __forceinline__ unsigned long long comp_key(uint32_t k, int i) {
  return (static_cast<unsigned long long>(k) << 32) |
         static_cast<unsigned long long>(0xFFFFFFFFu - static_cast<uint32_t>(i));
}

// Orders the LDS accesses of one wave (a wave's LDS operations execute in issue order;
// this keeps the compiler from moving them across the point).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The keys of one node: its request's memory range and tau (validated by the statistics
// kernel) and the order keys of its scores (entry lane + 64 j in kv[j], 0 for masked or
// missing entries, the valid ones flagged in bit j of vmask).  The score row and the
// node record are independent loads, so both are in flight together.
struct NodeKeys {
  int M;
  int64_t m0;
  float tau;
  bool ok;
  uint64_t vmask;
};

template <typename T, int NPL>
__device__ __forceinline__ NodeKeys load_node_keys(const SelectArgs<T>& a, int n, int lane,
                                                   uint32_t (&kv)[NPL]) {
  const float* srow = a.S + static_cast<int64_t>(n) * a.m_max;
  float sv[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) sv[j] = a.m_max > 0 ? srow[min(lane + 64 * j, a.m_max - 1)] : 0.f;
  // partial scores of the other k slices: every load issued before the first add
  float pv[kScoreMaxParts - 1][NPL];
#pragma unroll
  for (int p = 1; p < kScoreMaxParts; ++p)
#pragma unroll
    for (int j = 0; j < NPL; ++j)
      pv[p - 1][j] = p < a.s_parts && a.m_max > 0 ? srow[p * a.s_stride + min(lane + 64 * j, a.m_max - 1)] : 0.f;
#pragma unroll
  for (int p = 1; p < kScoreMaxParts; ++p)
#pragma unroll
    for (int j = 0; j < NPL; ++j)
      if (p < a.s_parts) sv[j] += pv[p - 1][j];
  const NodeInfo inf = a.info[n];
  NodeKeys r;
  r.ok = inf.M >= 0;
  r.M = r.ok ? inf.M : 0;
  r.m0 = inf.m0;
  r.tau = inf.tau;
  r.vmask = 0;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int i = lane + 64 * j;
    const bool v = i < r.M && (a.valid == nullptr || a.valid[r.m0 + i] != 0);
    kv[j] = v ? order_key(sv[j]) : 0u;
    r.vmask |= static_cast<uint64_t>(v) << j;
  }
  return r;
}

// Selection for one node by one wave: writes the selected indices and renormalised
// weights (rank order) to idx_o / alpha_o and returns K (-1 if the node is invalid, in
// which case its outputs have been written as NaN).
//  * the top min(nV, k_max) keys are found bit by bit (the k_max-th largest key), each
//    count read from one ballot per key slot;
//  * the candidates are compacted, ranked by counting (keys are made distinct by the
//    index), their masses placed in rank order and summed by a wave prefix scan in fp64;
//  * K_raw is the first rank whose prefix reaches tau Z, clamped to [k_min, k_max].
template <typename T, int NPL>
__device__ __forceinline__ int select_one_node(const SelectArgs<T>& a, int n, int lane,
                                               const NodeKeys& nk, const uint32_t (&kv)[NPL],
                                               unsigned long long* cand, double* pre_s,
                                               float* alpha_o, int* idx_o, float* mass_o) {
  if (!nk.ok) {
    write_invalid_node(a, n, lane, 64);
    return -1;
  }
  const int M = nk.M;
  uint32_t lmax = 0;
#pragma unroll
  for (int j = 0; j < NPL; ++j) lmax = max(lmax, kv[j]);
  int nV = M;  // without a mask every entry of the request is valid
  if (a.valid != nullptr) {
    nV = 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) nV += ballot_count((nk.vmask >> j) & 1);
  }
  const uint32_t kmax = __builtin_amdgcn_readfirstlane(wave_max_u32(lmax));
  int K = 0;
  double mass = 0.0;
  if (nV > 0) {
    // exp(s - smax) as 2^((s - smax) log2 e) on the hardware exp2 (relative error a few
    // 1e-7 for the entries that carry mass, far inside the score rounding band)
    const float smax = key_to_float(kmax);
    constexpr float kLog2e = 1.4426950408889634f;
    float ev[NPL];
    double z = 0.0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      ev[j] = kv[j] != 0u ? __builtin_amdgcn_exp2f((key_to_float(kv[j]) - smax) * kLog2e) : 0.f;
      z += static_cast<double>(ev[j]);
    }
    const double Z = wave_sum_f64(z);
    const int C = min(nV, a.k_max);
    uint32_t thr = 0u;
    int ithr = 0x7FFFFFFF;
    if (nV > a.k_max) {
      // the k_max-th largest key, bit by bit, under the invariant count(key >= thr) >=
      // k_max (masked entries hold 0; every tested threshold is >= 1, so they never
      // count).  With k_max <= 64 the search starts below the bits that the largest key
      // shares with the smallest lane maximum: each lane holds a key >= that minimum, so
      // at least 64 keys reach the shared prefix.  Once the count equals k_max the set
      // {key >= thr} is the top k_max and the lower bits are not needed.
      int bit = 31;
      if (a.k_max <= 64) {
        const uint32_t t0 = __builtin_amdgcn_readfirstlane(~wave_max_u32(~lmax));
        const uint32_t diff = t0 ^ kmax;
        bit = diff != 0u ? 31 - __builtin_clz(diff) : -1;
        thr = diff != 0u ? (kmax & ~((2u << bit) - 1u)) : kmax;
      }
      for (; bit >= 0; --bit) {
        const uint32_t t = thr | (1u << bit);
        const int cnt = count_ge<NPL>(kv, t);
        if (cnt >= a.k_max) thr = t;
        if (cnt == a.k_max) break;
      }
      if (bit < 0) {  // no exact count on the way down
        // thr is the k_max-th largest key itself and more than k_max keys reach it:
        // keep the tied entries with the lowest indices.  I is the largest index bound
        // with #(tied, index < I) < need, so the tied entries with index <= I stay.
        int gt = 0;
#pragma unroll
        for (int j = 0; j < NPL; ++j) gt += ballot_count(kv[j] > thr);
        const int need = a.k_max - gt;
        int I = 0;
        for (int b2 = 14; b2 >= 0; --b2) {
          const int t = I + (1 << b2);
          int f = 0;
#pragma unroll
          for (int j = 0; j < NPL; ++j) f += ballot_count(kv[j] == thr && lane + 64 * j < t);
          if (f < need) I = t;
        }
        ithr = I;
      }
    }
    // compact the C candidates (lane-major order; the ranking below orders them).  With
    // an exact threshold (ithr unset) the candidates are the keys >= thr.
    int nsel = 0;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int i = lane + 64 * j;
      nsel += (kv[j] != 0u && (nV <= a.k_max || kv[j] > thr || (kv[j] == thr && i <= ithr))) ? 1 : 0;
    }
    const int incl_sel = wave_incl_scan_i32(nsel);
    const int base = __builtin_amdgcn_readlane(incl_sel, 63);
    int pos = incl_sel - nsel;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int i = lane + 64 * j;
      const bool sel = kv[j] != 0u && (nV <= a.k_max || kv[j] > thr || (kv[j] == thr && i <= ithr));
      if (sel && pos < kWaveSelKmax) {
        cand[pos] = comp_key(kv[j], i);
        alpha_o[pos] = ev[j];  // scratch until the weights are written
      }
      pos += sel ? 1 : 0;
    }
    const int Cc = min(C, base);
    wave_lds_sync();
    const double tauZ = static_cast<double>(nk.tau) * Z;
    if (C <= 64) {
      // rank of lane t's candidate = number of larger candidates (keys are distinct); the
      // masses are placed in rank order and summed by an fp64 wave prefix scan, and the
      // first rank reaching tau Z is read from a ballot
      const unsigned long long x = lane < Cc ? cand[lane] : 0ull;
      const float ex = lane < Cc ? alpha_o[lane] : 0.f;
      int rk = 0;
      for (int u = 0; u < Cc; ++u) rk += cand[u] > x ? 1 : 0;
      double sumI;
      if (a.k_min == a.k_max) {
        // fixed cardinality: K = min(|V|, k_max) = C, every candidate is selected, and
        // only the total of their masses is needed (no prefix, no tau search)
        K = Cc;
        sumI = wave_sum_f64(lane < Cc ? static_cast<double>(ex) : 0.0);
      } else {
        wave_lds_sync();
        if (lane < Cc) pre_s[rk] = static_cast<double>(ex);
        wave_lds_sync();
        const double incl = wave_incl_scan_f64(lane < Cc ? pre_s[lane] : 0.0);
        const unsigned long long hit = __ballot(lane < Cc && incl >= tauZ);
        const int K_raw = hit ? __builtin_ctzll(hit) + 1 : (C == nV ? nV : a.k_max + 1);
        K = min(nV, min(a.k_max, max(a.k_min, K_raw)));
        const uint64_t iu = static_cast<uint64_t>(__double_as_longlong(incl));
        const uint32_t ilo = __builtin_amdgcn_readlane(static_cast<uint32_t>(iu), K - 1);
        const uint32_t ihi = __builtin_amdgcn_readlane(static_cast<uint32_t>(iu >> 32), K - 1);
        sumI = __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(ihi) << 32) | ilo));
      }
      mass = sumI / Z;
      const double rs = 1.0 / sumI;
      wave_lds_sync();
      if (lane < Cc && rk < K) {
        alpha_o[rk] = static_cast<float>(static_cast<double>(ex) * rs);
        idx_o[rk] = static_cast<int>(min(0xFFFFFFFFu - static_cast<uint32_t>(x), static_cast<uint32_t>(M - 1)));
      }
      *mass_o = static_cast<float>(mass);
      return K;
    }
    {
      // larger candidate sets: bitonic sort in LDS, then the prefix (masses from the same
      // hardware exp2 as Z, so that the prefix never exceeds Z by a differing rounding)
      int P = 128;
      while (P < C) P <<= 1;
      for (int i = Cc + lane; i < P; i += 64) cand[i] = 0ull;
      wave_lds_sync();
      for (int k2 = 2; k2 <= P; k2 <<= 1) {
        for (int j2 = k2 >> 1; j2 > 0; j2 >>= 1) {
          for (int i = lane; i < P; i += 64) {
            const int ixj = i ^ j2;
            if (ixj > i) {
              const unsigned long long x = cand[i], y = cand[ixj];
              const bool desc = (i & k2) == 0;
              if (desc ? (x < y) : (x > y)) {
                cand[i] = y;
                cand[ixj] = x;
              }
            }
          }
          wave_lds_sync();
        }
      }
      double e4[4], loc = 0.0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = 4 * lane + u;
        e4[u] = t < C ? static_cast<double>(__builtin_amdgcn_exp2f((key_to_float(static_cast<uint32_t>(cand[t] >> 32)) - smax) * kLog2e)) : 0.0;
        loc += e4[u];
        e4[u] = loc;
      }
      double incl = loc;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      const double off = incl - loc;
#pragma unroll
      for (int u = 0; u < 4; ++u) pre_s[4 * lane + u] = off + e4[u];
    }
    wave_lds_sync();
    // first rank whose prefix mass reaches tau
    int first = 0x7FFFFFFF;
    for (int t = lane; t < C; t += 64)
      if (pre_s[t] >= tauZ) first = min(first, t);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) first = min(first, __shfl_xor(first, o, kWave));
    const int K_raw = first != 0x7FFFFFFF ? first + 1 : (C == nV ? nV : a.k_max + 1);
    K = min(nV, min(a.k_max, max(a.k_min, K_raw)));
    const double sumI = pre_s[K - 1];
    mass = sumI / Z;
    for (int t = lane; t < K; t += 64) {
      const unsigned long long x = cand[t];
      const float et = __builtin_amdgcn_exp2f((key_to_float(static_cast<uint32_t>(x >> 32)) - smax) * kLog2e);
      alpha_o[t] = static_cast<float>(static_cast<double>(et) / sumI);
      idx_o[t] = static_cast<int>(min(0xFFFFFFFFu - static_cast<uint32_t>(x), static_cast<uint32_t>(M - 1)));
    }
  }
  *mass_o = static_cast<float>(mass);
  return K;
}

// ---------------------------------------------------------------------------------
// Selection and gather, two nodes per 256-thread block (memories of at most 64 * NPL
// entries, k_max <= 256, value rows of at most 64 * NCH 16-byte chunks).  Two waves
// select (above), one node each; then each node's K selected rows are split between
// two waves (ranks of one parity each), lane l owning chunks l, l + 64, .. of every
// row, and a batch of up to NR rows is one set of unconditional loads (slots past the
// wave's rows repeat its last row and are not accumulated), so K <= 2 NR costs one
// memory round trip.  The two partial sums are added in a fixed order through LDS.
// ---------------------------------------------------------------------------------

template <typename T, int NCH, int NR>
__device__ __forceinline__ void gather_rows(const T* __restrict__ vbase, int d_m, int cpr,
                                            const int* ix, const float* al, int t0, int stride,
                                            int nr, int lane, float (&acc)[NCH][Elem<T>::kPer16B]) {
  constexpr int VEC = Elem<T>::kPer16B;
  u32x4 raw[NR][NCH];
  int row[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) row[r] = ix[t0 + min(r, nr - 1) * stride];
#pragma unroll
  for (int r = 0; r < NR; ++r)
#pragma unroll
    for (int u = 0; u < NCH; ++u) {
      const int c = min(lane + 64 * u, cpr - 1);
      raw[r][u] = *reinterpret_cast<const u32x4*>(vbase + static_cast<int64_t>(row[r]) * d_m + c * VEC);
    }
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    if (r < nr) {  // wave-uniform: padding slots are skipped whole
      const float w = al[t0 + r * stride];
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const T* v = reinterpret_cast<const T*>(&raw[r][u]);
#pragma unroll
        for (int x = 0; x < VEC; ++x) acc[u][x] = fmaf(w, Elem<T>::to_f32(v[x]), acc[u][x]);
      }
    }
  }
}

// NPB nodes per block (2, or 1 for batches with fewer node pairs than compute units):
// each node's first wave selects; the gather of its K rows is split over the node's
// 4 / NPB waves (ranks w, w + 4 / NPB, ...) and summed in wave order.
template <typename T, int NPL, int NCH, int NPB = 2>
__global__ __launch_bounds__(256) void select_node_kernel(SelectArgs<T> a, int n_nodes) {
  static_assert(NPB == 1 || NPB == 2, "nodes per block");
  constexpr int VEC = Elem<T>::kPer16B;
  constexpr int NRB = 32 / NCH;  // largest row batch per wave
  constexpr int WPN = 4 / NPB;   // waves per node
  __shared__ unsigned long long cand[NPB][kWaveSelKmax];
  __shared__ double pre_s[NPB][kWaveSelKmax];
  __shared__ float alpha_s[NPB][kWaveSelKmax];
  __shared__ int idx_s[NPB][kWaveSelKmax];
  __shared__ __align__(16) float red[NPB][WPN - 1][64 * NCH * VEC];
  __shared__ int s_K[NPB];
  __shared__ int64_t s_m0[NPB];

  // a request's nodes share an XCD (and L2)
  const int pair = xcd_item(NPB == 2 ? (n_nodes + 1) / 2 : n_nodes);
  if (pair < 0) return;
  const int lane = threadIdx.x & 63;
  // waves are renumbered with the block so that the selecting waves of the blocks
  // resident on a CU fall on different SIMDs (a block's wave w runs on SIMD w)
  const int wave = ((threadIdx.x >> 6) + 2 * ((blockIdx.x >> 3) & 1)) & 3;
  const int nb = NPB == 2 ? (wave & 1) : 0;     // the node of the block this wave works on
  const int half = NPB == 2 ? (wave >> 1) : wave;  // 0: selects, then gathers its ranks
  const int cpr = a.d_m / VEC;
  {
    const int n = NPB * pair + nb;
    const bool live = n < n_nodes;
    if (half == 0) {
      uint32_t kv[NPL];
      NodeKeys nk;
      nk.ok = false;
      nk.m0 = 0;
      if (live) nk = load_node_keys<T, NPL>(a, n, lane, kv);
      int K = -1;
      float mass = 0.f;
      if (live) K = select_one_node<T, NPL>(a, n, lane, nk, kv, cand[nb], pre_s[nb], alpha_s[nb], idx_s[nb], &mass);
      if (lane == 0) {
        s_K[nb] = K;
        s_m0[nb] = nk.m0;
        if (K >= 0) {
          if (a.k_out) a.k_out[n] = K;
          if (a.mass_out) a.mass_out[n] = mass;
        }
      }
      if (K >= 0 && a.idx_out)
        for (int t = lane; t < a.k_max; t += 64) a.idx_out[static_cast<int64_t>(n) * a.k_max + t] = t < K ? idx_s[nb][t] : -1;
    }
    __syncthreads();
    const int K = s_K[nb];
    float acc[NCH][VEC];
#pragma unroll
    for (int u = 0; u < NCH; ++u)
#pragma unroll
      for (int x = 0; x < VEC; ++x) acc[u][x] = 0.f;
    if (K > 0) {
      const T* vbase = a.values + s_m0[nb] * a.d_m;
      const int* ix = idx_s[nb];
      const float* al = alpha_s[nb];
      const int mine = K > half ? (K - half + WPN - 1) / WPN : 0;  // ranks half, half + WPN, ...
      for (int q0 = 0; q0 < mine;) {
        const int left = mine - q0;
        const int t0 = half + WPN * q0;
        if (left >= NRB) {
          gather_rows<T, NCH, NRB>(vbase, a.d_m, cpr, ix, al, t0, WPN, NRB, lane, acc);
          q0 += NRB;
        } else if (left > NRB / 2) {
          gather_rows<T, NCH, NRB>(vbase, a.d_m, cpr, ix, al, t0, WPN, left, lane, acc);
          q0 += left;
        } else if (left > NRB / 4) {
          gather_rows<T, NCH, NRB / 2>(vbase, a.d_m, cpr, ix, al, t0, WPN, left, lane, acc);
          q0 += left;
        } else if (left > 2) {
          gather_rows<T, NCH, NRB / 4>(vbase, a.d_m, cpr, ix, al, t0, WPN, left, lane, acc);
          q0 += left;
        } else {
          gather_rows<T, NCH, 2>(vbase, a.d_m, cpr, ix, al, t0, WPN, left, lane, acc);
          q0 += left;
        }
      }
    }
    if (half > 0) {
#pragma unroll
      for (int u = 0; u < NCH; ++u)
#pragma unroll
        for (int x = 0; x < VEC; x += 4)
          *reinterpret_cast<f32x4*>(&red[nb][half - 1][(u * 64 + lane) * VEC + x]) =
              f32x4{acc[u][x], acc[u][x + 1], acc[u][x + 2], acc[u][x + 3]};
    }
    __syncthreads();
    if (half == 0 && K >= 0) {  // K < 0: invalid request, outputs already NaN
#pragma unroll
      for (int hh = 0; hh < WPN - 1; ++hh)
#pragma unroll
        for (int u = 0; u < NCH; ++u)
#pragma unroll
          for (int x = 0; x < VEC; x += 4) {
            const f32x4 p = *reinterpret_cast<const f32x4*>(&red[nb][hh][(u * 64 + lane) * VEC + x]);
            acc[u][x] += p[0];
            acc[u][x + 1] += p[1];
            acc[u][x + 2] += p[2];
            acc[u][x + 3] += p[3];
          }
      const int64_t rbase = static_cast<int64_t>(n) * a.d_m;
#pragma unroll
      for (int u = 0; u < NCH; ++u) {
        const int c = lane + 64 * u;
        if (c < cpr) {
          T outv[VEC];
#pragma unroll
          for (int x = 0; x < VEC; ++x) outv[x] = Elem<T>::from_f32(acc[u][x]);
          *reinterpret_cast<u32x4*>(a.rT + rbase + c * VEC) = *reinterpret_cast<const u32x4*>(outv);
          if (a.r_out) {
#pragma unroll
            for (int x = 0; x < VEC; x += 4)
              *reinterpret_cast<f32x4*>(a.r_out + rbase + c * VEC + x) =
                  f32x4{acc[u][x], acc[u][x + 1], acc[u][x + 2], acc[u][x + 3]};
          }
        }
      }
    }
  }
}

}  // namespace fovea
