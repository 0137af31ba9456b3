// Draft candidates from the corrected state: logits z = W_LM h_hat over the vocabulary
// and the top-k tokens of every node (paper, Eq. hidden_correction's z_n and Algorithm 1's
// tree expansion, which adds each node's K_c most likely tokens; K_c = 6 in the
// experimental setup).
//
// Two kernels:
//  * lm_kernel: the logit GEMM in 64, 128 or 256 x 128 tiles (the bf16
//    direct-to-LDS mainloop of gemm.hpp) with an epilogue that keeps, for every row of
//    the tile, its k largest logits and writes them as candidates [row][column tile][k]
//    - the logits themselves never reach memory;
//  * lm_merge_kernel: one block per row merges the row's candidates into its top k.
// A candidate is one 64-bit key: the logit mapped to an order-preserving unsigned
// integer in the high word and the complemented token id in the low word, so that one
// unsigned comparison orders by logit and then by ascending id.  A NaN logit and an
// empty slot are key 0, below every real logit (-inf included); key 0 decodes to id -1.
// Tile order (LmMap): XCD x owns the x-th eighth of the column tiles, so each weight
// row is pulled into one L2 only; inside its slice an XCD walks groups of up to eight
// row tiles with the row fastest, so the blocks in flight on it cover a patch of about
// 8 x 4 tiles that share their h rows and weight rows through the L2, and a head too
// large for the Infinity Cache (Qwen's 1.09 GB) is read from HBM once per eight row
// tiles rather than once per row tile (measured: 6% on 768 rows of that head).
// Selection has no serial rounds.  On 32-bit order-preserving images of the
// logits, every lane sorts its 8 values with a sorting network, then four butterfly
// steps over DPP row permutations each keep the 8 largest of two sorted lists (a
// bitonic half-cleaner and a bitonic sort of 8); all 16 lanes of a row then hold the
// row's 8 largest values, hence its k-th largest value T.  Each lane takes its values
// above T and, lowest ids first, the share of values equal to T that the k slots
// leave, placed by two row prefix counts (k = 9 .. 16 runs the same with 16-long
// lists).  With one wave per SIMD (the mainloop's LDS), a round-per-candidate selection
// was latency bound (about 43 us per round on 1920 x 32000 logits), and the same
// network on 64-bit (logit, id) keys spent most of its time in compare-to-select wait
// states.
#pragma once

#include <cfloat>

#include "common.hpp"
#include "gemm.hpp"

namespace fovea {

template <typename T, int BM>
using LmCfg = GemmCfg<T, BM, BM == 256 ? 3 : 4>;  // three 48 KB stages fit the 256-row tile

constexpr int kLmMaxK = 16;
constexpr int kLmMaxVocab = 1 << 24;
constexpr int kLmMaxRows = 1 << 20;

struct LmMap {
  int rb, cb;  // row and column tiles
  int rc;      // column tiles per XCD
  int gr;      // row tiles per group
  __device__ __forceinline__ bool map(int& tr, int& tc) const {
    const int x = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int g = slot / (gr * rc);
    const int r0 = g * gr;
    if (r0 >= rb) return false;
    const int gs = min(gr, rb - r0);
    const int loc = slot - g * gr * rc;
    tr = r0 + loc % gs;
    const int lc = loc / gs;
    tc = x * rc + lc;
    return lc < rc && tc < cb;
  }
};

inline LmMap make_lm_map(int rb, int cb) {
  LmMap m;
  m.rb = rb;
  m.cb = cb;
  m.rc = (cb + 7) / 8;
  m.gr = rb < 8 ? rb : 8;
  return m;
}

inline int lm_grid(const LmMap& m) { return 8 * m.rb * m.rc; }

// ---- candidate keys -------------------------------------------------------------

// order-preserving image of a logit (-0 taken as +0, so equal logits tie on the id);
// 0 for NaN, which is below the image of -inf
__device__ __forceinline__ uint32_t lm_ord(float v) {
  const uint32_t u = __float_as_uint(v + 0.0f);
  const uint32_t o = u ^ (static_cast<uint32_t>(static_cast<int32_t>(u) >> 31) | 0x80000000u);
  return v == v ? o : 0u;
}

__device__ __forceinline__ uint64_t lm_key_of(uint32_t o, int id) {
  return o == 0u ? 0ull : (static_cast<uint64_t>(o) << 32) | static_cast<uint32_t>(~id);
}

__device__ __forceinline__ uint64_t lm_key(float v, int id) { return lm_key_of(lm_ord(v), id); }

__device__ __forceinline__ int lm_key_id(uint64_t key) {
  return static_cast<int>(~static_cast<uint32_t>(key));
}

__device__ __forceinline__ float lm_key_val(uint64_t key) {
  if (key == 0ull) return -INFINITY;
  const uint32_t o = static_cast<uint32_t>(key >> 32);
  return __uint_as_float((o >> 31) ? (o ^ 0x80000000u) : ~o);
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

// a and b in descending order (larger first); for 32-bit keys these are v_max / v_min,
// which need no compare result (a 64-bit compare goes through VCC, and reading VCC right
// after writing it costs wait states on this chip)
template <typename K>
__device__ __forceinline__ void cas_desc(K& a, K& b) {
  const K hi = a > b ? a : b, lo = a > b ? b : a;
  a = hi;
  b = lo;
}

__device__ __forceinline__ uint32_t dpp_perm_k(uint32_t v, int sel) { return dpp_perm(v, sel); }

__device__ __forceinline__ uint64_t dpp_perm_k(uint64_t v, int sel) {
  const uint64_t lo = dpp_perm(static_cast<uint32_t>(v), sel);
  const uint64_t hi = dpp_perm(static_cast<uint32_t>(v >> 32), sel);
  return lo | (hi << 32);
}

// Batcher's odd-even merge sort of the first 8 keys, descending (19 comparators,
// depth 6).
template <int N, typename K>
__device__ __forceinline__ void sort8_desc(K (&a)[N]) {
  static_assert(N >= 8, "list length");
  cas_desc(a[0], a[1]); cas_desc(a[2], a[3]); cas_desc(a[4], a[5]); cas_desc(a[6], a[7]);
  cas_desc(a[0], a[2]); cas_desc(a[1], a[3]); cas_desc(a[4], a[6]); cas_desc(a[5], a[7]);
  cas_desc(a[1], a[2]); cas_desc(a[5], a[6]);
  cas_desc(a[0], a[4]); cas_desc(a[1], a[5]); cas_desc(a[2], a[6]); cas_desc(a[3], a[7]);
  cas_desc(a[2], a[4]); cas_desc(a[3], a[5]);
  cas_desc(a[1], a[2]); cas_desc(a[3], a[4]); cas_desc(a[5], a[6]);
}

// Sorts a bitonic sequence of N keys (N a power of two) into descending order.
template <int N, typename K>
__device__ __forceinline__ void bitonic_desc(K (&a)[N]) {
#pragma unroll
  for (int dd = N / 2; dd >= 1; dd >>= 1)
#pragma unroll
    for (int i = 0; i < N; ++i)
      if ((i & dd) == 0) cas_desc(a[i], a[i + dd]);
}

// One butterfly step: the N largest of this lane's sorted list and its DPP partner's
// (partner `sel` of dpp_perm), sorted.  Both partners end with the same list.
template <int N, typename K>
__device__ __forceinline__ void merge_step(K (&a)[N], int sel) {
  K p[N];
#pragma unroll
  for (int i = 0; i < N; ++i) p[i] = dpp_perm_k(a[N - 1 - i], sel);
#pragma unroll
  for (int i = 0; i < N; ++i) a[i] = a[i] > p[i] ? a[i] : p[i];
  bitonic_desc<N>(a);
}

// Largest key over each 16-lane row (all 16 lanes active), in all 16 lanes.
__device__ __forceinline__ uint64_t row16_max64(uint64_t v) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) v = umax64(v, dpp_perm_k(v, sel));
  return v;
}

// Largest key over the whole (fully active) wave, uniform.
__device__ __forceinline__ uint64_t wave_max64(uint64_t v) {
  v = row16_max64(v);
  uint64_t m = 0;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const uint64_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), 16 * r));
    const uint64_t hi =
        static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v >> 32), 16 * r));
    m = umax64(m, lo | (hi << 32));
  }
  return m;
}

// The k (<= LL) largest logits of two rows of a 128-column tile, each row spread over
// the 16 lanes of a DPP row (8 consecutive columns per lane, starting at col0), written
// in any order as the k candidates of (row, tile).  th = the row's k-th largest value,
// found on 32-bit order-preserving images with a sorting network and LL-long butterfly
// merges; every lane then takes its values above th and, lowest ids first, the share of
// values equal to th that the k slots leave, placed by two row prefix counts.
template <int LL>
__device__ __forceinline__ void lm_select_rows(const float (&v)[2][8], const int (&row)[2],
                                               int col0, int vocab, int k, int n,
                                               uint64_t* __restrict__ cand, int n_tiles,
                                               int tile) {
  uint32_t o[2][8], L[2][LL];
#pragma unroll
  for (int g = 0; g < 2; ++g) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // masked, not branched: columns past the vocabulary are empty
      o[g][e] = lm_ord(v[g][e]) & (0u - static_cast<uint32_t>(col0 + e < vocab));
      L[g][e] = o[g][e];
    }
#pragma unroll
    for (int e = 8; e < LL; ++e) L[g][e] = 0u;
  }
  sort8_desc(L[0]);  // the zero tail of an LL = 16 list is already in place
  sort8_desc(L[1]);
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) {
    merge_step<LL>(L[0], sel);
    merge_step<LL>(L[1], sel);
  }
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    uint32_t th = L[g][0];
#pragma unroll
    for (int q = 1; q < LL; ++q)
      if (q < k) th = min(th, L[g][q]);
    int c_gt = 0, n_gt = 0, n_eq = 0;
#pragma unroll
    for (int q = 0; q < LL; ++q) c_gt += (q < k) & (L[g][q] > th);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      n_gt += o[g][e] > th;
      n_eq += o[g][e] == th;
    }
    const int need = k - c_gt;  // slots left for values equal to th
    const int eq_before = row16_incl_scan_i32(n_eq) - n_eq;
    const int take = min(max(need - eq_before, 0), n_eq);
    const int nsel = n_gt + take;
    int slot = row16_incl_scan_i32(nsel) - nsel;
    if (row[g] < n) {
      uint64_t* dst = cand + (static_cast<int64_t>(row[g]) * n_tiles + tile) * k;
      int r = eq_before;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool eq = o[g][e] == th;
        const bool s = (o[g][e] > th) | (eq & (r < need));
        r += eq;
        if (s) dst[slot] = lm_key_of(o[g][e], col0 + e);
        slot += s;
      }
    }
  }
}

// ---- logits GEMM + per-tile candidates --------------------------------------------

template <typename T, int BM>
__global__ __launch_bounds__(256) void lm_kernel(LmMap tm, int n, const T* __restrict__ h, int d,
                                                 const T* __restrict__ W, int vocab, int k,
                                                 uint64_t* __restrict__ cand) {
  using C = LmCfg<T, BM>;
  // the pipeline's stages, then the whole tile of fp32 logits
  constexpr int kTileBytes = C::BM * C::SLD * 4;
  constexpr int kSmem = C::SMEM_BYTES > kTileBytes ? C::SMEM_BYTES : kTileBytes;
  static_assert(kSmem <= 160 * 1024, "LDS");
  __shared__ __align__(16) unsigned char smem[kSmem];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, h, d, n, W, d, vocab, d, m0, n0, smem);

  // stage the whole tile in LDS (the accumulators are then dead), then select: the 16
  // threads of a row are 16 consecutive lanes (one DPP row), each holding 8 consecutive
  // logits; each thread handles GPT rows, two at a time so that their independent
  // selections interleave without spilling
  float* so = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  constexpr int GPT = C::BM * (C::BN / 8) / C::NT;
  static_assert(GPT % 2 == 0 && C::BN / 8 == 16, "epilogue mapping");
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        so[(wm * C::SROWS + i * 16 + 4 * (lane >> 4) + v) * C::SLD + wn * C::TN * 16 + j * 16 +
           (lane & 15)] = acc[i][j][v];
  __syncthreads();
  const int c8 = threadIdx.x & 15;
  const int col0 = n0 + c8 * 8;
#pragma unroll
  for (int g0 = 0; g0 < GPT; g0 += 2) {
    int row[2];
    float v[2][8];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const int r = ((g0 + g) * C::NT + static_cast<int>(threadIdx.x)) >> 4;
      row[g] = m0 + r;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8 + 4);
      v[g][0] = lo[0]; v[g][1] = lo[1]; v[g][2] = lo[2]; v[g][3] = lo[3];
      v[g][4] = hi[0]; v[g][5] = hi[1]; v[g][6] = hi[2]; v[g][7] = hi[3];
    }
    if (k <= 8)
      lm_select_rows<8>(v, row, col0, vocab, k, n, cand, tm.cb, tc);
    else
      lm_select_rows<16>(v, row, col0, vocab, k, n, cand, tm.cb, tc);
  }
}

// ---- merge of a row's candidates --------------------------------------------------

// One block per row.  Every thread keeps the KM largest of the keys it reads (a sorted
// register list, updated by compare-and-swap down the list; its loads are issued eight
// at a time so that their latencies overlap).  For k <= 8 (KM = 8) the lists are then
// merged by the butterfly of the logits kernel: within each 16-lane row, then the
// sixteen row winners of the block in wave 0.  For larger k every wave extracts its
// k largest in k rounds and wave 0 ranks the 4 k survivors by counting.
template <int KM>
__global__ __launch_bounds__(256) void lm_merge_kernel(int n_cand, int k,
                                                       const uint64_t* __restrict__ cand,
                                                       int32_t* __restrict__ idx_out,
                                                       float* __restrict__ logit_out) {
  __shared__ uint64_t sk[16 * KM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = blockIdx.x;
  uint64_t l[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) l[j] = 0ull;
  const uint64_t* cr = cand + row * n_cand;
  constexpr int U = 8;
  for (int t0 = 0; t0 < n_cand; t0 += 256 * U) {
    uint64_t c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * 256 + static_cast<int>(threadIdx.x);
      c[u] = t < n_cand ? cr[t] : 0ull;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      uint64_t x = c[u];
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        const uint64_t t = l[j];
        l[j] = umax64(t, x);
        x = t > x ? x : t;
      }
    }
  }
  if constexpr (KM == 8) {
#pragma unroll
    for (int sel = 0; sel < 4; ++sel) merge_step<8>(l, sel);
    if ((lane & 15) == 0) {
#pragma unroll
      for (int j = 0; j < 8; ++j) sk[(wave * 4 + (lane >> 4)) * 8 + j] = l[j];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int j = 0; j < 8; ++j) l[j] = lane < 16 ? sk[lane * 8 + j] : 0ull;
#pragma unroll
    for (int sel = 0; sel < 4; ++sel) merge_step<8>(l, sel);
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        if (q < k) {
          idx_out[row * k + q] = lm_key_id(l[q]);
          if (logit_out != nullptr) logit_out[row * k + q] = lm_key_val(l[q]);
        }
    }
  } else {
    for (int q = 0; q < k; ++q) {
      const uint64_t b = wave_max64(l[0]);
      if (lane == 0) sk[wave * KM + q] = b;
      if (l[0] == b) {
#pragma unroll
        for (int j = 0; j + 1 < KM; ++j) l[j] = l[j + 1];
        l[KM - 1] = 0ull;
      }
    }
    __syncthreads();
    if (wave != 0 || lane >= 4 * k) return;
    // rank among the 4 k survivors; equal keys (only 0) rank by position
    const uint64_t x = sk[(lane / k) * KM + lane % k];
    int rank = 0;
    for (int j = 0; j < 4 * k; ++j) {
      const uint64_t y = sk[(j / k) * KM + j % k];
      rank += (y > x) | ((y == x) & (j < lane));
    }
    if (rank < k) {
      idx_out[row * k + rank] = lm_key_id(x);
      if (logit_out != nullptr) logit_out[row * k + rank] = lm_key_val(x);
    }
  }
}

}  // namespace fovea
