// Draft candidates from the corrected state: logits z = W_LM h_hat over the vocabulary
// and the top-k tokens of every node (paper, Algorithm 1: the drafter's head expands
// each node into its K_c most likely tokens; experimental setup: tree with K_c = 6).
//
// Two kernels:
//  * lm_kernel: the logit GEMM in 128 x 128 tiles (the bf16 direct-to-LDS mainloop of
//    gemm.hpp) with an epilogue that keeps, for every row of the tile, its k largest
//    logits (ties to the lower token id) and writes them as candidates
//    [row][column tile][k] - the logits themselves never reach memory;
//  * lm_merge_kernel: one block per row merges the row's candidates into its top k.
// Tile order (LmMap): XCD x owns the x-th eighth of the column tiles, so each weight
// row is pulled into one L2 only; inside its slice an XCD walks groups of up to eight
// row tiles with the row fastest, so the blocks in flight on it cover a patch of about
// 8 x 4 tiles that share their h rows and weight rows through the L2, and a head too
// large for the Infinity Cache (Qwen's 1.09 GB) is read from HBM once per eight row
// tiles rather than once per row tile (measured: 6% on 768 rows of that head).
#pragma once

#include <cfloat>

#include "common.hpp"
#include "gemm.hpp"

namespace fovea {

template <typename T, int BM>
using LmCfg = GemmCfg<T, BM, 4>;

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

constexpr int kLmMaxK = 16;
constexpr int kLmMaxVocab = 1 << 24;
constexpr int kLmMaxRows = 1 << 20;

struct LmCand {
  float v;
  int32_t i;
};

// (v, i) ranks before (w, j): larger logit first, then the lower token id.  Bitwise
// operators on purpose: no short-circuit, so no branches.
__device__ __forceinline__ bool lm_before(float v, int i, float w, int j) {
  return (v > w) | ((v == w) & (i < j));
}

// The best (v, i) of each row of 16 lanes, in all 16 lanes: a butterfly over DPP row
// permutations (no LDS round trips).  All 16 lanes of the row must be active.
__device__ __forceinline__ void row16_best(float& bv, int& bi) {
#pragma unroll
  for (int sel = 0; sel < 4; ++sel) {
    const float ov = __uint_as_float(dpp_perm(__float_as_uint(bv), sel));
    const int oi = static_cast<int>(dpp_perm(static_cast<uint32_t>(bi), sel));
    if (lm_before(ov, oi, bv, bi)) {
      bv = ov;
      bi = oi;
    }
  }
}

// The best (v, i) over the whole (fully active) wave, uniform.
__device__ __forceinline__ void wave_best(float& bv, int& bi) {
  row16_best(bv, bi);
  float v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 0));
  int i = __builtin_amdgcn_readlane(bi, 0);
#pragma unroll
  for (int r = 1; r < 4; ++r) {
    const float ov = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bv), 16 * r));
    const int oi = __builtin_amdgcn_readlane(bi, 16 * r);
    if (lm_before(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
  bv = v;
  bi = i;
}

constexpr int kLmNone = 0x7FFFFFFF;  // id of an empty candidate slot

template <typename T, int BM>
__global__ __launch_bounds__(256) void lm_kernel(LmMap tm, int n, const T* __restrict__ h, int d,
                                                 const T* __restrict__ W, int vocab, int k,
                                                 LmCand* __restrict__ cand) {
  using C = LmCfg<T, BM>;
  __shared__ __align__(16) unsigned char smem[C::SMEM_BYTES];
  int tr, tc;
  if (!tm.map(tr, tc)) return;
  const int m0 = tr * C::BM, n0 = tc * C::BN;
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, h, d, n, W, d, vocab, d, m0, n0, smem);

  // stage one wave-row of the tile at a time (as gemm_epilogue does); the 16 threads of
  // a row are 16 consecutive lanes (one DPP row), each holding 8 consecutive logits.
  // Each thread handles GPT rows at once: their selection chains are independent, so
  // interleaving them hides the latency of each chain (one wave per SIMD here).
  float* so = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  constexpr int GROUPS = C::SROWS * (C::BN / 8);
  constexpr int GPT = GROUPS / C::NT;
  static_assert(GROUPS % C::NT == 0 && C::BN / 8 == 16, "epilogue mapping");
  const int c8 = threadIdx.x & 15;
  const int col0 = n0 + c8 * 8;
  const int nval = min(max(vocab - col0, 0), 8);  // valid logits of this thread
#pragma unroll
  for (int p = 0; p < C::WM; ++p) {
    if (wm == p) {
#pragma unroll
      for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
          for (int v = 0; v < 4; ++v)
            so[(i * 16 + 4 * (lane >> 4) + v) * C::SLD + wn * C::TN * 16 + j * 16 + (lane & 15)] =
                acc[i][j][v];
    }
    __syncthreads();
    float v[GPT][8];
    uint32_t avail[GPT];  // bit e: logit e not yet taken
#pragma unroll
    for (int g = 0; g < GPT; ++g) {
      const int r = (g * C::NT + static_cast<int>(threadIdx.x)) >> 4;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8 + 4);
      v[g][0] = lo[0]; v[g][1] = lo[1]; v[g][2] = lo[2]; v[g][3] = lo[3];
      v[g][4] = hi[0]; v[g][5] = hi[1]; v[g][6] = hi[2]; v[g][7] = hi[3];
      avail[g] = (1u << nval) - 1u;
    }
    // k rounds: each thread offers its best available logit, the row's 16 lanes agree
    // on the best of those, and its owner marks it taken
    for (int q = 0; q < k; ++q) {
      float bv[GPT];
      int bi[GPT];
#pragma unroll
      for (int g = 0; g < GPT; ++g) {
        bv[g] = -INFINITY;
        bi[g] = kLmNone;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          // ids ascend with e, so a later equal logit never displaces an earlier one
          const bool take = ((avail[g] >> e) & 1u) & lm_before(v[g][e], col0 + e, bv[g], bi[g]);
          bv[g] = take ? v[g][e] : bv[g];
          bi[g] = take ? col0 + e : bi[g];
        }
      }
#pragma unroll
      for (int sel = 0; sel < 4; ++sel) {
#pragma unroll
        for (int g = 0; g < GPT; ++g) {
          const float ov = __uint_as_float(dpp_perm(__float_as_uint(bv[g]), sel));
          const int oi = static_cast<int>(dpp_perm(static_cast<uint32_t>(bi[g]), sel));
          const bool b = lm_before(ov, oi, bv[g], bi[g]);
          bv[g] = b ? ov : bv[g];
          bi[g] = b ? oi : bi[g];
        }
      }
#pragma unroll
      for (int g = 0; g < GPT; ++g) {
        const uint32_t e = static_cast<uint32_t>(bi[g] - col0);
        avail[g] &= e < 8u ? ~(1u << e) : ~0u;
        const int row = m0 + p * C::SROWS + ((g * C::NT + static_cast<int>(threadIdx.x)) >> 4);
        if (c8 == 0 && row < n) {
          LmCand cd;
          cd.v = bv[g];
          cd.i = bi[g];
          cand[(static_cast<int64_t>(row) * tm.cb + tc) * k + q] = cd;
        }
      }
    }
    __syncthreads();
  }
}

// One block per row.  Every thread keeps the KM best of the candidates it reads (a
// sorted register list, updated by compare-and-swap down the list; its loads are issued
// eight at a time so their latencies overlap), each wave then extracts its k best in k
// rounds of wave_best (popping the winner from its owner's list), and wave 0 merges the
// four waves' k best the same way.
template <int KM>
__global__ __launch_bounds__(256) void lm_merge_kernel(int n_cand, int k,
                                                       const LmCand* __restrict__ cand,
                                                       int32_t* __restrict__ idx_out,
                                                       float* __restrict__ logit_out) {
  __shared__ float sv[4 * KM];
  __shared__ int si[4 * KM];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row = blockIdx.x;
  float lv[KM];
  int li[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    lv[j] = -INFINITY;
    li[j] = kLmNone;
  }
  const LmCand* cr = cand + row * n_cand;
  constexpr int U = 8;
  for (int t0 = 0; t0 < n_cand; t0 += 256 * U) {
    LmCand c[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int t = t0 + u * 256 + static_cast<int>(threadIdx.x);
      if (t < n_cand) {
        c[u] = cr[t];
      } else {
        c[u].v = -INFINITY;
        c[u].i = kLmNone;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float cv = c[u].v;
      int ci = c[u].i;
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        const bool sw = lm_before(cv, ci, lv[j], li[j]);
        const float tv = lv[j];
        const int ti = li[j];
        lv[j] = sw ? cv : tv;
        li[j] = sw ? ci : ti;
        cv = sw ? tv : cv;
        ci = sw ? ti : ci;
      }
    }
  }
  // each wave's k best; ids are distinct across the row's candidates, except the
  // empty-slot id, whose duplicates all pop harmlessly
  for (int q = 0; q < k; ++q) {
    float bv = lv[0];
    int bi = li[0];
    wave_best(bv, bi);
    if (lane == 0) {
      sv[wave * KM + q] = bv;
      si[wave * KM + q] = bi;
    }
    if (li[0] == bi) {
#pragma unroll
      for (int j = 0; j + 1 < KM; ++j) {
        lv[j] = lv[j + 1];
        li[j] = li[j + 1];
      }
      lv[KM - 1] = -INFINITY;
      li[KM - 1] = kLmNone;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  // lane l holds the (l % k)-th best of wave l / k (4 k <= 64 lanes)
  float cv = -INFINITY;
  int ci = kLmNone;
  if (lane < 4 * k) {
    cv = sv[(lane / k) * KM + lane % k];
    ci = si[(lane / k) * KM + lane % k];
  }
  for (int q = 0; q < k; ++q) {
    float bv = cv;
    int bi = ci;
    wave_best(bv, bi);
    if (lane == 0) {
      idx_out[row * k + q] = bi == kLmNone ? -1 : bi;
      if (logit_out != nullptr) logit_out[row * k + q] = bv;
    }
    if (ci == bi) {
      cv = -INFINITY;
      ci = kLmNone;
    }
  }
}

}  // namespace fovea
