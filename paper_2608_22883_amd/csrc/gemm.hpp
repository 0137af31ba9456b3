// MFMA GEMM for gfx950: acc[m, n] = sum_k A[m, k] * B[n, k], with an LDS-staged epilogue.
//
// A is a row-major activation [rows, K] (K contiguous); B is a row-major weight [N, K]
// (the nn.Linear layout).  Block tile BM x 128 run by 2 x 2 wave64s; each wave owns a
// TM x TN grid of 16x16 MFMA accumulators.  Rows past M and columns past N are clamped
// on load; the epilogue hands them to the caller's functor, which drops them.
//
// bf16 mainloop: global -> LDS by direct-to-LDS loads (no register staging), NST LDS
// stages, k-tile kt + NST - 1 in flight while the matrix cores work on tile kt, one
// barrier per k-step.  A k-tile row is 64 bf16 = 128 B = 8 chunks of 16 B, stored with
// chunk c of row r at slot c ^ ((r >> 1) & 7): the 16 rows read by one fragment load
// then fall on distinct bank groups.  A direct-to-LDS load writes lane L's 16 bytes at
// LDS base + 16 L, so the swizzle is applied by choosing which global chunk each lane
// fetches.  The wait before each barrier counts this thread's outstanding loads
// exactly (loads retire in issue order), so tiles further ahead stay in flight.
//
// fp32 mainloop: register-staged copy into a double-buffered, padded LDS tile
// (MFMA 16x16x4 f32).
//
// Epilogue: the accumulators go through LDS (fp32, one wave-row of the tile per pass),
// and each thread then owns 8 consecutive columns of a row, so stores and the loads of
// epilogue operands are 16-byte, row-contiguous.  The 16 threads of a row are 16
// consecutive lanes; a per-row value returned by the functor is summed over them.
//
// Tiles are mapped to XCDs (blocks are dispatched round-robin over the 8 XCDs): the
// tile grid is cut into an xr x xc grid of regions and region x runs on XCD x, so the
// blocks sharing an XCD's L2 share A rows and B columns.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace fovea {

typedef __attribute__((address_space(3))) void* lds_void_ptr;

template <typename T, int BM_, int NST_ = 4>
struct GemmCfg {
  static constexpr int BM = BM_, BN = 128, WM = 2, WN = 2;
  static constexpr int NT = WM * WN * kWave;
  static constexpr int TM = BM / WM / 16;
  static constexpr int TN = BN / WN / 16;
  static constexpr int VEC = Elem<T>::kPer16B;  // elements per 16-byte chunk
  static constexpr int BK = 8 * VEC;            // k-tile: 64 bf16 or 32 fp32
  static constexpr bool DMA = VEC == 8;         // bf16: direct-to-LDS pipeline
  static constexpr int NST = DMA ? NST_ : 2;
  // bf16 rows are 128 B (swizzled), fp32 rows padded by one chunk
  static constexpr int LDK = DMA ? BK : BK + VEC;
  static constexpr int STAGE_BYTES = (BM + BN) * LDK * static_cast<int>(sizeof(T));
  // direct-to-LDS loads per wave per k-tile (one load moves 8 rows)
  static constexpr int A_DMA = BM / 8 / 4;
  static constexpr int B_DMA = BN / 8 / 4;
  // fp32 register staging: 16-byte chunks per thread per k-tile
  static constexpr int A_CHUNKS = BM * 8 / NT;
  static constexpr int B_CHUNKS = BN * 8 / NT;
  // epilogue staging: one wave-row (TM * 16 rows) of fp32 with a 4-float pad
  static constexpr int SROWS = TM * 16;
  static constexpr int SLD = BN + 4;
  static constexpr int OUT_BYTES = SROWS * SLD * 4;
  static constexpr int PIPE_BYTES = NST * STAGE_BYTES;
  static constexpr int SMEM_BYTES = PIPE_BYTES > OUT_BYTES ? PIPE_BYTES : OUT_BYTES;
  static_assert(BM == 64 || BM == 128 || BM == 256, "block rows");
  static_assert(NST >= 2 && NST <= 5, "pipeline depth");
  static_assert(SMEM_BYTES <= 160 * 1024, "LDS");
};

// Position of a block's tile in the (row-block, column-block) grid; false for padding.
struct TileMap {
  int rb, cb;  // tiles along M and N
  int xr, xc;  // XCD regions along M and N (xr * xc == 8)
  __device__ __forceinline__ bool map(int& tr, int& tc) const {
    const int xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int rr = (rb + xr - 1) / xr, rc = (cb + xc - 1) / xc;
    const int lr = slot / rc, lc = slot % rc;
    tr = (xcd / xc) * rr + lr;
    tc = (xcd % xc) * rc + lc;
    return lr < rr && tr < rb && tc < cb;
  }
};

inline TileMap make_tile_map(int rb, int cb, double a_bytes, double b_bytes) {
  // region grid minimising the bytes pulled into the 8 L2s: xc copies of A, xr of B
  TileMap m{rb, cb, 8, 1};
  double best = -1.0;
  for (int xr = 1; xr <= 8; xr *= 2) {
    const int xc = 8 / xr;
    const double cost = xc * a_bytes + xr * b_bytes;
    if (best < 0.0 || cost < best) {
      best = cost;
      m.xr = xr;
      m.xc = xc;
    }
  }
  return m;
}

__host__ __device__ inline int tile_grid(const TileMap& m) {
  return 8 * ((m.rb + m.xr - 1) / m.xr) * ((m.cb + m.xc - 1) / m.xc);
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits 3:0 and
// 15:14, expcnt and lgkmcnt fields at their maxima, i.e. not waited on).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `ahead` k-tiles of direct-to-LDS loads (NI loads each) are still
// outstanding; ahead is clamped to MAXA (the pipeline's steady-state lead).
template <int NI, int MAXA>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if constexpr (MAXA <= 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= MAXA)
      wait_vmcnt<MAXA * NI>();
    else
      wait_tiles<NI, MAXA - 1>(ahead);
  }
}

// Workgroup barrier without a memory fence: a fence would also wait for the
// direct-to-LDS loads still in flight.  The compiler barriers keep LDS accesses on
// their side of it.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <class C>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[C::TM][C::TN]) {
#pragma unroll
  for (int i = 0; i < C::TM; ++i)
#pragma unroll
    for (int j = 0; j < C::TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// bf16 mainloop (direct-to-LDS pipeline).  A: [M, K] row-major with leading dim lda.
template <class C>
__device__ __forceinline__ void gemm_mainloop_dma(f32x4 (&acc)[C::TM][C::TN],
                                                  const bf16_t* __restrict__ A, int64_t lda, int M,
                                                  const bf16_t* __restrict__ Bw, int64_t ldb, int N,
                                                  int K, int m0, int n0, unsigned char* smem) {
  constexpr int TM = C::TM, TN = C::TN, NST = C::NST;
  constexpr int NI = C::A_DMA + C::B_DMA;
  constexpr int NH = TM + TN;  // fragments per 32-wide k half
  const int lane = threadIdx.x & 63;
  // the wave index is uniform: derived addresses (the direct-to-LDS destinations above
  // all) stay in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) >> 6);
  const int wm = wave / C::WN, wn = wave % C::WN;
  zero_acc<C>(acc);

  // sources and LDS row offsets of this thread's direct-to-LDS loads
  const bf16_t* ga[C::A_DMA];
  const bf16_t* gb[C::B_DMA];
  int da[C::A_DMA], db[C::B_DMA];
#pragma unroll
  for (int j = 0; j < C::A_DMA; ++j) {
    const int r0 = (wave * C::A_DMA + j) * 8;
    const int row = r0 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    ga[j] = A + static_cast<int64_t>(min(m0 + row, M - 1)) * lda + c * 8;
    da[j] = r0 * 128;
  }
#pragma unroll
  for (int j = 0; j < C::B_DMA; ++j) {
    const int r0 = (wave * C::B_DMA + j) * 8;
    const int row = r0 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    gb[j] = Bw + static_cast<int64_t>(min(n0 + row, N - 1)) * ldb + c * 8;
    db[j] = (C::BM + r0) * 128;
  }
  // fragment byte offsets (within a stage) for the two 32-wide k halves of a tile:
  // lane reads chunk 4 h + lane / 16 of row (.. + lane % 16); the swizzle term is the
  // same for all 16-row blocks of the lane
  const int arow = wm * TM * 16 + (lane & 15);
  const int brow = C::BM + wn * TN * 16 + (lane & 15);
  int fa[2], fb[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    fa[h] = arow * 128 + (((4 * h + (lane >> 4)) ^ ((arow >> 1) & 7)) << 4);
    fb[h] = brow * 128 + (((4 * h + (lane >> 4)) ^ ((brow >> 1) & 7)) << 4);
  }
  const int nk = K / C::BK;
  // fragment r (0 .. NH - 1) of half h of the tile in stage st, in the order the i-major
  // MFMAs first use them: A0, B0 .. B(TN-1), A1 .. A(TM-1)
  auto read_frag = [&](const unsigned char* st, int h, int r, bf16x8 (&af)[TM], bf16x8 (&bf)[TN]) {
    if (r == 0)
      af[0] = *reinterpret_cast<const bf16x8*>(st + fa[h]);
    else if (r <= TN)
      bf[r - 1] = *reinterpret_cast<const bf16x8*>(st + fb[h] + (r - 1) * 16 * 128);
    else
      af[r - TN] = *reinterpret_cast<const bf16x8*>(st + fa[h] + (r - TN) * 16 * 128);
  };
  // load q (0 .. NI - 1) of tile kt into its stage
  auto issue_one = [&](int kt, int q) {
    unsigned char* sn = smem + (kt % NST) * C::STAGE_BYTES;
    const int k0 = kt * C::BK;
    if (q < C::A_DMA)
      __builtin_amdgcn_global_load_lds(ga[q] + k0, (lds_void_ptr)(sn + da[q]), 16, 0, 0);
    else
      __builtin_amdgcn_global_load_lds(gb[q - C::A_DMA] + k0, (lds_void_ptr)(sn + db[q - C::A_DMA]), 16, 0, 0);
  };
  // Step kt, with the first k half of tile kt already in registers (set P):
  //   1. its MFMAs, each followed by one read of the tile's second half and then by one
  //      load of tile kt + NST - 1 (into the stage tile kt - 1 used);
  //   2. this wave's reads done, its loads of tile kt + 1 done, then the barrier: tile
  //      kt + 1 is visible and every wave has finished reading stage kt;
  //   3. the second half's MFMAs, each followed by one read of tile kt + 1's first half
  //      (set 1 - P), so that read latency hides behind matrix work.
  // Loads are issued for every step (past the last tile the last tile is loaded again
  // into a stage nobody reads), so the wait is a fixed count of this thread's loads
  // (they retire in issue order).  After the last step the reads of step 3 touch a stage
  // whose contents are not used.  The compiler barriers keep each access in its slot.
  bf16x8 af0[2][TM], bf0[2][TN], af1[TM], bf1[TN];
  auto step = [&](int kt, auto P) {
    constexpr int p = decltype(P)::value;
    const unsigned char* st = smem + (kt % NST) * C::STAGE_BYTES;
    const unsigned char* sn = smem + ((kt + 1) % NST) * C::STAGE_BYTES;
    const int knext = min(kt + NST - 1, nk - 1);
#pragma unroll
    for (int m = 0; m < TM * TN; ++m) {
      mfma_bf16_16x16x32_acc(acc[m / TN][m % TN], af0[p][m / TN], bf0[p][m % TN]);
      if (m < NH)
        read_frag(st, 1, m, af1, bf1);
      else if (m - NH < NI)
        issue_one(knext, m - NH);
      asm volatile("" ::: "memory");
    }
#pragma unroll
    for (int q = TM * TN - NH; q < NI; ++q) issue_one(knext, q);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's reads of the stage done
    wait_vmcnt<(NST - 2) * NI>();
    lds_barrier();
#pragma unroll
    for (int m = 0; m < TM * TN; ++m) {
      mfma_bf16_16x16x32_acc(acc[m / TN][m % TN], af1[m / TN], bf1[m % TN]);
      if (m < NH) read_frag(sn, 0, m, af0[1 - p], bf0[1 - p]);
      asm volatile("" ::: "memory");
    }
  };
  // prologue: tiles 0 .. NST - 2, each tile's loads together (in issue order)
#pragma unroll
  for (int s = 0; s < NST - 1; ++s)
#pragma unroll
    for (int q = 0; q < NI; ++q) issue_one(min(s, nk - 1), q);
  wait_vmcnt<(NST - 2) * NI>();
  lds_barrier();
#pragma unroll
  for (int r = 0; r < NH; ++r) read_frag(smem, 0, r, af0[0], bf0[0]);
  asm volatile("" ::: "memory");
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    step(kt, std::integral_constant<int, 0>());
    step(kt + 1, std::integral_constant<int, 1>());
  }
  if (kt < nk) step(kt, std::integral_constant<int, 0>());
  // the extra loads of the last steps land before the LDS is reused
  wait_vmcnt<0>();
  mfma_results_ready();
  lds_barrier();
}

// fp32 mainloop: register-staged, double-buffered LDS.
template <class C>
__device__ __forceinline__ void gemm_mainloop_f32(f32x4 (&acc)[C::TM][C::TN],
                                                  const float* __restrict__ A, int64_t lda, int M,
                                                  const float* __restrict__ Bw, int64_t ldb, int N,
                                                  int K, int m0, int n0, unsigned char* smem_raw) {
  constexpr int TM = C::TM, TN = C::TN;
  float* smem = reinterpret_cast<float*>(smem_raw);
  constexpr int STAGE = (C::BM + C::BN) * C::LDK;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  zero_acc<C>(acc);
  const float* ga[C::A_CHUNKS];
  const float* gb[C::B_CHUNKS];
  int la[C::A_CHUNKS], lb[C::B_CHUNKS];
#pragma unroll
  for (int j = 0; j < C::A_CHUNKS; ++j) {
    const int c = tid + j * C::NT;
    ga[j] = A + static_cast<int64_t>(min(m0 + (c >> 3), M - 1)) * lda + (c & 7) * 4;
    la[j] = (c >> 3) * C::LDK + (c & 7) * 4;
  }
#pragma unroll
  for (int j = 0; j < C::B_CHUNKS; ++j) {
    const int c = tid + j * C::NT;
    gb[j] = Bw + static_cast<int64_t>(min(n0 + (c >> 3), N - 1)) * ldb + (c & 7) * 4;
    lb[j] = (C::BM + (c >> 3)) * C::LDK + (c & 7) * 4;
  }
  const int aoff = (wm * TM * 16 + (lane & 15)) * C::LDK + (lane >> 4);
  const int boff = (C::BM + wn * TN * 16 + (lane & 15)) * C::LDK + (lane >> 4);
  const int nk = K / C::BK;
  u32x4 ra[C::A_CHUNKS], rb[C::B_CHUNKS];
#pragma unroll
  for (int j = 0; j < C::A_CHUNKS; ++j) ra[j] = *reinterpret_cast<const u32x4*>(ga[j]);
#pragma unroll
  for (int j = 0; j < C::B_CHUNKS; ++j) rb[j] = *reinterpret_cast<const u32x4*>(gb[j]);
  for (int kt = 0; kt < nk; ++kt) {
    float* st = smem + (kt & 1) * STAGE;
#pragma unroll
    for (int j = 0; j < C::A_CHUNKS; ++j) *reinterpret_cast<u32x4*>(st + la[j]) = ra[j];
#pragma unroll
    for (int j = 0; j < C::B_CHUNKS; ++j) *reinterpret_cast<u32x4*>(st + lb[j]) = rb[j];
    const int k1 = min(kt + 1, nk - 1) * C::BK;
#pragma unroll
    for (int j = 0; j < C::A_CHUNKS; ++j) ra[j] = *reinterpret_cast<const u32x4*>(ga[j] + k1);
#pragma unroll
    for (int j = 0; j < C::B_CHUNKS; ++j) rb[j] = *reinterpret_cast<const u32x4*>(gb[j] + k1);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < C::BK; kk += 4) {
      float af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = st[aoff + i * 16 * C::LDK + kk];
#pragma unroll
      for (int j = 0; j < TN; ++j) bf[j] = st[boff + j * 16 * C::LDK + kk];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma_f32_16x16x4(af[i], bf[j], acc[i][j]);
    }
  }
  __syncthreads();
}

template <class C, typename T>
__device__ __forceinline__ void gemm_mainloop(f32x4 (&acc)[C::TM][C::TN], const T* A, int64_t lda,
                                              int M, const T* Bw, int64_t ldb, int N, int K, int m0,
                                              int n0, unsigned char* smem) {
  if constexpr (C::DMA)
    gemm_mainloop_dma<C>(acc, A, lda, M, Bw, ldb, N, K, m0, n0, smem);
  else
    gemm_mainloop_f32<C>(acc, A, lda, M, Bw, ldb, N, K, m0, n0, smem);
}

// LDS-staged epilogue.  f(row, col0, v) sees the 8 accumulators of columns
// col0 .. col0 + 7 of `row` (rows and columns past the matrix included: f drops them)
// and returns a per-row contribution; fr(row, sum) receives the sum of the
// contributions over the tile's 128 columns (lane order fixed, so deterministic).
// Must be reached by every thread of the block.
template <class C, class F, class FR>
__device__ __forceinline__ void gemm_epilogue(const f32x4 (&acc)[C::TM][C::TN],
                                              unsigned char* smem, int m0, int n0, F&& f,
                                              FR&& fr) {
  float* so = reinterpret_cast<float*>(smem);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  constexpr int GROUPS = C::SROWS * (C::BN / 8);
  static_assert(GROUPS % C::NT == 0 && C::BN / 8 == 16, "epilogue mapping");
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
#pragma unroll
    for (int g0 = 0; g0 < GROUPS; g0 += C::NT) {
      const int g = g0 + static_cast<int>(threadIdx.x);
      const int r = g >> 4, c8 = g & 15;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(so + r * C::SLD + c8 * 8 + 4);
      const float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      const int row = m0 + p * C::SROWS + r;
      float s;
      // functors that take the group index gi (compile-time after unrolling) can hold
      // operands prefetched per group (epilogue_group)
      if constexpr (std::is_invocable_v<F, int, int, const float(&)[8], int>)
        s = f(row, n0 + c8 * 8, v, p * (GROUPS / C::NT) + g0 / C::NT);
      else
        s = f(row, n0 + c8 * 8, v);
      s = sum16(s);
      if ((lane & 15) == 0) fr(row, s);
    }
    __syncthreads();
  }
}

// Row and first column of epilogue group gi of this thread (gemm_epilogue's mapping):
// groups per thread C::WM * C::SROWS * 16 / C::NT.
template <class C>
__device__ __forceinline__ void epilogue_group(int gi, int m0, int n0, int& row, int& col0) {
  constexpr int PER = C::SROWS * 16 / C::NT;
  const int p = gi / PER, g = (gi % PER) * C::NT + static_cast<int>(threadIdx.x);
  row = m0 + p * C::SROWS + (g >> 4);
  col0 = n0 + (g & 15) * 8;
}

struct NoRowSum {
  __device__ __forceinline__ void operator()(int, float) const {}
};

// Split-K for GEMMs with too few output tiles to fill the chip: block (tile, y) contracts
// K slice y (Kc = K / ks columns, a multiple of BK) and stores its fp32 partial tile in
// part[y][M][N]; a combine kernel then sums the slices in order and runs the fused
// kernel's epilogue (splitk_combine), so the result does not depend on timing.
template <class C, typename T>
__device__ __forceinline__ void gemm_splitk_partial(const T* A, int64_t lda, int M, const T* Bw,
                                                    int64_t ldb, int N, int K, int ks, int m0,
                                                    int n0, float* __restrict__ part,
                                                    unsigned char* smem) {
  const int Kc = K / ks;
  const int k0 = static_cast<int>(blockIdx.y) * Kc;
  f32x4 acc[C::TM][C::TN];
  gemm_mainloop<C>(acc, A + k0, lda, M, Bw + k0, ldb, N, Kc, m0, n0, smem);
  float* pp = part + static_cast<int64_t>(blockIdx.y) * M * N;
  gemm_epilogue<C>(
      acc, smem, m0, n0,
      [&](int row, int col0, const float(&v)[8]) -> float {
        if (row < M && col0 < N) store8(pp + static_cast<int64_t>(row) * N + col0, v);
        return 0.f;
      },
      NoRowSum{});
}

// One block of 256 threads per (16 rows, 128-column tile blockIdx.x): thread t owns
// columns 8 (t % 16) .. + 7 of row 16 blockIdx.y + t / 16, sums the ks partials in slice
// order and calls f(row, col0, v) and fr(row, sum over the tile's 128 columns) exactly
// as gemm_epilogue does (rows and columns past the matrix included: f drops them).
template <class F, class FR>
__device__ __forceinline__ void splitk_combine(int M, int N, int ks, const float* __restrict__ part,
                                               F&& f, FR&& fr) {
  const int row = static_cast<int>(blockIdx.y) * 16 + static_cast<int>(threadIdx.x >> 4);
  const int col0 = static_cast<int>(blockIdx.x) * 128 + static_cast<int>(threadIdx.x & 15) * 8;
  float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (row < M && col0 < N) {
    // eight slices' loads in flight at a time, added in slice order
    for (int y0 = 0; y0 < ks; y0 += 8) {
      float t[8][8];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (y0 + u < ks) load8(part + (static_cast<int64_t>(y0 + u) * M + row) * N + col0, t[u]);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (y0 + u < ks)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += t[u][e];
    }
  }
  float s = f(row, col0, v);
  s = sum16(s);
  if ((threadIdx.x & 15) == 0) fr(row, s);
}

// Number of K slices for a GEMM of `tiles` output tiles: powers of two while the grid
// stays within one block per compute unit and every slice keeps >= 2 k-tiles.
inline int splitk_slices(int tiles, int K, int BK) {
  int ks = 1;
  if (tiles >= 128) return 1;
  while (tiles * ks * 2 <= 256 && K % (BK * ks * 2) == 0 && K / (ks * 2) >= 2 * BK) ks *= 2;
  return ks;
}

}  // namespace fovea
