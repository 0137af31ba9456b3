// Host side of the C ABI declared in include/fovea.h: argument validation, the
// context with its packed weights, the workspace layout and the launch sequence.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "fovea.h"
#include "backward_kernels.hpp"
#include "correct_kernels.hpp"
#include "lm_kernels.hpp"
#include "retrieve_kernels.hpp"

using namespace fovea;

static_assert(FOVEA_MAX_M == kMaxM && FOVEA_MAX_KMAX == kMaxKmax, "header limits");
static_assert(FOVEA_DATA_BAD_NODE_OFFSETS == kErrNodeOff && FOVEA_DATA_BAD_MEM_OFFSETS == kErrMemOff &&
                  FOVEA_DATA_BAD_DEPTH == kErrDepth && FOVEA_DATA_BAD_TAU == kErrTau &&
                  FOVEA_DATA_BAD_SELECTION == kErrSelection,
              "error bits");
static_assert(FOVEA_LM_MAX_K == kLmMaxK && FOVEA_LM_MAX_VOCAB == kLmMaxVocab &&
                  FOVEA_LM_MAX_ROWS == kLmMaxRows,
              "header limits");

struct fovea_ctx {
  fovea_dims dims;
  int device;
  bool bf16;
  size_t es;  // bytes per stored element
  void* block;  // one allocation holding every packed array below
  float* q_c1;  // [d_m] row sums of the folded W_Q
  float* q_c2;  // [n_depth, d_m] W_Q (q_ln_b + E_dep[l])
  void* W_KU;   // [2 d_m, d_v] [W_K ; W_U] diag(mem_ln_g)
  float* m_c1;  // [2 d_m]
  float* m_c2;  // [2 d_m] [W_K ; W_U] mem_ln_b
  void* W_hq;   // [d_m + 2 d_c, d] [W_Q diag(q_ln_g) ; W_c1[:, :d] ; W_g1[:, :d]]
  void* W1r;    // [2 d_c, d_m]    [W_c1[:, d:] ; W_g1[:, d:]]
  float* b1;    // [2 d_c]
  void* W_c2;   // [d, d_c]
  float* b_c2;  // [d]
  float* w_g2;  // [d_c]
  float b_g2;
  float* rms_w;  // [d] or null
  uint32_t* err;  // sticky device-data error bits
  void* scratch;  // device address of this device's no-allocation workspace
  size_t lds_limit[5];  // dynamic LDS limit of each LdsKernel
  // one completion event per stream that calls have enqueued work on: fovea_destroy
  // waits for these (not for the whole device) before it frees the packed weights
  struct StreamUse {
    hipStream_t stream;
    hipEvent_t done;
  };
  std::vector<StreamUse> uses;
  // diagnostics: HIP event pairs around each launched kernel
  bool prof;
  struct ProfRec {
    int slot;
    hipEvent_t e0, e1;
  };
  std::vector<ProfRec> prof_recs;
  std::vector<hipEvent_t> prof_pool;
};

// kernels whose dynamic LDS limit the context sets (raise_lds_limits)
enum LdsKernel { kLdsSelBf16, kLdsSelF32, kLdsBwdMem, kLdsBwdSelFwd, kLdsBwdSel, kNumLdsKernels };

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  if (a == nullptr || b == nullptr || na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

// Byte offsets of the retrieve_fuse workspace regions.
// k-sliced scores (score_parts): batches of at most kScoreSplitNodes nodes may split
// the score GEMM's d_m into up to kScoreMaxParts slices
constexpr int kScoreSplitNodes = 256;

struct WsLayout {
  size_t node_req, info, stats, q, P, S, rT, a_c, gate_part, rms_part, splitk, total;
};

// K slices of the three forward GEMMs (hidden-state GEMM, layer 1, layer 2) at n rows
struct SplitK {
  int hq, c1, c2;
};

SplitK forward_splitk(const fovea_dims& D, int64_t n) {
  const int bk = D.dtype == FOVEA_BF16 ? 64 : 32;
  const int ni = static_cast<int>(n);
  SplitK k;
  // at most 8 slices (one request: 16 slices of 256 columns 56.0 -> 8 of 512 53.8 us per
  // step, the combine reading half the partials); the combine merges the slices' LayerNorm
  // statistics in registers (at most kHqMaxKs)
  static_assert(kHqMaxKs >= 8, "query GEMM slices");
  k.hq = std::min(splitk_slices(((ni + 127) / 128) * ((D.d_m + 2 * D.d_c + 127) / 128), D.d, bk), 8);
  k.c1 = splitk_slices(((ni + 63) / 64) * ((2 * D.d_c + 127) / 128), D.d_m, bk);
  k.c2 = splitk_slices(((ni + 127) / 128) * ((D.d + 127) / 128), D.d_c, bk);
  return k;
}

WsLayout ws_layout(const fovea_dims& dm, int64_t n, int64_t m_max) {
  const size_t es = dm.dtype == FOVEA_BF16 ? 2 : 4;
  WsLayout L;
  size_t o = 0;
  L.node_req = o; o = align_up(o + n * 4);
  L.info = o; o = align_up(o + n * sizeof(NodeInfo));
  // LayerNorm statistics: (mean, rstd) per node, or with a split-K query GEMM the
  // slices' (mean, M2) per node
  L.stats = o; o = align_up(o + std::max(1, forward_splitk(dm, n).hq) * n * 8);
  L.q = o; o = align_up(o + n * dm.d_m * (dm.dtype == FOVEA_BF16 ? 2 * kQSplitBf16 : 4));
  L.P = o; o = align_up(o + n * 2 * dm.d_c * 4);
  // scores; small bf16 batches may hold k-sliced partial scores (score_parts)
  const int64_t s_arrays = dm.dtype == FOVEA_BF16 && n <= kScoreSplitNodes ? kScoreMaxParts : 1;
  L.S = o; o = align_up(o + s_arrays * n * m_max * 4);
  L.rT = o; o = align_up(o + n * dm.d_m * es);
  L.a_c = o; o = align_up(o + n * dm.d_c * es);
  L.gate_part = o; o = align_up(o + n * n_parts(2 * dm.d_c) * 4);
  L.rms_part = o; o = align_up(o + n * n_parts(dm.d) * 4);
  {
    const SplitK k = forward_splitk(dm, n);
    size_t need = 0;
    if (k.hq > 1) need = std::max(need, static_cast<size_t>(k.hq) * n * (dm.d_m + 2 * dm.d_c));
    if (k.c1 > 1) need = std::max(need, static_cast<size_t>(k.c1) * n * 2 * dm.d_c);
    if (k.c2 > 1) need = std::max(need, static_cast<size_t>(k.c2) * n * dm.d);
    L.splitk = o; o = align_up(o + need * 4);
  }
  L.total = o;
  return L;
}

bool dims_ok(const fovea_dims* d) {
  if (d == nullptr) return false;
  if (d->dtype != FOVEA_F32 && d->dtype != FOVEA_BF16) return false;
  if (d->d <= 0 || d->d_v <= 0 || d->d_m <= 0 || d->d_c <= 0 || d->n_depth <= 0) return false;
  if (!(d->ln_eps >= 0.f) || !(d->rms_eps >= 0.f) || !std::isfinite(d->ln_eps) ||
      !std::isfinite(d->rms_eps))
    return false;
  return true;
}

bool dims_supported(const fovea_dims* d) {
  return d->d % 64 == 0 && d->d_v % 64 == 0 && d->d_m % 64 == 0 && d->d_c % 64 == 0 &&
         d->d <= (1 << 20) && d->d_v <= (1 << 20) && d->d_m <= (1 << 16) && d->d_c <= (1 << 16);
}

#define FOVEA_HIP(call)                                   \
  do {                                                    \
    if ((call) != hipSuccess) return FOVEA_ERR_DEVICE;    \
  } while (0)

enum KernelSlot {
  kRowStats, kHq, kScore, kSelect, kCorr1, kCorr2, kRms, kMemStats, kMemProj, kLmHead, kLmMerge,
  kBwdFill, kBwdStats, kBwdTranspose, kBwdPrep, kBwdGemm, kBwdSelFwd, kBwdRmsGate, kBwdSel,
  kBwdLn, kBwdReduce, kBwdMem, kNumSlots
};
const char* const kSlotNames[kNumSlots] = {
    "row_stats",     "hq",           "score",       "select_gather", "corr1",
    "corr2",         "rms",          "mem_row_stats", "mem_proj",    "lm_head",
    "lm_merge",      "bwd_fill",     "bwd_stats",   "bwd_transpose", "bwd_prep",
    "bwd_gemm",      "bwd_sel_fwd",  "bwd_rms_gate", "bwd_sel",      "bwd_ln",
    "bwd_reduce",    "bwd_memory"};

hipEvent_t prof_event(fovea_ctx* c) {
  if (!c->prof_pool.empty()) {
    hipEvent_t e = c->prof_pool.back();
    c->prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Brackets one kernel launch with events when profiling is on.
struct ProfScope {
  fovea_ctx* c;
  int slot;
  hipStream_t s;
  hipEvent_t e0 = nullptr;
  // c_ == nullptr: no events (the no-allocation entry point creates none)
  ProfScope(fovea_ctx* c_, int slot_, hipStream_t s_) : c(c_), slot(slot_), s(s_) {
    if (c != nullptr && c->prof && (e0 = prof_event(c)) != nullptr) (void)hipEventRecord(e0, s);
  }
  ~ProfScope() {
    if (e0 == nullptr) return;
    hipEvent_t e1 = prof_event(c);
    if (e1 == nullptr) {
      c->prof_pool.push_back(e0);
      return;
    }
    (void)hipEventRecord(e1, s);
    c->prof_recs.push_back({slot, e0, e1});
  }
};

// Marks the end of a call's work on `s` (the event of that stream is re-recorded).
fovea_status record_use(fovea_ctx* c, hipStream_t s) {
  for (auto& u : c->uses)
    if (u.stream == s) return hipEventRecord(u.done, s) == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return FOVEA_ERR_DEVICE;
  c->uses.push_back({s, e});
  return hipEventRecord(e, s) == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
}

// Kernels launched with a large dynamic LDS: their limit is set once, in fovea_create,
// to what the compute unit's 160 KB leaves beside the kernel's static LDS, and kept in
// the context for each launch to check its own size against.
constexpr int kLdsBytes = 160 * 1024;

fovea_status raise_lds_limits(fovea_ctx* c) {
  const void* kernels[kNumLdsKernels] = {
      reinterpret_cast<const void*>(select_gather_kernel<bf16_t>),
      reinterpret_cast<const void*>(select_gather_kernel<float>),
      reinterpret_cast<const void*>(bwd_mem_grad_kernel),
      reinterpret_cast<const void*>(bwd_sel_fwd_kernel),
      reinterpret_cast<const void*>(bwd_sel_kernel)};
  for (int i = 0; i < kNumLdsKernels; ++i) {
    hipFuncAttributes at;
    FOVEA_HIP(hipFuncGetAttributes(&at, kernels[i]));
    const int limit = kLdsBytes - static_cast<int>(at.sharedSizeBytes);
    if (limit <= 0) return FOVEA_ERR_DEVICE;
    FOVEA_HIP(hipFuncSetAttribute(kernels[i], hipFuncAttributeMaxDynamicSharedMemorySize, limit));
    c->lds_limit[i] = static_cast<size_t>(limit);
  }
  return FOVEA_OK;
}

template <typename T>
fovea_status pack_weights(fovea_ctx* c, const fovea_params* p, hipStream_t s) {
  const fovea_dims& D = c->dims;
  const int d = D.d, d_v = D.d_v, d_m = D.d_m, d_c = D.d_c;
  auto T_ = [](const void* x) { return static_cast<const T*>(x); };
  // folded projections
  hipLaunchKernelGGL(fold_gain_kernel<T>, dim3(1024), dim3(256), 0, s, T_(p->W_Q), T_(p->q_ln_g),
                     static_cast<int64_t>(d_m), d, static_cast<T*>(c->W_hq));
  hipLaunchKernelGGL(fold_gain_kernel<T>, dim3(1024), dim3(256), 0, s, T_(p->W_K), T_(p->mem_ln_g),
                     static_cast<int64_t>(d_m), d_v, static_cast<T*>(c->W_KU));
  hipLaunchKernelGGL(fold_gain_kernel<T>, dim3(1024), dim3(256), 0, s, T_(p->W_U), T_(p->mem_ln_g),
                     static_cast<int64_t>(d_m), d_v, static_cast<T*>(c->W_KU) + static_cast<int64_t>(d_m) * d_v);
  // row sums of the folded weights and the bias / depth terms
  auto rows = [](int items) { return dim3((items + 3) / 4); };
  hipLaunchKernelGGL(row_dot_kernel<T>, rows(d_m), dim3(256), 0, s, static_cast<const T*>(c->W_hq),
                     d_m, d, static_cast<const T*>(nullptr), static_cast<const T*>(nullptr), 1, c->q_c1);
  hipLaunchKernelGGL(row_dot_kernel<T>, rows(d_m * D.n_depth), dim3(256), 0, s, T_(p->W_Q), d_m, d,
                     T_(p->q_ln_b), T_(p->E_dep), D.n_depth, c->q_c2);
  hipLaunchKernelGGL(row_dot_kernel<T>, rows(2 * d_m), dim3(256), 0, s, static_cast<const T*>(c->W_KU),
                     2 * d_m, d_v, static_cast<const T*>(nullptr), static_cast<const T*>(nullptr), 1, c->m_c1);
  hipLaunchKernelGGL(row_dot_kernel<T>, rows(d_m), dim3(256), 0, s, T_(p->W_K), d_m, d_v,
                     T_(p->mem_ln_b), static_cast<const T*>(nullptr), 1, c->m_c2);
  hipLaunchKernelGGL(row_dot_kernel<T>, rows(d_m), dim3(256), 0, s, T_(p->W_U), d_m, d_v,
                     T_(p->mem_ln_b), static_cast<const T*>(nullptr), 1, c->m_c2 + d_m);
  // correction / gate nets
  const size_t es = sizeof(T);
  // first layer of both nets split by input: the h half joins W_Q in the hidden-state
  // GEMM, the r half is its own GEMM
  const size_t src_pitch = static_cast<size_t>(d + d_m) * es;
  char* hq_rows = static_cast<char*>(c->W_hq) + static_cast<size_t>(d_m) * d * es;
  FOVEA_HIP(hipMemcpy2DAsync(hq_rows, d * es, p->W_c1, src_pitch, d * es, d_c, hipMemcpyDeviceToDevice, s));
  FOVEA_HIP(hipMemcpy2DAsync(hq_rows + static_cast<size_t>(d_c) * d * es, d * es, p->W_g1, src_pitch,
                             d * es, d_c, hipMemcpyDeviceToDevice, s));
  FOVEA_HIP(hipMemcpy2DAsync(c->W1r, d_m * es, static_cast<const char*>(p->W_c1) + d * es, src_pitch,
                             d_m * es, d_c, hipMemcpyDeviceToDevice, s));
  FOVEA_HIP(hipMemcpy2DAsync(static_cast<char*>(c->W1r) + static_cast<size_t>(d_c) * d_m * es,
                             d_m * es, static_cast<const char*>(p->W_g1) + d * es, src_pitch,
                             d_m * es, d_c, hipMemcpyDeviceToDevice, s));
  FOVEA_HIP(hipMemcpyAsync(c->W_c2, p->W_c2, static_cast<size_t>(d) * d_c * es,
                           hipMemcpyDeviceToDevice, s));
  hipLaunchKernelGGL(to_f32_kernel<T>, dim3(8), dim3(256), 0, s, T_(p->b_c1), d_c, c->b1);
  hipLaunchKernelGGL(to_f32_kernel<T>, dim3(8), dim3(256), 0, s, T_(p->b_g1), d_c, c->b1 + d_c);
  hipLaunchKernelGGL(to_f32_kernel<T>, dim3(64), dim3(256), 0, s, T_(p->b_c2), d, c->b_c2);
  hipLaunchKernelGGL(to_f32_kernel<T>, dim3(8), dim3(256), 0, s, T_(p->w_g2), d_c, c->w_g2);
  if (c->rms_w)
    hipLaunchKernelGGL(to_f32_kernel<T>, dim3(64), dim3(256), 0, s, T_(p->rms_w), d, c->rms_w);
  FOVEA_HIP(hipGetLastError());
  return FOVEA_OK;
}

template <typename T>
fovea_status run_build(fovea_ctx* c, int n, const void* V, void* keys, void* values,
                       float2* build_stats, hipStream_t s) {
  const fovea_dims& D = c->dims;
  {
    ProfScope ps(c, kMemStats, s);
    hipLaunchKernelGGL(row_stats_kernel<T>, dim3((n + 3) / 4), dim3(256), 0, s, n,
                       static_cast<const T*>(V), D.d_v, D.ln_eps, build_stats,
                       static_cast<const int32_t*>(nullptr), 0, static_cast<const int32_t*>(nullptr),
                       0, 0, static_cast<const float*>(nullptr),
                       static_cast<const int64_t*>(nullptr), int64_t{0}, 0,
                       static_cast<int32_t*>(nullptr), static_cast<NodeInfo*>(nullptr), c->err);
  }
  // 256-row tiles once the grid still holds at least 256 of them (bf16 only)
  const bool tall = std::is_same<T, bf16_t>::value &&
                    static_cast<int64_t>((n + 255) / 256) * ((2 * D.d_m + 127) / 128) >= 256;
  const int BMv = tall ? 256 : 128;
  const TileMap tm = make_tile_map((n + BMv - 1) / BMv, (2 * D.d_m + 127) / 128,
                                   static_cast<double>(n) * D.d_v, 2.0 * D.d_m * D.d_v);
  {
    ProfScope ps(c, kMemProj, s);
    hipLaunchKernelGGL((tall ? mem_proj_kernel<T, 256> : mem_proj_kernel<T, 128>), dim3(tile_grid(tm)),
                       dim3(256), 0, s, tm, n, static_cast<const T*>(V), D.d_v,
                       static_cast<const T*>(c->W_KU), D.d_m, build_stats, c->m_c1, c->m_c2,
                       static_cast<T*>(keys), static_cast<T*>(values));
  }
  FOVEA_HIP(hipGetLastError());
  return FOVEA_OK;
}

struct RFArgs {
  int B;
  const int64_t* mem_off;
  int64_t n_mem;
  int m_max;
  const void* keys;
  const void* values;
  const uint8_t* valid;
  const int32_t* node_off;
  int n;
  int t_max;
  const void* h;
  const int32_t* depth;
  const float* tau;
  int k_min, k_max;
  void* h_out;
  int32_t* k_out;
  int32_t* idx_out;
  float* gate_out;
  float* mass_out;
  float* r_out;
  char* ws;
  bool track;  // profiling events and the per-stream completion event (false: create none)
};

// Keys per score block: 16 kb, kb in {1, 2, 4, 5, 6}, whichever spreads B * tiles blocks
// over the 256 compute units in the fewest waves of work per unit.  A block streams its
// keys (32 kb d_m bytes) and its 64 nodes' two q planes (256 d_m bytes), so the work of
// one block counts as kb + 8 units (few large blocks win at large B, many small blocks
// at small B).
int score_keys_per_block(int B, int m_max) {
  static const int kbs[] = {1, 2, 4, 5, 6};
  int best = 4;
  long best_cost = -1;
  for (int kb : kbs) {
    const long blocks = static_cast<long>(B) * ((m_max + 16 * kb - 1) / (16 * kb));
    const long cost = ((blocks + 255) / 256) * (kb + 8);
    if (best_cost < 0 || cost < best_cost) {
      best_cost = cost;
      best = kb;
    }
  }
  return 16 * best;
}

typedef void (*ScoreKernel)(int, const int64_t*, int64_t, int, const int32_t*, int, int,
                            const bf16_t*, int, const bf16_t*, float, float*, int, int);

template <int NKC>
ScoreKernel score_kernel_kb(int kb) {
  switch (kb) {
    case 1: return score_bf16_kernel<NKC, 1>;
    case 2: return score_bf16_kernel<NKC, 2>;
    case 5: return score_bf16_kernel<NKC, 5>;
    case 6: return score_bf16_kernel<NKC, 6>;
    default: return score_bf16_kernel<NKC, 4>;
  }
}

ScoreKernel score_kernel_for(int nkc, int kb) {
  switch (nkc) {
    case 4: return score_kernel_kb<4>(kb);
    case 8: return score_kernel_kb<8>(kb);
    case 12: return score_kernel_kb<12>(kb);
    case 14: return score_kernel_kb<14>(kb);
    case 16: return score_kernel_kb<16>(kb);
    case 20: return score_kernel_kb<20>(kb);
    case 24: return score_kernel_kb<24>(kb);
    case 64: return score_kernel_kb<64>(kb);
    default: return score_bf16_any_kernel;
  }
}

// k slices of the bf16 score GEMM.  A small batch's score grid leaves most compute units
// idle while each block streams all of its nodes' q (256 d_m bytes), so d_m is cut into
// 2 or 4 slices (each an instantiated chunk count) whose partial scores the selection
// adds in order.  Only batches of at most kScoreSplitNodes nodes, for which the
// workspace holds kScoreMaxParts score arrays.

int score_parts(const fovea_dims& D, int B, int n, int m_max, int t_max) {
  if (D.dtype != FOVEA_BF16 || n > kScoreSplitNodes || m_max == 0 || t_max == 0) return 1;
  const int kb = score_keys_per_block(B, m_max) / 16;
  const int64_t blocks = static_cast<int64_t>(B) * ((m_max + 16 * kb - 1) / (16 * kb)) *
                         ((t_max + 63) / 64);
  const int nkc = D.d_m / score_cfg::KC;
  int best = 1;
  for (int p = 2; p <= kScoreMaxParts; p *= 2)
    if (nkc % p == 0 && blocks * p <= 256 && score_kernel_for(nkc / p, kb) != score_bf16_any_kernel)
      best = p;
  return best;
}

template <typename T>
fovea_status run_retrieve_fuse(fovea_ctx* c, const RFArgs& a, hipStream_t s) {
  const fovea_dims& D = c->dims;
  fovea_ctx* const pc = a.track ? c : nullptr;  // profiling context, if any
  const WsLayout L = ws_layout(D, a.n, a.m_max);
  const SplitK ksp = forward_splitk(D, a.n);
  float* splitk = reinterpret_cast<float*>(a.ws + L.splitk);
  int32_t* node_req = reinterpret_cast<int32_t*>(a.ws + L.node_req);
  NodeInfo* info = reinterpret_cast<NodeInfo*>(a.ws + L.info);
  float2* stats = reinterpret_cast<float2*>(a.ws + L.stats);
  T* q = reinterpret_cast<T*>(a.ws + L.q);
  float* P = reinterpret_cast<float*>(a.ws + L.P);
  float* S = reinterpret_cast<float*>(a.ws + L.S);
  const int s_parts = score_parts(D, a.B, a.n, a.m_max, a.t_max);
  T* rT = reinterpret_cast<T*>(a.ws + L.rT);
  T* a_c = reinterpret_cast<T*>(a.ws + L.a_c);
  float* gate_part = reinterpret_cast<float*>(a.ws + L.gate_part);
  float* rms_part = reinterpret_cast<float*>(a.ws + L.rms_part);
  const T* h = static_cast<const T*>(a.h);

  // 1. LayerNorm statistics of h, node -> request map, depth / tau / offset checks (with
  // a split-K query GEMM its slices and its combine do this, without a launch of its own)
  const bool split_stats = ksp.hq > 1;
  if (!split_stats) {
    ProfScope ps(pc, kRowStats, s);
    hipLaunchKernelGGL(row_stats_kernel<T>, dim3((a.n + 3) / 4), dim3(256), 0, s, a.n, h, D.d,
                       D.ln_eps, stats, a.depth, D.n_depth, a.node_off, a.B, a.t_max, a.tau,
                       a.mem_off, a.n_mem, a.m_max, node_req, info, c->err);
  }
  // 2. everything that depends on h alone: q = W_Q (LN(h) + E_dep[l]) and P = h W1h^T
  {
    using C = HqCfg<T>;
    const int N = D.d_m + 2 * D.d_c;
    const TileMap tm = make_tile_map((a.n + C::BM - 1) / C::BM, (N + C::BN - 1) / C::BN,
                                     static_cast<double>(a.n) * D.d, static_cast<double>(N) * D.d);
    HqEpi<T> epi;
    epi.n = a.n;
    epi.d_m = D.d_m;
    epi.N = N;
    epi.n_depth = D.n_depth;
    epi.n_p = 2 * D.d_c;
    epi.stats = stats;
    epi.depth = a.depth;
    epi.node_req = node_req;
    epi.c1 = c->q_c1;
    epi.c2 = c->q_c2;
    epi.q = q;
    epi.P = P;
    const int ks = ksp.hq;
    ProfScope ps(pc, kHq, s);
    // at most 64 rows: the same single row of tiles in 64-row tiles (no clamped rows)
    float2* stat_part = split_stats ? stats : nullptr;
    NodeMapArgs nm;
    {
      nm.node_off = a.node_off;
      nm.B = a.B;
      nm.t_max = a.t_max;
      nm.n = a.n;
      nm.depth = a.depth;
      nm.n_depth = D.n_depth;
      nm.tau = a.tau;
      nm.mem_off = a.mem_off;
      nm.n_mem = a.n_mem;
      nm.m_max = a.m_max;
      nm.node_req = node_req;
      nm.info = info;
      nm.err = c->err;
    }
    hipLaunchKernelGGL((a.n <= 64 ? hq_kernel<T, 64> : hq_kernel<T>), dim3(tile_grid(tm), ks),
                       dim3(C::NT), 0, s, tm, a.n, h, D.d, static_cast<const T*>(c->W_hq), epi, ks, splitk,
                       stat_part, nm);
    if (ks > 1)
      hipLaunchKernelGGL(hq_combine_kernel<T>, dim3((N + 127) / 128, (a.n + 15) / 16), dim3(256), 0, s,
                         epi, ks, static_cast<const float*>(splitk),
                         static_cast<const float2*>(stat_part), D.d, D.ln_eps);
  }
  // 3. scores for every (node, key) of each request
  if (a.m_max > 0) {
    const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(D.d_m)));
    ProfScope ps(pc, kScore, s);
    if constexpr (std::is_same<T, bf16_t>::value) {
      const int kb = score_keys_per_block(a.B, a.m_max) / 16;
      const int tiles = (a.m_max + 16 * kb - 1) / (16 * kb);
      auto kern = score_kernel_for(D.d_m / score_cfg::KC / s_parts, kb);
      const int nch = (a.t_max + 63) / 64;
      // ragged memories (their total well below B m_max): spread the tiles over the XCDs
      const int spread = a.n_mem * 4 < static_cast<int64_t>(a.B) * a.m_max * 3 ? 1 : 0;
      const int grid = xcd_grid(kern == score_bf16_any_kernel ? a.B * ((a.m_max + 63) / 64)
                                                              : a.B * tiles * nch * s_parts);
      hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, s, a.B, a.mem_off, a.n_mem, a.m_max,
                         a.node_off, a.n, a.t_max, static_cast<const bf16_t*>(a.keys), D.d_m,
                         reinterpret_cast<const bf16_t*>(q), scale, S, s_parts, spread);
    } else {
      const int tiles = (a.m_max + 63) / 64;
      hipLaunchKernelGGL(score_f32_kernel, dim3(xcd_grid(a.B * tiles)), dim3(256), 0, s, a.B,
                         a.mem_off, a.n_mem, a.m_max, a.node_off, a.n, a.t_max,
                         static_cast<const float*>(a.keys), D.d_m, reinterpret_cast<const float*>(q),
                         scale, S);
    }
  }
  // 4. selection and gather, one block per node
  SelectArgs<T> sa;
  sa.mem_off = a.mem_off;
  sa.n_mem = a.n_mem;
  sa.m_max = a.m_max;
  sa.node_req = node_req;
  sa.info = info;
  sa.tau = a.tau;
  sa.valid = a.valid;
  sa.values = static_cast<const T*>(a.values);
  sa.d_m = D.d_m;
  sa.S = S;
  sa.s_parts = s_parts;
  sa.s_stride = static_cast<int64_t>(a.n) * a.m_max;
  sa.k_min = a.k_min;
  sa.k_max = a.k_max;
  sa.rT = rT;
  sa.r_out = a.r_out;
  sa.k_out = a.k_out;
  sa.idx_out = a.idx_out;
  sa.mass_out = a.mass_out;
  sa.err = c->err;
  {
    ProfScope ps(pc, kSelect, s);
    const int VEC = D.dtype == FOVEA_BF16 ? 8 : 4;
    const int nch = (D.d_m / VEC + 63) / 64;  // 16-byte chunks per lane per value row
    // one wave selects a node of at most 1024 entries (16 keys per lane); larger memories
    // go to the block-wide kernel, whose radix threshold and counting rank use all four
    // waves (ragged Qwen workload, memories of up to 4096: 98.6 -> 41.4 us)
    const bool wave_path = a.k_max <= kWaveSelKmax && a.m_max <= 1024 && nch <= 4;
    if (wave_path) {
      // one node per block when the pairs would leave compute units idle: the gather of a
      // node then runs on four waves instead of two
      const bool one = (a.n + 1) / 2 < 256;
      const dim3 grid(xcd_grid(one ? a.n : (a.n + 1) / 2)), blk(256);
      const int npl = (a.m_max + 63) / 64;
#define FOVEA_SEL_C(N, C)                                                              \
  if (one)                                                                             \
    hipLaunchKernelGGL((select_node_kernel<T, N, C, 1>), grid, blk, 0, s, sa, a.n);    \
  else                                                                                 \
    hipLaunchKernelGGL((select_node_kernel<T, N, C, 2>), grid, blk, 0, s, sa, a.n)
#define FOVEA_SEL(N)              \
  if (nch <= 1) FOVEA_SEL_C(N, 1); \
  else if (nch <= 2) FOVEA_SEL_C(N, 2); \
  else FOVEA_SEL_C(N, 4)
      if (npl <= 1) { FOVEA_SEL(1); }
      else if (npl <= 2) { FOVEA_SEL(2); }
      else if (npl <= 4) { FOVEA_SEL(4); }
      else if (npl <= 6) { FOVEA_SEL(6); }
      else if (npl <= 9) { FOVEA_SEL(9); }
      else if (npl <= 12) { FOVEA_SEL(12); }
      else { FOVEA_SEL(16); }
#undef FOVEA_SEL
#undef FOVEA_SEL_C
    } else {
      // the order keys (later the gather's partial sums) and the candidate arrays
      const size_t sel_smem = static_cast<size_t>(select_gather_smem(a.m_max, a.k_max, VEC));
      if (sel_smem > c->lds_limit[std::is_same<T, bf16_t>::value ? kLdsSelBf16 : kLdsSelF32])
        return FOVEA_ERR_UNSUPPORTED;
      // few nodes: each node's row is also split into column slices over several blocks
      // (each repeats the selection) so that the gathers run on more compute units
      const int cpr64 = (D.d_m / VEC + 63) / 64;
      const int slices = std::max(1, std::min(cpr64, 512 / std::max(a.n, 1)));
      hipLaunchKernelGGL(select_gather_kernel<T>, dim3(a.n, slices), dim3(256), sel_smem, s, sa);
    }
  }
  // 5. correction layer 1: the r half, plus P, bias and SiLU (+ gate logit partials)
  {
    using C = Corr1Cfg<T>;
    const TileMap tm = make_tile_map((a.n + C::BM - 1) / C::BM, (2 * D.d_c + C::BN - 1) / C::BN,
                                     static_cast<double>(a.n) * D.d_m, 2.0 * D.d_c * D.d_m);
    Corr1Epi<T> epi;
    epi.n = a.n;
    epi.d_c = D.d_c;
    epi.N = 2 * D.d_c;
    epi.P = P;
    epi.b1 = c->b1;
    epi.w_g2 = c->w_g2;
    epi.a_c = a_c;
    ProfScope ps(pc, kCorr1, s);
    hipLaunchKernelGGL(corr1_kernel<T>, dim3(tile_grid(tm), ksp.c1), dim3(C::NT), 0, s, tm, rT, D.d_m,
                       static_cast<const T*>(c->W1r), epi, gate_part, ksp.c1, splitk);
    if (ksp.c1 > 1)
      hipLaunchKernelGGL(corr1_combine_kernel<T>, dim3((epi.N + 127) / 128, (a.n + 15) / 16), dim3(256), 0,
                         s, epi, gate_part, ksp.c1, static_cast<const float*>(splitk));
  }
  // 6. correction layer 2, gate, residual (+ RMS partials)
  T* h_out = static_cast<T*>(a.h_out);
  bool fused_rms = false;
  {
    using C = Corr2Cfg<T>;
    const TileMap tm = make_tile_map((a.n + C::BM - 1) / C::BM, (D.d + C::BN - 1) / C::BN,
                                     static_cast<double>(a.n) * D.d_c, static_cast<double>(D.d) * D.d_c);
    Corr2Epi<T> epi;
    epi.n = a.n;
    epi.d = D.d;
    epi.b_c2 = c->b_c2;
    epi.h = h;
    epi.h_out = h_out;
    epi.sg = nullptr;
    epi.m0 = 0;
    Corr2Args ca;
    ca.d_c = D.d_c;
    ca.gate_part = gate_part;
    ca.b_g2 = c->b_g2;
    ca.gate_out = a.gate_out;
    ca.rms_part = c->rms_w ? rms_part : nullptr;
    // split-K with the RMSNorm: the slices' sum, the residual and the norm in one pass
    fused_rms = ksp.c2 > 1 && c->rms_w != nullptr && D.d <= kCorr2RmsMaxD;
    {
      ProfScope ps(pc, kCorr2, s);
      hipLaunchKernelGGL((a.n <= 64 ? corr2_kernel<T, 64> : corr2_kernel<T>), dim3(tile_grid(tm), ksp.c2),
                         dim3(C::NT), 0, s, tm, a_c, static_cast<const T*>(c->W_c2), epi, ca, ksp.c2,
                         splitk);
      if (ksp.c2 > 1 && !fused_rms)
        hipLaunchKernelGGL(corr2_combine_kernel<T>, dim3((D.d + 127) / 128, (a.n + 15) / 16), dim3(256), 0, s,
                           epi, ca, ksp.c2, static_cast<const float*>(splitk));
    }
    if (fused_rms) {
      ProfScope ps(pc, kRms, s);
      hipLaunchKernelGGL(corr2_rms_kernel<T>, dim3(a.n), dim3(256), 0, s, epi, ca, ksp.c2,
                         static_cast<const float*>(splitk), c->rms_w, D.rms_eps);
    }
  }
  // 7. RMSNorm
  if (c->rms_w && !fused_rms) {
    ProfScope ps(pc, kRms, s);
    hipLaunchKernelGGL(rms_kernel<T>, dim3((a.n + 3) / 4), dim3(256), 0, s, a.n, D.d, rms_part, c->rms_w,
                       D.rms_eps, h_out);
  }
  FOVEA_HIP(hipGetLastError());
  return FOVEA_OK;
}

size_t lm_cand_bytes(int n, int vocab, int k) {
  const size_t cb = (static_cast<size_t>(vocab) + 127) / 128;
  return align_up(static_cast<size_t>(n) * cb * k * sizeof(uint64_t));
}

template <typename T, int BM>
void launch_lm(int n, const T* h, int d, const T* W, int vocab, int k, uint64_t* cand,
               hipStream_t s) {
  const LmMap m = make_lm_map((n + BM - 1) / BM, (vocab + 127) / 128);
  hipLaunchKernelGGL((lm_kernel<T, BM>), dim3(lm_grid(m)), dim3(256), 0, s, m, n, h, d, W, vocab,
                     k, cand);
}

template <typename T>
fovea_status run_lm_topk(fovea_ctx* c, int n, const void* h, const void* W, int vocab, int k,
                         int32_t* idx, float* logit, uint64_t* cand, hipStream_t s) {
  const int d = c->dims.d;
  {
    ProfScope ps(c, kLmHead, s);
    // row tiles: 64 for one small batch, 256 for many rows (half the operand bytes per
    // MAC of a 128-row tile), 128 between
    if (n <= 64)
      launch_lm<T, 64>(n, static_cast<const T*>(h), d, static_cast<const T*>(W), vocab, k, cand, s);
    else if (n < 768)
      launch_lm<T, 128>(n, static_cast<const T*>(h), d, static_cast<const T*>(W), vocab, k, cand, s);
    else
      launch_lm<T, 256>(n, static_cast<const T*>(h), d, static_cast<const T*>(W), vocab, k, cand, s);
  }
  {
    const int n_cand = (vocab + 127) / 128 * k;
    ProfScope ps(c, kLmMerge, s);
    if (k <= 8)
      hipLaunchKernelGGL(lm_merge_kernel<8>, dim3(n), dim3(256), 0, s, n_cand, k, cand, idx, logit);
    else
      hipLaunchKernelGGL(lm_merge_kernel<kLmMaxK>, dim3(n), dim3(256), 0, s, n_cand, k, cand, idx,
                         logit);
  }
  return hipGetLastError() == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
}

// ---------------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------------

struct BwdLayout {
  int npad;
  size_t node_req, info, stats, tau0, ok, dlogit;
  size_t xhat, xe, y, q, alpha, z, a, c, hn, dc, dz, dr, dq, dxe, wa, wsel;
  size_t part, sa, sb;
  size_t total;
};

BwdLayout bwd_layout(const fovea_dims& D, int B, int n, int k_max, int m_max) {
  BwdLayout L;
  const size_t d = D.d, dm = D.d_m, dc = D.d_c, nn = n;
  const size_t np = (nn + 63) / 64 * 64;
  L.npad = static_cast<int>(np);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L.node_req = take(nn * 4);
  L.info = take(nn * sizeof(NodeInfo));
  L.stats = take(nn * 8);
  L.tau0 = take(static_cast<size_t>(B) * 4);
  L.ok = take(nn * 4);
  L.dlogit = take(np * 4);
  L.xhat = take(nn * d * 4);
  L.xe = take(nn * d * 4);
  L.y = take(nn * (d + dm) * 4);
  L.q = take(nn * dm * 4);
  L.alpha = take(nn * static_cast<size_t>(k_max) * 4);
  L.z = take(nn * 2 * dc * 4);
  L.a = take(nn * 2 * dc * 4);
  L.c = take(nn * d * 4);
  L.hn = take(nn * d * 4);
  L.dc = take(nn * d * 4);
  L.dz = take(nn * 2 * dc * 4);
  L.dr = take(nn * dm * 4);
  L.dq = take(nn * dm * 4);
  L.dxe = take(nn * d * 4);
  L.wa = take(nn * static_cast<size_t>(m_max) * 4);
  L.wsel = take(nn * static_cast<size_t>(m_max) * 4);
  // column-sum partials: b_c2, b_c1, b_g1, w_g2 and rms_w one slot each; dxe two plus
  // one per depth
  L.part = take(static_cast<size_t>(kColChunks) * (d * (D.n_depth + 4) + 3 * dc) * 4);
  // bf16 planes of the largest A and B operand of the backward's GEMMs ([rows, 3 K])
  const size_t mk[] = {nn * d, nn * (d + dm), nn * dc, nn * 2 * dc, nn * dm, d * np, 2 * dc * np, dm * np};
  const size_t nk[] = {dm * d, 2 * dc * (d + dm), d * dc, dc * d, (d + dm) * 2 * dc, d * dm,
                       dc * np, (d + dm) * np, d * np};
  size_t ma = 0, mb = 0;
  for (size_t v : mk) ma = std::max(ma, v);
  for (size_t v : nk) mb = std::max(mb, v);
  L.sa = take(ma * 3 * 2);
  L.sb = take(mb * 3 * 2);
  L.total = o;
  return L;
}

struct BwdArgs {
  const fovea_params* P;
  int B;
  const int64_t* mem_off;
  int64_t n_mem;
  int m_max;
  const float* keys;
  const float* values;
  const int32_t* node_off;
  int n, t_max;
  const float* h;
  const int32_t* depth;
  const int32_t* K;
  const int32_t* idx;
  int k_max;
  const float* dh_hat;
  float* dh;
  float* dkeys;
  float* dvalues;
  const fovea_grads* G;
  char* ws;
};

void launch_fill(float* p, int64_t count, hipStream_t s) {
  if (count <= 0) return;
  const int64_t blocks = std::min<int64_t>((count + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_f32_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, count, p, 0.f);
}

void launch_transpose(int R, int R_pad, int C, const float* src, int64_t lds, float* dst,
                      int64_t ldd, hipStream_t s) {
  hipLaunchKernelGGL(transpose_f32_kernel, dim3((C + 63) / 64, (R_pad + 63) / 64), dim3(256), 0, s,
                     R, R_pad, C, src, lds, dst, ldd);
}

template <int EPI, typename T, int BM>
void launch_bwd_gemm_bm(const BwdGemm& g, hipStream_t s) {
  using C = BwdCfg<T, BM>;
  const TileMap tm = make_tile_map((g.M + C::BM - 1) / C::BM, (g.N + C::BN - 1) / C::BN,
                                   static_cast<double>(g.M) * g.K, static_cast<double>(g.N) * g.K);
  hipLaunchKernelGGL((bwd_gemm_kernel<EPI, T, BM>), dim3(tile_grid(tm)), dim3(C::NT), 0, s, tm, g);
}

// 64-row tiles, or 128-row ones where they take fewer rounds of the 256 compute units
// at about 1.5 times the time of a 64-row tile per round (bf16 operands only)
template <int EPI>
void launch_bwd_gemm(const BwdGemm& g, hipStream_t s) {
  auto rounds = [&](int bm) {
    const int64_t tiles = static_cast<int64_t>((g.M + bm - 1) / bm) * ((g.N + 127) / 128);
    return (tiles + 255) / 256;
  };
  if (!g.bf16)
    launch_bwd_gemm_bm<EPI, float, 64>(g, s);
  else if (3 * rounds(128) < 2 * rounds(64))
    launch_bwd_gemm_bm<EPI, bf16_t, 128>(g, s);
  else
    launch_bwd_gemm_bm<EPI, bf16_t, 64>(g, s);
}

void launch_split3(int R, int C, const float* src, int64_t lds, bf16_t* dst, int pattern,
                   hipStream_t s) {
  hipLaunchKernelGGL(split3_kernel, dim3((C + 1023) / 1024, R), dim3(256), 0, s, R, C, src, lds, dst,
                     pattern);
}

BwdGemm bwd_gemm(int M, int N, int K, const float* A, int64_t lda, const float* B, int64_t ldb,
                 float* out, int64_t ldo) {
  BwdGemm g{};
  g.M = M;
  g.N = N;
  g.K = K;
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.out = out;
  g.ldo = ldo;
  return g;
}

void launch_transpose_split3(int R, int R_pad, int C, const float* src, int64_t lds, bf16_t* dst,
                             int W, int r_off, int pattern, hipStream_t s) {
  hipLaunchKernelGGL(transpose_split3_kernel, dim3((C + 63) / 64, (R_pad + 63) / 64), dim3(256), 0, s,
                     R, R_pad, C, src, lds, dst, W, r_off, pattern);
}

// A GEMM over bf16 planes already in sa (A', [M, 3 K]) and sb (B', [N, 3 K]).
BwdGemm planes_gemm(int M, int N, int K, bf16_t* sa, bf16_t* sb, float* out, int64_t ldo) {
  BwdGemm g = bwd_gemm(M, N, 3 * K, nullptr, 3 * K, nullptr, 3 * K, out, ldo);
  g.A = sa;
  g.B = sb;
  g.bf16 = true;
  return g;
}

// Splits A [M, K] and B [N, K] (fp32) into bf16 planes in sa / sb and returns the GEMM
// over them (K' = 3 K); the caller launches it before the next split reuses sa / sb.
BwdGemm split_gemm(int M, int N, int K, const float* A, int64_t lda, const float* B, int64_t ldb,
                   float* out, int64_t ldo, bf16_t* sa, bf16_t* sb, hipStream_t s) {
  launch_split3(M, K, A, lda, sa, 0, s);
  launch_split3(N, K, B, ldb, sb, 1, s);
  BwdGemm g = bwd_gemm(M, N, 3 * K, nullptr, 3 * K, nullptr, 3 * K, out, ldo);
  g.A = sa;
  g.B = sb;
  g.bf16 = true;
  return g;
}

// The weight-gradient GEMM dW = X^T Y over the node axis: X [n, M] (ld ldx) and
// Y [n, N] (ld ldy) are transposed into bf16 planes (K = n_pad) in sa / sb.
BwdGemm split_gemm_nodes(int n, int n_pad, int M, int N, const float* X, int64_t ldx,
                         const float* Y, int64_t ldy, float* out, int64_t ldo, bf16_t* sa,
                         bf16_t* sb, hipStream_t s) {
  launch_transpose_split3(n, n_pad, M, X, ldx, sa, n_pad, 0, 0, s);
  launch_transpose_split3(n, n_pad, N, Y, ldy, sb, n_pad, 0, 1, s);
  BwdGemm g = bwd_gemm(M, N, 3 * n_pad, nullptr, 3 * n_pad, nullptr, 3 * n_pad, out, ldo);
  g.A = sa;
  g.B = sb;
  g.bf16 = true;
  return g;
}

// Column-sum jobs launched together (up to kColJobs per launch pair); every job's
// partials get their own region of part, at increasing offsets, so part must hold
// kColChunks x (sum over the jobs of slots x cols) floats.
struct ColSums {
  ColJobs js{};
  int max_cols = 0;
  int64_t off = 0;
  int n;
  float* part;
  hipStream_t s;
  ColSums(int n_rows, float* part_ws, hipStream_t stream) : n(n_rows), part(part_ws), s(stream) {}
  static ColJob job(int cols, const float* X, int64_t ldx) {
    ColJob j{};
    j.X = X;
    j.ldx = ldx;
    j.cols = cols;
    return j;
  }
  void add(ColJob jb) {
    if (js.n_jobs == kColJobs) flush();
    const int slots = (jb.out_x != nullptr) + (jb.out_xy != nullptr) + (jb.out_grp != nullptr ? jb.ng : 0);
    jb.part_off = off;
    off += static_cast<int64_t>(kColChunks) * slots * jb.cols;
    js.job[js.n_jobs++] = jb;
    max_cols = std::max(max_cols, jb.cols);
  }
  // the sums of x grouped by grp (n_groups groups), kColGroups groups per job; the first
  // job also takes base's other outputs
  void add_grouped(ColJob base, const int32_t* grp, int n_groups, float* out) {
    for (int g0 = 0; g0 < n_groups; g0 += kColGroups) {
      ColJob jb = base;
      if (g0 > 0) jb.out_x = jb.out_xy = nullptr;
      jb.grp = grp;
      jb.out_grp = out;
      jb.g0 = g0;
      jb.ng = std::min(kColGroups, n_groups - g0);
      jb.n_grp_total = n_groups;
      add(jb);
    }
  }
  void flush() {
    if (js.n_jobs == 0) return;
    hipLaunchKernelGGL(colsum_multi_kernel, dim3((max_cols + 1023) / 1024, kColChunks, js.n_jobs),
                       dim3(256), 0, s, n, js, part);
    hipLaunchKernelGGL(colsum_multi_final_kernel, dim3((max_cols + 255) / 256, kColSlots, js.n_jobs),
                       dim3(256), 0, s, js, part);
    js.n_jobs = 0;
    max_cols = 0;
  }
};

void launch_rowsum(int rows, int len, const float* X, int64_t ldx, const float* sc, float* out,
                   hipStream_t s) {
  hipLaunchKernelGGL(rowsum_kernel, dim3((rows + 3) / 4), dim3(256), 0, s, rows, len, X, ldx, sc, out);
}

fovea_status run_backward(fovea_ctx* c, const BwdArgs& a, hipStream_t s) {
  const fovea_dims& D = c->dims;
  const int n = a.n, d = D.d, dm = D.d_m, dc = D.d_c, nd = D.n_depth;
  const BwdLayout L = bwd_layout(D, a.B, n, a.k_max, a.m_max);
  const int np = L.npad;
  char* w = a.ws;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(w + off); };
  // every GEMM of the backward runs on the bf16 matrix cores over its operands' planes
  auto bwd_gemm = [&](int M, int N, int K, const float* A, int64_t lda, const float* B,
                      int64_t ldb, float* out, int64_t ldo) {
    return split_gemm(M, N, K, A, lda, B, ldb, out, ldo, reinterpret_cast<bf16_t*>(w + L.sa),
                      reinterpret_cast<bf16_t*>(w + L.sb), s);
  };
  int32_t* node_req = reinterpret_cast<int32_t*>(w + L.node_req);
  NodeInfo* info = reinterpret_cast<NodeInfo*>(w + L.info);
  float2* stats = reinterpret_cast<float2*>(w + L.stats);
  int32_t* ok = reinterpret_cast<int32_t*>(w + L.ok);
  const float* W_Q = static_cast<const float*>(a.P->W_Q);
  const float* W_c1 = static_cast<const float*>(a.P->W_c1);
  const float* W_g1 = static_cast<const float*>(a.P->W_g1);
  const float* W_c2 = static_cast<const float*>(a.P->W_c2);
  const float* rms_w = static_cast<const float*>(a.P->rms_w);
  const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(dm)));
  const fovea_grads& G = *a.G;
  // per-node kernels keep q, dr and the selection's scores in LDS
  const size_t sm_fwd = static_cast<size_t>(dm + a.k_max) * 4;
  const size_t sm_bwd = static_cast<size_t>(dm + a.k_max) * 4;
  const size_t sm_mem = static_cast<size_t>(a.t_max) * kMemRows * 2 * 4;
  if (sm_mem > c->lds_limit[kLdsBwdMem] || sm_fwd > c->lds_limit[kLdsBwdSelFwd] ||
      sm_bwd > c->lds_limit[kLdsBwdSel])
    return FOVEA_ERR_UNSUPPORTED;
  {
    ProfScope ps(c, kBwdFill, s);
    launch_fill(F(L.tau0), a.B, s);
    launch_fill(F(L.dlogit), np, s);
    if (a.n_mem > 0)
      hipLaunchKernelGGL(bwd_mem_gaps_kernel, dim3(static_cast<unsigned>((a.n_mem + 15) / 16)), dim3(256), 0,
                         s, dm, a.m_max, a.t_max, a.B, a.mem_off, a.node_off, n, a.n_mem, a.dkeys,
                         a.dvalues);
  }
  {
    ProfScope ps(c, kBwdStats, s);
    hipLaunchKernelGGL(row_stats_kernel<float>, dim3((n + 3) / 4), dim3(256), 0, s, n, a.h, d,
                       D.ln_eps, stats, a.depth, nd, a.node_off, a.B, a.t_max, F(L.tau0), a.mem_off,
                       a.n_mem, a.m_max, node_req, info, c->err);
  }
  bf16_t* sa = reinterpret_cast<bf16_t*>(w + L.sa);
  bf16_t* sb = reinterpret_cast<bf16_t*>(w + L.sb);
  {
    ProfScope ps(c, kBwdPrep, s);
    hipLaunchKernelGGL(bwd_prep_kernel, dim3(n), dim3(256), 0, s, n, d, dm, a.h, stats, node_req,
                       a.depth, nd, static_cast<const float*>(a.P->q_ln_g),
                       static_cast<const float*>(a.P->q_ln_b), static_cast<const float*>(a.P->E_dep),
                       F(L.xhat), F(L.xe), F(L.y));
  }
  {
    ProfScope ps(c, kBwdGemm, s);
    launch_bwd_gemm<kEpiStore>(bwd_gemm(n, dm, d, F(L.xe), d, W_Q, d, F(L.q), dm), s);
  }
  {
    ProfScope ps(c, kBwdSelFwd, s);
    hipLaunchKernelGGL(bwd_sel_fwd_kernel, dim3(n), dim3(256), sm_fwd, s, n, d, dm, a.k_max, info, a.K,
                       a.idx, F(L.q), a.keys, a.values, scale, F(L.alpha), F(L.y), ok, c->err);
  }
  {
    ProfScope ps(c, kBwdGemm, s);
    // layer 1 of both nets in one GEMM (2 d_c columns); the bias is [b_c1; b_g1]
    // B = [W_c1; W_g1], split straight from the two weights
    launch_split3(n, d + dm, F(L.y), d + dm, sa, 0, s);
    launch_split3(dc, d + dm, W_c1, d + dm, sb, 1, s);
    launch_split3(dc, d + dm, W_g1, d + dm, sb + static_cast<int64_t>(dc) * 3 * (d + dm), 1, s);
    BwdGemm g = planes_gemm(n, 2 * dc, d + dm, sa, sb, F(L.z), 2 * dc);
    g.bias = static_cast<const float*>(a.P->b_c1);
    g.bias2 = static_cast<const float*>(a.P->b_g1);
    g.split = dc;
    g.out2 = F(L.a);
    g.ldo2 = 2 * dc;
    launch_bwd_gemm<kEpiZ>(g, s);
    BwdGemm g2 = bwd_gemm(n, d, dc, F(L.a), 2 * dc, W_c2, dc, F(L.c), d);
    g2.bias = static_cast<const float*>(a.P->b_c2);
    launch_bwd_gemm<kEpiStore>(g2, s);
  }
  {
    ProfScope ps(c, kBwdRmsGate, s);
    hipLaunchKernelGGL(bwd_rms_gate_kernel, dim3(n), dim3(256), 0, s, n, d, dc, a.h, F(L.c), F(L.z),
                       F(L.a), static_cast<const float*>(a.P->w_g2), a.P->b_g2, rms_w, D.rms_eps,
                       a.dh_hat, ok, a.dh, F(L.dc), F(L.hn), F(L.dlogit), F(L.dz));
  }
  {
    ProfScope ps(c, kBwdGemm, s);
    // B = W_c2^T, transposed straight into its planes
    launch_split3(n, d, F(L.dc), d, sa, 0, s);
    launch_transpose_split3(d, d, dc, W_c2, dc, sb, d, 0, 1, s);
    BwdGemm g = planes_gemm(n, dc, d, sa, sb, F(L.dz), 2 * dc);
    g.aux = F(L.z);
    g.ldaux = 2 * dc;
    launch_bwd_gemm<kEpiDsilu>(g, s);
    // B = [W_c1; W_g1]^T: the two weights transposed side by side along K
    launch_split3(n, 2 * dc, F(L.dz), 2 * dc, sa, 0, s);
    launch_transpose_split3(dc, dc, d + dm, W_c1, d + dm, sb, 2 * dc, 0, 1, s);
    launch_transpose_split3(dc, dc, d + dm, W_g1, d + dm, sb, 2 * dc, dc, 1, s);
    BwdGemm g2 = planes_gemm(n, d + dm, 2 * dc, sa, sb, a.dh, d);
    g2.split = d;
    g2.out2 = F(L.dr);
    g2.ldo2 = dm;
    launch_bwd_gemm<kEpiSplit>(g2, s);
  }
  {
    ProfScope ps(c, kBwdSel, s);
    hipLaunchKernelGGL(bwd_sel_kernel, dim3(n), dim3(256), sm_bwd, s, n, dm, a.k_max, a.m_max, info,
                       a.K, a.idx, ok, F(L.alpha), F(L.dr), a.keys, a.values, scale, F(L.dq),
                       F(L.wa), F(L.wsel));
    if (a.m_max > 0)
      hipLaunchKernelGGL(bwd_mem_grad_kernel, dim3((dm + 255) / 256, (a.m_max + kMemRows - 1) / kMemRows, a.B),
                         dim3(256), sm_mem, s, dm, a.m_max, a.t_max, a.mem_off, a.node_off, n, a.n_mem,
                         F(L.wa), F(L.wsel), F(L.dr), F(L.q), a.dkeys, a.dvalues);
  }
  {
    ProfScope ps(c, kBwdGemm, s);
    launch_split3(n, dm, F(L.dq), dm, sa, 0, s);
    launch_transpose_split3(dm, dm, d, W_Q, d, sb, dm, 0, 1, s);
    launch_bwd_gemm<kEpiStore>(planes_gemm(n, d, dm, sa, sb, F(L.dxe), d), s);
  }
  {
    ProfScope ps(c, kBwdLn, s);
    hipLaunchKernelGGL(bwd_ln_kernel, dim3(n), dim3(256), 0, s, n, d, F(L.dxe), F(L.xhat),
                       static_cast<const float*>(a.P->q_ln_g), stats, ok, a.dh);
  }
  {
    // weight gradients: GEMMs over the node axis, operands transposed into bf16 planes
    ProfScope ps(c, kBwdGemm, s);
    launch_bwd_gemm<kEpiStore>(split_gemm_nodes(n, np, d, dc, F(L.dc), d, F(L.a), 2 * dc, G.W_c2, dc, sa, sb, s), s);
    BwdGemm g1 = split_gemm_nodes(n, np, 2 * dc, d + dm, F(L.dz), 2 * dc, F(L.y), d + dm, G.W_c1, d + dm, sa, sb, s);
    g1.split = dc;
    g1.out2 = G.W_g1;
    g1.ldo2 = d + dm;
    launch_bwd_gemm<kEpiRows>(g1, s);
    launch_bwd_gemm<kEpiStore>(split_gemm_nodes(n, np, dm, d, F(L.dq), dm, F(L.xe), d, G.W_Q, d, sa, sb, s), s);
  }
  {
    ProfScope ps(c, kBwdReduce, s);
    ColSums cs(n, F(L.part), s);
    ColJob jb = ColSums::job(d, F(L.dc), d);
    jb.out_x = G.b_c2;
    cs.add(jb);
    jb = ColSums::job(dc, F(L.dz), 2 * dc);
    jb.out_x = G.b_c1;
    cs.add(jb);
    jb = ColSums::job(dc, F(L.dz) + dc, 2 * dc);
    jb.out_x = G.b_g1;
    cs.add(jb);
    jb = ColSums::job(dc, F(L.a) + dc, 2 * dc);
    jb.rs = F(L.dlogit);
    jb.out_x = G.w_g2;
    cs.add(jb);
    if (rms_w != nullptr) {
      jb = ColSums::job(d, a.dh_hat, d);
      jb.Y = F(L.hn);
      jb.ldy = d;
      jb.out_xy = G.rms_w;
      cs.add(jb);
    }
    // dxe read once for the LayerNorm bias and gain and the depth embeddings
    jb = ColSums::job(d, F(L.dxe), d);
    jb.Y = F(L.xhat);
    jb.ldy = d;
    jb.out_x = G.q_ln_b;
    jb.out_xy = G.q_ln_g;
    cs.add_grouped(jb, a.depth, nd, G.E_dep);
    cs.flush();
    launch_rowsum(1, np, F(L.dlogit), np, nullptr, G.b_g2, s);
  }
  FOVEA_HIP(hipGetLastError());
  return FOVEA_OK;
}

// memory-build backward: workspace layout and launches
struct MemBwdLayout {
  int npad;
  size_t stats, xhat, xn, dxn, WKT, WUT, part, sa, sb, total;
};

MemBwdLayout mem_bwd_layout(const fovea_dims& D, int64_t n) {
  MemBwdLayout L;
  const size_t dv = D.d_v, dm = D.d_m, nn = static_cast<size_t>(n);
  const size_t np = (nn + 63) / 64 * 64;
  L.npad = static_cast<int>(np);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L.stats = take(nn * 8);
  L.xhat = take(nn * dv * 4);
  L.xn = take(nn * dv * 4);
  L.dxn = take(nn * dv * 4);
  L.WKT = take(dv * dm * 4);
  L.WUT = take(dv * dm * 4);
  L.part = take(static_cast<size_t>(kColChunks) * 2 * dv * 4);
  L.sa = take(std::max(dm * np, nn * dm) * 3 * 2);
  L.sb = take(std::max(dv * np, dv * dm) * 3 * 2);
  L.total = o;
  return L;
}

fovea_status run_mem_backward(fovea_ctx* c, const fovea_params* P, int n, const float* V,
                              const float* dk, const float* du, float* dW_K, float* dW_U,
                              float* dg, float* db, float* dV, char* w, hipStream_t s) {
  const fovea_dims& D = c->dims;
  const int dv = D.d_v, dm = D.d_m;
  const MemBwdLayout L = mem_bwd_layout(D, n);
  const int np = L.npad;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(w + off); };
  auto bwd_gemm = [&](int M, int N, int K, const float* A, int64_t lda, const float* B,
                      int64_t ldb, float* out, int64_t ldo) {
    return split_gemm(M, N, K, A, lda, B, ldb, out, ldo, reinterpret_cast<bf16_t*>(w + L.sa),
                      reinterpret_cast<bf16_t*>(w + L.sb), s);
  };
  float2* stats = reinterpret_cast<float2*>(w + L.stats);
  const float* W_K = static_cast<const float*>(P->W_K);
  const float* W_U = static_cast<const float*>(P->W_U);
  ProfScope ps(c, kBwdMem, s);
  hipLaunchKernelGGL(row_stats_kernel<float>, dim3((n + 3) / 4), dim3(256), 0, s, n, V, dv, D.ln_eps,
                     stats, static_cast<const int32_t*>(nullptr), 0, static_cast<const int32_t*>(nullptr),
                     0, 0, static_cast<const float*>(nullptr), static_cast<const int64_t*>(nullptr),
                     int64_t{0}, 0, static_cast<int32_t*>(nullptr), static_cast<NodeInfo*>(nullptr), c->err);
  hipLaunchKernelGGL(ln_apply_kernel, dim3(n), dim3(256), 0, s, n, dv, V, stats,
                     static_cast<const float*>(P->mem_ln_g), static_cast<const float*>(P->mem_ln_b),
                     F(L.xhat), F(L.xn));
  launch_transpose(dm, dm, dv, W_K, dv, F(L.WKT), dm, s);
  launch_transpose(dm, dm, dv, W_U, dv, F(L.WUT), dm, s);
  // weight gradients over the row axis
  bf16_t* sa = reinterpret_cast<bf16_t*>(w + L.sa);
  bf16_t* sb = reinterpret_cast<bf16_t*>(w + L.sb);
  launch_bwd_gemm<kEpiStore>(split_gemm_nodes(n, np, dm, dv, dk, dm, F(L.xn), dv, dW_K, dv, sa, sb, s), s);
  launch_bwd_gemm<kEpiStore>(split_gemm_nodes(n, np, dm, dv, du, dm, F(L.xn), dv, dW_U, dv, sa, sb, s), s);
  // dL/dLN(v) = dk W_K + du W_U
  launch_bwd_gemm<kEpiStore>(bwd_gemm(n, dv, dm, dk, dm, F(L.WKT), dm, F(L.dxn), dv), s);
  BwdGemm g2 = bwd_gemm(n, dv, dm, du, dm, F(L.WUT), dm, F(L.dxn), dv);
  g2.split = dv;  // every column accumulates into dxn
  launch_bwd_gemm<kEpiSplit>(g2, s);
  ColSums cs(n, F(L.part), s);
  ColJob jb = ColSums::job(dv, F(L.dxn), dv);
  jb.Y = F(L.xhat);
  jb.ldy = dv;
  jb.out_x = db;
  jb.out_xy = dg;
  cs.add(jb);
  cs.flush();
  if (dV != nullptr) {
    launch_fill(dV, static_cast<int64_t>(n) * dv, s);
    hipLaunchKernelGGL(bwd_ln_kernel, dim3(n), dim3(256), 0, s, n, dv, F(L.dxn), F(L.xhat),
                       static_cast<const float*>(P->mem_ln_g), stats, static_cast<const int32_t*>(nullptr),
                       dV);
  }
  FOVEA_HIP(hipGetLastError());
  return FOVEA_OK;
}

}  // namespace

// ---------------------------------------------------------------------------------
// Workspace of the no-allocation entry point: one array in the code object's device
// data (zero-initialised storage: no space in the library file), which each GPU the
// library runs on holds until the process ends.  Host code never passes `scratch`
// itself (on the host it is only a stand-in symbol): its device address on each GPU
// is read once, with that GPU current, by hipGetSymbolAddress, and only that address
// reaches kernels.  Every call on one GPU shares the array.
// ---------------------------------------------------------------------------------
static __device__ __align__(256) unsigned char scratch[FOVEA_STATIC_WORKSPACE_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices];

// Device address of `scratch` on `device`, which must be the current device.
fovea_status scratch_address(int device, void** out) {
  *out = nullptr;
  if (device < 0 || device >= kMaxDevices) return FOVEA_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[device] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return FOVEA_ERR_DEVICE;
    g_scratch_addr[device] = p;
  }
  *out = g_scratch_addr[device];
  return FOVEA_OK;
}

}  // namespace

extern "C" {

int fovea_abi_version(void) { return FOVEA_ABI_VERSION; }

const char* fovea_status_str(fovea_status st) {
  switch (st) {
    case FOVEA_OK: return "ok";
    case FOVEA_ERR_INVALID_ARG: return "invalid argument";
    case FOVEA_ERR_UNSUPPORTED: return "unsupported size";
    case FOVEA_ERR_WORKSPACE: return "workspace too small or misaligned";
    case FOVEA_ERR_DEVICE: return "HIP runtime error";
    case FOVEA_ERR_DATA: return "device-side data error";
  }
  return "unknown status";
}

fovea_status fovea_create(fovea_ctx** out, const fovea_dims* dims, const fovea_params* p,
                          hipStream_t stream) {
  if (out == nullptr) return FOVEA_ERR_INVALID_ARG;
  *out = nullptr;
  if (!dims_ok(dims) || p == nullptr) return FOVEA_ERR_INVALID_ARG;
  const void* required[] = {p->mem_ln_g, p->mem_ln_b, p->W_K, p->W_U, p->q_ln_g, p->q_ln_b,
                            p->E_dep,    p->W_Q,      p->W_c1, p->b_c1, p->W_c2, p->b_c2,
                            p->W_g1,     p->b_g1,     p->w_g2};
  for (const void* r : required)
    if (r == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (std::isnan(p->b_g2)) return FOVEA_ERR_INVALID_ARG;
  if (!dims_supported(dims)) return FOVEA_ERR_UNSUPPORTED;

  fovea_ctx* c = new (std::nothrow) fovea_ctx();
  if (c == nullptr) return FOVEA_ERR_DEVICE;
  c->dims = *dims;
  c->bf16 = dims->dtype == FOVEA_BF16;
  c->es = c->bf16 ? 2 : 4;
  c->b_g2 = p->b_g2;
  if (hipGetDevice(&c->device) != hipSuccess || scratch_address(c->device, &c->scratch) != FOVEA_OK) {
    delete c;
    return FOVEA_ERR_DEVICE;
  }
  const int64_t d = dims->d, d_v = dims->d_v, d_m = dims->d_m, d_c = dims->d_c, nd = dims->n_depth;
  size_t o = 0;
  const size_t oWhq = o; o = align_up(o + (d_m + 2 * d_c) * d * c->es);
  const size_t oQc1 = o; o = align_up(o + d_m * 4);
  const size_t oQc2 = o; o = align_up(o + nd * d_m * 4);
  const size_t oWKU = o; o = align_up(o + 2 * d_m * d_v * c->es);
  const size_t oMc1 = o; o = align_up(o + 2 * d_m * 4);
  const size_t oMc2 = o; o = align_up(o + 2 * d_m * 4);
  const size_t oW1r = o; o = align_up(o + 2 * d_c * d_m * c->es);
  const size_t oB1 = o; o = align_up(o + 2 * d_c * 4);
  const size_t oWc2 = o; o = align_up(o + d * d_c * c->es);
  const size_t oBc2 = o; o = align_up(o + d * 4);
  const size_t oWg2 = o; o = align_up(o + d_c * 4);
  const size_t oRms = o; o = align_up(o + d * 4);
  const size_t oErr = o; o = align_up(o + 4);
  if (hipMalloc(&c->block, o) != hipSuccess) {
    delete c;
    return FOVEA_ERR_DEVICE;
  }
  char* base = static_cast<char*>(c->block);
  c->W_hq = base + oWhq;
  c->q_c1 = reinterpret_cast<float*>(base + oQc1);
  c->q_c2 = reinterpret_cast<float*>(base + oQc2);
  c->W_KU = base + oWKU;
  c->m_c1 = reinterpret_cast<float*>(base + oMc1);
  c->m_c2 = reinterpret_cast<float*>(base + oMc2);
  c->W1r = base + oW1r;
  c->b1 = reinterpret_cast<float*>(base + oB1);
  c->W_c2 = base + oWc2;
  c->b_c2 = reinterpret_cast<float*>(base + oBc2);
  c->w_g2 = reinterpret_cast<float*>(base + oWg2);
  c->rms_w = p->rms_w ? reinterpret_cast<float*>(base + oRms) : nullptr;
  c->err = reinterpret_cast<uint32_t*>(base + oErr);
  fovea_status st = hipMemsetAsync(c->err, 0, 4, stream) == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
  if (st == FOVEA_OK) st = raise_lds_limits(c);
  if (st == FOVEA_OK) st = c->bf16 ? pack_weights<bf16_t>(c, p, stream) : pack_weights<float>(c, p, stream);
  if (st == FOVEA_OK && hipStreamSynchronize(stream) != hipSuccess) st = FOVEA_ERR_DEVICE;
  if (st != FOVEA_OK) {
    (void)hipFree(c->block);
    delete c;
    return st;
  }
  *out = c;
  return FOVEA_OK;
}

void fovea_destroy(fovea_ctx* c) {
  if (c == nullptr) return;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(c->device);
  // wait for the last call enqueued on each stream this context was used on
  for (auto& u : c->uses) {
    (void)hipEventSynchronize(u.done);
    (void)hipEventDestroy(u.done);
  }
  (void)hipFree(c->block);
  for (auto& r : c->prof_recs) {
    (void)hipEventDestroy(r.e0);
    (void)hipEventDestroy(r.e1);
  }
  for (hipEvent_t e : c->prof_pool) (void)hipEventDestroy(e);
  (void)hipSetDevice(cur);
  delete c;
}

size_t fovea_build_memory_workspace(const fovea_ctx* c, int64_t n_rows) {
  if (c == nullptr || n_rows < 0) return 0;
  return align_up(static_cast<size_t>(n_rows) * sizeof(float2)) + kAlign;
}

fovea_status fovea_build_memory(fovea_ctx* c, int64_t n_rows, const void* V, void* keys,
                                void* values, void* workspace, size_t workspace_bytes,
                                hipStream_t stream) {
  if (c == nullptr || n_rows < 0) return FOVEA_ERR_INVALID_ARG;
  if (n_rows == 0) return FOVEA_OK;
  if (V == nullptr || keys == nullptr || values == nullptr || workspace == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  if (n_rows > (int64_t{1} << 30)) return FOVEA_ERR_UNSUPPORTED;
  if (!aligned16(V) || !aligned16(keys) || !aligned16(values)) return FOVEA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return FOVEA_ERR_WORKSPACE;
  if (workspace_bytes < fovea_build_memory_workspace(c, n_rows)) return FOVEA_ERR_WORKSPACE;
  const size_t nv = static_cast<size_t>(n_rows) * c->dims.d_v * c->es;
  const size_t nk = static_cast<size_t>(n_rows) * c->dims.d_m * c->es;
  if (overlaps(keys, nk, V, nv) || overlaps(values, nk, V, nv) || overlaps(keys, nk, values, nk) ||
      overlaps(workspace, workspace_bytes, keys, nk) || overlaps(workspace, workspace_bytes, values, nk))
    return FOVEA_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (cur != c->device) return FOVEA_ERR_INVALID_ARG;
  const int n = static_cast<int>(n_rows);
  float2* stats = static_cast<float2*>(workspace);
  const fovea_status st = c->bf16 ? run_build<bf16_t>(c, n, V, keys, values, stats, stream)
                                  : run_build<float>(c, n, V, keys, values, stats, stream);
  return st == FOVEA_OK ? record_use(c, stream) : st;
}

size_t fovea_retrieve_fuse_workspace(const fovea_ctx* c, int32_t B, int32_t n_nodes_total,
                                     int64_t n_mem_total, int32_t m_max, int32_t k_max) {
  if (c == nullptr || B < 0 || n_nodes_total < 0 || n_mem_total < 0 || m_max < 0 || k_max < 1)
    return 0;
  return ws_layout(c->dims, n_nodes_total, m_max).total;
}

static fovea_status retrieve_fuse_checked(fovea_ctx* c, int32_t B, const int64_t* mem_off,
                                 int64_t n_mem_total, int32_t m_max, const void* keys,
                                 const void* values, const uint8_t* valid,
                                 const int32_t* node_off, int32_t n_nodes_total, int32_t t_max,
                                 const void* h, const int32_t* depth, const float* tau,
                                 int32_t k_min, int32_t k_max, void* h_out, int32_t* k_out,
                                 int32_t* idx_out, float* gate_out, float* mass_out, float* r_out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 bool track) {
  if (c == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (B < 0 || n_mem_total < 0 || m_max < 0 || n_nodes_total < 0 || t_max < 0) return FOVEA_ERR_INVALID_ARG;
  if (k_max < 1 || k_min < 0 || k_min > k_max) return FOVEA_ERR_INVALID_ARG;
  if (n_nodes_total > 0 && (B == 0 || t_max == 0)) return FOVEA_ERR_INVALID_ARG;
  if (n_nodes_total == 0) return FOVEA_OK;
  if (mem_off == nullptr || node_off == nullptr || h == nullptr || depth == nullptr ||
      tau == nullptr || h_out == nullptr || workspace == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  if (n_mem_total > 0 && (keys == nullptr || values == nullptr)) return FOVEA_ERR_INVALID_ARG;
  if (m_max > kMaxM || k_max > kMaxKmax) return FOVEA_ERR_UNSUPPORTED;
  if (n_mem_total > (int64_t{1} << 40)) return FOVEA_ERR_UNSUPPORTED;
  if (!aligned16(keys) || !aligned16(values) || !aligned16(h) || !aligned16(h_out))
    return FOVEA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return FOVEA_ERR_WORKSPACE;
  const fovea_dims& D = c->dims;
  const WsLayout L = ws_layout(D, n_nodes_total, m_max);
  if (workspace_bytes < L.total) return FOVEA_ERR_WORKSPACE;
  const size_t nh = static_cast<size_t>(n_nodes_total) * D.d * c->es;
  const size_t nk = static_cast<size_t>(n_mem_total) * D.d_m * c->es;
  if (overlaps(h_out, nh, h, nh) || overlaps(h_out, nh, keys, nk) || overlaps(h_out, nh, values, nk) ||
      overlaps(h_out, nh, workspace, L.total))
    return FOVEA_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (cur != c->device) return FOVEA_ERR_INVALID_ARG;

  RFArgs a;
  a.B = B;
  a.mem_off = mem_off;
  a.n_mem = n_mem_total;
  a.m_max = m_max;
  a.keys = keys;
  a.values = values;
  a.valid = valid;
  a.node_off = node_off;
  a.n = n_nodes_total;
  a.t_max = t_max;
  a.h = h;
  a.depth = depth;
  a.tau = tau;
  a.k_min = k_min;
  a.k_max = k_max;
  a.h_out = h_out;
  a.k_out = k_out;
  a.idx_out = idx_out;
  a.gate_out = gate_out;
  a.mass_out = mass_out;
  a.r_out = r_out;
  a.ws = static_cast<char*>(workspace);
  a.track = track;
  const fovea_status st = c->bf16 ? run_retrieve_fuse<bf16_t>(c, a, stream) : run_retrieve_fuse<float>(c, a, stream);
  return st == FOVEA_OK && track ? record_use(c, stream) : st;
}

fovea_status fovea_retrieve_fuse(fovea_ctx* c, int32_t B, const int64_t* mem_off,
                                 int64_t n_mem_total, int32_t m_max, const void* keys,
                                 const void* values, const uint8_t* valid,
                                 const int32_t* node_off, int32_t n_nodes_total, int32_t t_max,
                                 const void* h, const int32_t* depth, const float* tau,
                                 int32_t k_min, int32_t k_max, void* h_out, int32_t* k_out,
                                 int32_t* idx_out, float* gate_out, float* mass_out, float* r_out,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return retrieve_fuse_checked(c, B, mem_off, n_mem_total, m_max, keys, values, valid, node_off,
                               n_nodes_total, t_max, h, depth, tau, k_min, k_max, h_out, k_out,
                               idx_out, gate_out, mass_out, r_out, workspace, workspace_bytes,
                               stream, true);
}

fovea_status fovea_retrieve_fuse_noalloc(fovea_ctx* c, int32_t B, const int64_t* mem_off,
                                         int64_t n_mem_total, int32_t m_max, const void* keys,
                                         const void* values, const uint8_t* valid,
                                         const int32_t* node_off, int32_t n_nodes_total,
                                         int32_t t_max, const void* h, const int32_t* depth,
                                         const float* tau, int32_t k_min, int32_t k_max,
                                         void* h_out, int32_t* k_out, int32_t* idx_out,
                                         float* gate_out, float* mass_out, float* r_out,
                                         hipStream_t stream) {
  if (c == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (c->scratch == nullptr) return FOVEA_ERR_DEVICE;
  if (B >= 0 && n_nodes_total >= 0 && n_mem_total >= 0 && m_max >= 0 && k_max >= 1 &&
      ws_layout(c->dims, n_nodes_total, m_max).total > FOVEA_STATIC_WORKSPACE_BYTES)
    return FOVEA_ERR_WORKSPACE;
  return retrieve_fuse_checked(c, B, mem_off, n_mem_total, m_max, keys, values, valid, node_off,
                               n_nodes_total, t_max, h, depth, tau, k_min, k_max, h_out, k_out,
                               idx_out, gate_out, mass_out, r_out, c->scratch,
                               FOVEA_STATIC_WORKSPACE_BYTES, stream, false);
}

fovea_status fovea_last_error(fovea_ctx* c, hipStream_t stream, uint32_t* bits) {
  if (c == nullptr) return FOVEA_ERR_INVALID_ARG;
  uint32_t v = 0;
  if (hipStreamSynchronize(stream) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (hipMemcpy(&v, c->err, 4, hipMemcpyDeviceToHost) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (v != 0 && hipMemset(c->err, 0, 4) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (bits) *bits = v;
  return v ? FOVEA_ERR_DATA : FOVEA_OK;
}

fovea_status fovea_profile(fovea_ctx* c, int32_t enable) {
  if (c == nullptr) return FOVEA_ERR_INVALID_ARG;
  c->prof = enable != 0;
  return FOVEA_OK;
}

int32_t fovea_profile_read(fovea_ctx* c, int32_t max_kernels, const char** names, float* total_ms,
                           int32_t* launches) {
  if (c == nullptr || max_kernels < 0) return -1;
  float ms[kNumSlots] = {};
  int32_t cnt[kNumSlots] = {};
  bool ok = true;
  for (auto& r : c->prof_recs) {
    float t = 0.f;
    if (hipEventSynchronize(r.e1) != hipSuccess || hipEventElapsedTime(&t, r.e0, r.e1) != hipSuccess)
      ok = false;
    ms[r.slot] += t;
    cnt[r.slot] += 1;
    c->prof_pool.push_back(r.e0);
    c->prof_pool.push_back(r.e1);
  }
  c->prof_recs.clear();
  if (!ok) return -1;
  int32_t w = 0;
  for (int i = 0; i < kNumSlots && w < max_kernels; ++i) {
    if (cnt[i] == 0) continue;
    if (names) names[w] = kSlotNames[i];
    if (total_ms) total_ms[w] = ms[i];
    if (launches) launches[w] = cnt[i];
    ++w;
  }
  return w;
}

size_t fovea_lm_topk_workspace(const fovea_ctx* c, int32_t n_rows, int32_t vocab, int32_t k) {
  if (c == nullptr || n_rows < 0 || k < 1 || k > kLmMaxK || vocab < k || vocab > kLmMaxVocab ||
      n_rows > kLmMaxRows)
    return 0;
  return lm_cand_bytes(n_rows, vocab, k);
}

fovea_status fovea_lm_topk(fovea_ctx* c, int32_t n_rows, const void* h, const void* W_LM,
                           int32_t vocab, int32_t k, int32_t* idx_out, float* logit_out,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (c == nullptr || n_rows < 0 || k < 1 || vocab < k) return FOVEA_ERR_INVALID_ARG;
  if (k > kLmMaxK || vocab > kLmMaxVocab || n_rows > kLmMaxRows) return FOVEA_ERR_UNSUPPORTED;
  if (n_rows == 0) return FOVEA_OK;
  if (h == nullptr || W_LM == nullptr || idx_out == nullptr || workspace == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  if (!aligned16(h) || !aligned16(W_LM)) return FOVEA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return FOVEA_ERR_WORKSPACE;
  const size_t need = lm_cand_bytes(n_rows, vocab, k);
  if (workspace_bytes < need) return FOVEA_ERR_WORKSPACE;
  const size_t ni = static_cast<size_t>(n_rows) * k * 4;
  if (overlaps(idx_out, ni, workspace, need) || overlaps(logit_out, ni, workspace, need) ||
      overlaps(idx_out, ni, logit_out, ni))
    return FOVEA_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (cur != c->device) return FOVEA_ERR_INVALID_ARG;
  uint64_t* cand = static_cast<uint64_t*>(workspace);
  const fovea_status st =
      c->bf16 ? run_lm_topk<bf16_t>(c, n_rows, h, W_LM, vocab, k, idx_out, logit_out, cand, stream)
              : run_lm_topk<float>(c, n_rows, h, W_LM, vocab, k, idx_out, logit_out, cand, stream);
  return st == FOVEA_OK ? record_use(c, stream) : st;
}

size_t fovea_retrieve_fuse_backward_workspace(const fovea_ctx* c, int32_t B, int32_t n_nodes_total,
                                              int32_t m_max, int32_t k_max) {
  if (c == nullptr || B < 0 || n_nodes_total < 0 || m_max < 0 || m_max > kMaxM || k_max < 1 ||
      k_max > kMaxKmax)
    return 0;
  return bwd_layout(c->dims, B, n_nodes_total, k_max, m_max).total;
}

fovea_status fovea_retrieve_fuse_backward(
    fovea_ctx* c, const fovea_params* p, int32_t B, const int64_t* mem_off, int64_t n_mem_total,
    int32_t m_max, const float* keys, const float* values, const int32_t* node_off,
    int32_t n_nodes_total, int32_t t_max, const float* h, const int32_t* depth, const int32_t* K,
    const int32_t* idx, int32_t k_max, const float* dh_hat, float* dh, float* dkeys,
    float* dvalues, const fovea_grads* g, void* workspace, size_t workspace_bytes,
    hipStream_t stream) {
  if (c == nullptr || p == nullptr || g == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (c->bf16) return FOVEA_ERR_UNSUPPORTED;
  if (B < 0 || n_mem_total < 0 || m_max < 0 || n_nodes_total < 0 || t_max < 0 || k_max < 1)
    return FOVEA_ERR_INVALID_ARG;
  if (n_nodes_total > 0 && (B == 0 || t_max == 0)) return FOVEA_ERR_INVALID_ARG;
  if (m_max > kMaxM || k_max > kMaxKmax || n_mem_total > (int64_t{1} << 40)) return FOVEA_ERR_UNSUPPORTED;
  if ((static_cast<size_t>(c->dims.d_m) + k_max) * 4 > 150 * 1024) return FOVEA_ERR_UNSUPPORTED;
  if (static_cast<size_t>(t_max) * kMemRows * 2 * 4 > 150 * 1024) return FOVEA_ERR_UNSUPPORTED;
  const void* wreq[] = {p->q_ln_g, p->q_ln_b, p->E_dep, p->W_Q, p->W_c1, p->b_c1,
                        p->W_c2,   p->b_c2,   p->W_g1,  p->b_g1, p->w_g2};
  for (const void* r : wreq)
    if (r == nullptr || !aligned16(r)) return FOVEA_ERR_INVALID_ARG;
  if (p->rms_w != nullptr && !aligned16(p->rms_w)) return FOVEA_ERR_INVALID_ARG;
  float* greq[] = {g->W_Q, g->q_ln_g, g->q_ln_b, g->E_dep, g->W_c1, g->b_c1, g->W_c2,
                   g->b_c2, g->W_g1, g->b_g1, g->w_g2, g->b_g2};
  for (float* r : greq)
    if (r == nullptr || !aligned16(r)) return FOVEA_ERR_INVALID_ARG;
  if ((p->rms_w != nullptr) != (g->rms_w != nullptr)) return FOVEA_ERR_INVALID_ARG;
  if (std::isnan(p->b_g2)) return FOVEA_ERR_INVALID_ARG;
  if (mem_off == nullptr || node_off == nullptr || workspace == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (n_nodes_total > 0 && dh == nullptr) return FOVEA_ERR_INVALID_ARG;
  if (n_mem_total > 0 && (dkeys == nullptr || dvalues == nullptr)) return FOVEA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return FOVEA_ERR_WORKSPACE;
  const BwdLayout L = bwd_layout(c->dims, B, n_nodes_total, k_max, m_max);
  if (workspace_bytes < L.total) return FOVEA_ERR_WORKSPACE;
  const fovea_dims& D = c->dims;
  if (n_nodes_total == 0) {
    // no node: every gradient is zero
    const int64_t sizes[] = {int64_t{D.d_m} * D.d, D.d, D.d, int64_t{D.n_depth} * D.d,
                             int64_t{D.d_c} * (D.d + D.d_m), D.d_c, int64_t{D.d} * D.d_c, D.d,
                             int64_t{D.d_c} * (D.d + D.d_m), D.d_c, D.d_c, 1};
    for (int i = 0; i < 12; ++i) launch_fill(greq[i], sizes[i], stream);
    if (g->rms_w) launch_fill(g->rms_w, D.d, stream);
    launch_fill(dkeys, n_mem_total * D.d_m, stream);
    launch_fill(dvalues, n_mem_total * D.d_m, stream);
    return hipGetLastError() == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
  }
  if (h == nullptr || depth == nullptr || K == nullptr || idx == nullptr || dh_hat == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  if (n_mem_total > 0 && (keys == nullptr || values == nullptr)) return FOVEA_ERR_INVALID_ARG;
  if (!aligned16(h) || !aligned16(dh_hat) || !aligned16(dh) || !aligned16(keys) ||
      !aligned16(values) || !aligned16(dkeys) || !aligned16(dvalues))
    return FOVEA_ERR_INVALID_ARG;
  const size_t nh = static_cast<size_t>(n_nodes_total) * D.d * 4;
  const size_t nk = static_cast<size_t>(n_mem_total) * D.d_m * 4;
  if (overlaps(dh, nh, h, nh) || overlaps(dh, nh, dh_hat, nh) || overlaps(dh, nh, workspace, L.total) ||
      overlaps(dkeys, nk, keys, nk) || overlaps(dkeys, nk, values, nk) ||
      overlaps(dvalues, nk, keys, nk) || overlaps(dvalues, nk, values, nk) ||
      overlaps(dkeys, nk, dvalues, nk) || overlaps(dkeys, nk, workspace, L.total) ||
      overlaps(dvalues, nk, workspace, L.total))
    return FOVEA_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (cur != c->device) return FOVEA_ERR_INVALID_ARG;
  BwdArgs a;
  a.P = p;
  a.B = B;
  a.mem_off = mem_off;
  a.n_mem = n_mem_total;
  a.m_max = m_max;
  a.keys = keys;
  a.values = values;
  a.node_off = node_off;
  a.n = n_nodes_total;
  a.t_max = t_max;
  a.h = h;
  a.depth = depth;
  a.K = K;
  a.idx = idx;
  a.k_max = k_max;
  a.dh_hat = dh_hat;
  a.dh = dh;
  a.dkeys = dkeys;
  a.dvalues = dvalues;
  a.G = g;
  a.ws = static_cast<char*>(workspace);
  const fovea_status st = run_backward(c, a, stream);
  return st == FOVEA_OK ? record_use(c, stream) : st;
}

size_t fovea_build_memory_backward_workspace(const fovea_ctx* c, int64_t n_rows) {
  if (c == nullptr || n_rows < 0 || n_rows > (int64_t{1} << 30)) return 0;
  return mem_bwd_layout(c->dims, n_rows).total;
}

fovea_status fovea_build_memory_backward(fovea_ctx* c, const fovea_params* p, int64_t n_rows,
                                         const float* V, const float* dkeys, const float* dvalues,
                                         float* dW_K, float* dW_U, float* dmem_ln_g,
                                         float* dmem_ln_b, float* dV, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
  if (c == nullptr || p == nullptr || n_rows < 0) return FOVEA_ERR_INVALID_ARG;
  if (c->bf16) return FOVEA_ERR_UNSUPPORTED;
  if (n_rows > (int64_t{1} << 30)) return FOVEA_ERR_UNSUPPORTED;
  if (p->W_K == nullptr || p->W_U == nullptr || p->mem_ln_g == nullptr || p->mem_ln_b == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  float* outs[] = {dW_K, dW_U, dmem_ln_g, dmem_ln_b};
  for (float* o : outs)
    if (o == nullptr || !aligned16(o)) return FOVEA_ERR_INVALID_ARG;
  const fovea_dims& D = c->dims;
  if (n_rows == 0) {
    launch_fill(dW_K, int64_t{D.d_m} * D.d_v, stream);
    launch_fill(dW_U, int64_t{D.d_m} * D.d_v, stream);
    launch_fill(dmem_ln_g, D.d_v, stream);
    launch_fill(dmem_ln_b, D.d_v, stream);
    return hipGetLastError() == hipSuccess ? FOVEA_OK : FOVEA_ERR_DEVICE;
  }
  if (V == nullptr || dkeys == nullptr || dvalues == nullptr || workspace == nullptr)
    return FOVEA_ERR_INVALID_ARG;
  if (!aligned16(V) || !aligned16(dkeys) || !aligned16(dvalues) || !aligned16(dV))
    return FOVEA_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(workspace) & (kAlign - 1)) != 0) return FOVEA_ERR_WORKSPACE;
  const MemBwdLayout L = mem_bwd_layout(D, n_rows);
  if (workspace_bytes < L.total) return FOVEA_ERR_WORKSPACE;
  const size_t nv = static_cast<size_t>(n_rows) * D.d_v * 4;
  if (overlaps(dV, nv, V, nv) || overlaps(dV, nv, workspace, L.total)) return FOVEA_ERR_INVALID_ARG;
  int cur = -1;
  if (hipGetDevice(&cur) != hipSuccess) return FOVEA_ERR_DEVICE;
  if (cur != c->device) return FOVEA_ERR_INVALID_ARG;
  const fovea_status st = run_mem_backward(c, p, static_cast<int>(n_rows), V, dkeys, dvalues, dW_K, dW_U,
                                           dmem_ln_g, dmem_ln_b, dV, static_cast<char*>(workspace), stream);
  return st == FOVEA_OK ? record_use(c, stream) : st;
}

}  // extern "C"
