/*
 * fovea.h - C ABI of the MI355X (gfx950) library for FOVEA's per-draft-step
 * visual-evidence retrieval and fusion.
 *
 * What it computes (paper, Method section):
 *   memory build, once per image ("Image-specific visual memory"):
 *       k_i = W_K LN(v_i),  u_i = W_U LN(v_i)
 *   per draft step, for every draft-tree node n of request b
 *   ("State-conditioned top-K retrieval", Algorithm 1's inner loop):
 *       q_n   = W_Q (LN(h_n) + E_dep[l_n])
 *       s_n,i = q_n . k_i / sqrt(d_m)                  over the valid keys of request b
 *       alpha~ = softmax(s_n) over the valid keys
 *       K_raw = smallest k whose top-k mass (descending score) reaches tau_b
 *       K     = min(|V_b|, k_max, max(k_min, K_raw)),  I_n = top-K indices
 *       r_n   = sum_{i in I_n} softmax over I_n (s_n,i) * u_i
 *   ("Cache-friendly hidden-vector correction", Eq. hidden_correction, and the
 *   appendix paragraph "Visual correction module"):
 *       y     = [h_n ; r_n]
 *       c_n   = W_c2 SiLU(W_c1 y + b_c1) + b_c2          (d outputs)
 *       g_n   = sigmoid(w_g2 . SiLU(W_g1 y + b_g1) + b_g2)  (scalar)
 *       h_hat = RMSNorm(h_n + g_n c_n) * rms_w            (or h_n + g_n c_n if rms_w NULL)
 *
 * Readings where the paper is silent: equal scores rank by ascending memory index;
 * if the prefix mass never reaches tau, K_raw = |V_b| (tau = 1 is dense retrieval);
 * |V_b| = 0 gives K = 0 and r_n = 0; every node passed is corrected (depth gating is
 * the caller's policy).
 *
 * Conventions
 *   - All tensor pointers are DEVICE pointers, row-major [rows, cols], weights are
 *     [out, in].  Every floating-point tensor argument has the storage dtype given
 *     in fovea_dims.dtype (fp32 or bf16) unless its type says otherwise.
 *   - The caller owns every buffer.  The context owns only the packed weight copies
 *     it makes in fovea_create (the caller's weight buffers may be freed afterwards).
 *   - All work is enqueued on `stream` (NULL = the default stream); calls return
 *     without synchronising.  fovea_retrieve_fuse allocates nothing.
 *   - Host-detectable errors return a status before anything is enqueued.  Errors
 *     that depend on device data (offsets, depth, tau) set sticky bits in the
 *     context, write NaN into the affected nodes' outputs, and are read with
 *     fovea_last_error.  Nothing throws across this ABI.
 *   - Calls that share one context may run on different streams, but they share
 *     the context's error word: one sticky word per context (not per workspace), so
 *     data errors of calls on two streams are reported together.
 */
#ifndef FOVEA_H_
#define FOVEA_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FOVEA_ABI_VERSION 1

typedef enum {
  FOVEA_OK = 0,
  FOVEA_ERR_INVALID_ARG = 1,  /* null pointer, negative size, bad k bounds, aliasing */
  FOVEA_ERR_UNSUPPORTED = 2,  /* a width not a multiple of 64, m_max/k_max over limit */
  FOVEA_ERR_WORKSPACE = 3,    /* workspace too small or misaligned */
  FOVEA_ERR_DEVICE = 4,       /* a HIP runtime error */
  FOVEA_ERR_DATA = 5          /* fovea_last_error: a device-side data error was seen */
} fovea_status;

typedef enum { FOVEA_F32 = 0, FOVEA_BF16 = 1 } fovea_dtype;

/* Sticky device-data error bits reported by fovea_last_error. */
#define FOVEA_DATA_BAD_NODE_OFFSETS 0x1u /* node_off not monotone / outside [0, n_nodes_total] / T_b > t_max */
#define FOVEA_DATA_BAD_MEM_OFFSETS 0x2u  /* mem_off not monotone / outside [0, n_mem_total] / M_b > m_max */
#define FOVEA_DATA_BAD_DEPTH 0x4u        /* depth outside [0, n_depth) */
#define FOVEA_DATA_BAD_TAU 0x8u          /* tau outside [0, 1] or NaN */

/* Limits of this build. */
#define FOVEA_MAX_M 16384   /* entries in one request's memory (m_max) */
#define FOVEA_MAX_KMAX 1024 /* k_max */

typedef struct {
  int32_t d;       /* drafter hidden size d_h; multiple of 64 */
  int32_t d_v;     /* visual token width (input of the memory build); multiple of 64 */
  int32_t d_m;     /* key and value width d_k = d_u; multiple of 64 */
  int32_t d_c;     /* hidden width of the correction and gate nets (512 in the paper); multiple of 64 */
  int32_t n_depth; /* rows of E_dep: tree depths 0..D (D = 6 in the paper, so 7) */
  fovea_dtype dtype;
  float ln_eps;    /* LayerNorm epsilon (query and memory LayerNorms) */
  float rms_eps;   /* RMSNorm epsilon */
} fovea_dims;

/* Weights, all device pointers in the storage dtype, read during fovea_create only. */
typedef struct {
  const void* mem_ln_g; /* [d_v]  LayerNorm of the memory build (Method, memory) */
  const void* mem_ln_b; /* [d_v] */
  const void* W_K;      /* [d_m, d_v] key projection, no bias */
  const void* W_U;      /* [d_m, d_v] value projection, no bias */
  const void* q_ln_g;   /* [d]    LayerNorm of the query (Method, retrieval) */
  const void* q_ln_b;   /* [d] */
  const void* E_dep;    /* [n_depth, d] depth embedding */
  const void* W_Q;      /* [d_m, d] query projection, no bias */
  const void* W_c1;     /* [d_c, d + d_m] correction net layer 1 over [h; r] */
  const void* b_c1;     /* [d_c] */
  const void* W_c2;     /* [d, d_c]       correction net layer 2 */
  const void* b_c2;     /* [d] */
  const void* W_g1;     /* [d_c, d + d_m] gate net layer 1 over [h; r] */
  const void* b_g1;     /* [d_c] */
  const void* w_g2;     /* [d_c]          gate net layer 2 (scalar output) */
  float b_g2;           /* gate output bias (host scalar; +-inf allowed) */
  const void* rms_w;    /* [d] RMSNorm weight, or NULL for h + g c without RMSNorm */
} fovea_params;

typedef struct fovea_ctx fovea_ctx;

int fovea_abi_version(void);
const char* fovea_status_str(fovea_status s);

/* Create a context on the current HIP device: validates dims, copies and packs the
 * weights (the query and memory LayerNorm gains are folded into W_Q and [W_K; W_U]
 * and, for bf16, the folded products are stored in bf16).  Enqueued on `stream` and
 * synchronised before returning.  The context's one allocation (the packed weights and
 * its error word) is made here; no later call allocates device memory.  *out is NULL
 * on failure. */
fovea_status fovea_create(fovea_ctx** out, const fovea_dims* dims, const fovea_params* params,
                          hipStream_t stream);
/* Waits for the last call enqueued through this context on each stream it was used on,
 * then frees the context.  NULL is a no-op. */
void fovea_destroy(fovea_ctx* ctx);

/* Bytes of workspace fovea_build_memory needs for n_rows tokens (0 on bad arguments). */
size_t fovea_build_memory_workspace(const fovea_ctx* ctx, int64_t n_rows);

/* Memory build (Method, image-specific visual memory): for each of the n_rows visual
 * tokens V[i] ([n_rows, d_v]) write keys[i] = W_K LN(V[i]) and values[i] = W_U LN(V[i])
 * ([n_rows, d_m] each).  Rows are independent, so the memories of many images (a
 * ragged batch packed by offsets) are built by one call over all of their rows; no
 * offsets are needed.  keys/values must not overlap V, each other or the workspace.
 * workspace: at least fovea_build_memory_workspace(ctx, n_rows) bytes, 256-byte
 * aligned, clobbered (the rows' LayerNorm statistics). */
fovea_status fovea_build_memory(fovea_ctx* ctx, int64_t n_rows, const void* V, void* keys,
                                void* values, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* Bytes of workspace fovea_retrieve_fuse needs for a call with these sizes (0 on bad
 * arguments): B requests, n_nodes_total nodes, n_mem_total memory rows, at most m_max
 * rows per request, k_max. */
size_t fovea_retrieve_fuse_workspace(const fovea_ctx* ctx, int32_t B, int32_t n_nodes_total,
                                     int64_t n_mem_total, int32_t m_max, int32_t k_max);

/* One draft step over a ragged batch of B requests (Algorithm 1, retrieval and
 * correction for every node passed).
 *   mem_off  [B+1] int64, device: request b owns memory rows mem_off[b]..mem_off[b+1]
 *            of keys/values ([n_mem_total, d_m]); M_b <= m_max (host scalar).
 *   valid    [n_mem_total] uint8, device, or NULL: 0 marks a padded entry (mask m_i).
 *   node_off [B+1] int32, device: request b owns nodes node_off[b]..node_off[b+1] of
 *            h ([n_nodes_total, d]) and depth ([n_nodes_total] int32); T_b <= t_max.
 *   tau      [B] float32, device: mass threshold rho per request, in [0, 1].
 *   k_min, k_max: host scalars, 0 <= k_min <= k_max, 1 <= k_max <= FOVEA_MAX_KMAX.
 * Outputs (device):
 *   h_out    [n_nodes_total, d] storage dtype: h_hat (must not overlap any input).
 *   k_out    [n_nodes_total] int32 or NULL: K per node.
 *   idx_out  [n_nodes_total, k_max] int32 or NULL: selected memory indices local to
 *            the request, in descending-score order, -1 after the first K.
 *   gate_out [n_nodes_total] float32 or NULL: g_n.
 *   mass_out [n_nodes_total] float32 or NULL: normalised mass of the selected set.
 *   r_out    [n_nodes_total, d_m] float32 or NULL: the readout r_n.
 * workspace: device memory of at least fovea_retrieve_fuse_workspace(...) bytes,
 * 256-byte aligned; its contents need no initialisation and are clobbered. */
fovea_status fovea_retrieve_fuse(fovea_ctx* ctx, int32_t B, const int64_t* mem_off,
                                 int64_t n_mem_total, int32_t m_max, const void* keys,
                                 const void* values, const uint8_t* valid,
                                 const int32_t* node_off, int32_t n_nodes_total, int32_t t_max,
                                 const void* h, const int32_t* depth, const float* tau,
                                 int32_t k_min, int32_t k_max, void* h_out, int32_t* k_out,
                                 int32_t* idx_out, float* gate_out, float* mass_out,
                                 float* r_out, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* Size of the device array behind fovea_retrieve_fuse_noalloc (one per GPU). */
#define FOVEA_STATIC_WORKSPACE_BYTES (64u << 20)

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): fovea_retrieve_fuse with the same
 * arguments and results, minus the workspace.  Its workspace is a fixed array of
 * FOVEA_STATIC_WORKSPACE_BYTES in the library's device data, one per GPU, reserved when
 * the library's code is loaded on that GPU and held until the process ends; its device
 * address is read once per GPU by fovea_create.  This call allocates nothing, creates
 * no events (the context's profiling and fovea_destroy's wait do not cover it: the
 * caller synchronises its stream before fovea_destroy) and returns FOVEA_ERR_WORKSPACE
 * when the sizes need more than the array holds (fovea_retrieve_fuse_workspace gives
 * the need; e.g. 32 requests x 60 nodes with 576-entry memories at d = 4096, d_m = 1024
 * need about 26 MB).  Every call on one GPU uses the same array, whose contents the
 * previous call leaves behind (the call needs none of it): calls that overlap on one
 * GPU (on different streams, or from different threads) race and must be serialised
 * by the caller. */
fovea_status fovea_retrieve_fuse_noalloc(fovea_ctx* ctx, int32_t B, const int64_t* mem_off,
                                         int64_t n_mem_total, int32_t m_max, const void* keys,
                                         const void* values, const uint8_t* valid,
                                         const int32_t* node_off, int32_t n_nodes_total,
                                         int32_t t_max, const void* h, const int32_t* depth,
                                         const float* tau, int32_t k_min, int32_t k_max,
                                         void* h_out, int32_t* k_out, int32_t* idx_out,
                                         float* gate_out, float* mass_out, float* r_out,
                                         hipStream_t stream);

/* Sticky bit of fovea_retrieve_fuse_backward: a node's K or selected index is outside
 * [0, min(k_max, M_b)] / [0, M_b) (its gradients are skipped and its dh row is NaN). */
#define FOVEA_DATA_BAD_SELECTION 0x10u

/* Gradient outputs of fovea_retrieve_fuse_backward: fp32 device arrays shaped like the
 * weights of fovea_params (raw, unfolded), overwritten.  rms_w is required exactly when
 * the weights passed have an RMSNorm weight. */
typedef struct {
  float* W_Q;    /* [d_m, d] */
  float* q_ln_g; /* [d] */
  float* q_ln_b; /* [d] */
  float* E_dep;  /* [n_depth, d] */
  float* W_c1;   /* [d_c, d + d_m] */
  float* b_c1;   /* [d_c] */
  float* W_c2;   /* [d, d_c] */
  float* b_c2;   /* [d] */
  float* W_g1;   /* [d_c, d + d_m] */
  float* b_g1;   /* [d_c] */
  float* w_g2;   /* [d_c] */
  float* b_g2;   /* [1] */
  float* rms_w;  /* [d] or NULL */
} fovea_grads;

/* Bytes of workspace fovea_retrieve_fuse_backward needs (0 on bad arguments). */
size_t fovea_retrieve_fuse_backward_workspace(const fovea_ctx* ctx, int32_t B,
                                              int32_t n_nodes_total, int32_t m_max,
                                              int32_t k_max);

/* Backward of one draft step, for training the module (Method, training objective;
 * appendix, draft model training, where the retrieval cardinality is held at K_r = 16):
 * given dL/dh_hat, the gradients of the states, the memory and every per-step weight.
 * The selected sets are a discrete choice and are held fixed: the caller passes the
 * forward's K and idx (fovea_retrieve_fuse's k_out and idx_out, local indices).
 * Requires a context created with dtype FOVEA_F32; all arithmetic is fp32.
 *   params   the raw (unfolded) weights as fp32 device arrays, as given to fovea_create
 *            (the memory-build weights are not read); b_g2 and rms_w as there.
 *   B, mem_off, n_mem_total, m_max, keys, values, node_off, n_nodes_total, t_max, h,
 *   depth    as for fovea_retrieve_fuse (fp32 arrays).
 *   K        [n_nodes_total] int32, idx [n_nodes_total, k_max] int32: the selection
 *            (a node's first K indices must be distinct, as the forward writes them).
 *   dh_hat   [n_nodes_total, d] fp32: dL/dh_hat.
 * Outputs (fp32 device arrays, overwritten):
 *   dh       [n_nodes_total, d]   dL/dh (through the retrieval and the correction).
 *   dkeys, dvalues [n_mem_total, d_m]: dL/dk_i, dL/du_i (zero for unselected rows).
 * Every output is deterministic (fixed summation orders).
 *   grads    the weight gradients (see fovea_grads).
 * Nodes that fail validation (offsets, depth, selection) contribute nothing, get a NaN
 * dh row and set sticky bits read by fovea_last_error.  workspace: at least
 * fovea_retrieve_fuse_backward_workspace(...) bytes, 256-byte aligned; every array
 * 16-byte aligned. */
fovea_status fovea_retrieve_fuse_backward(
    fovea_ctx* ctx, const fovea_params* params, int32_t B, const int64_t* mem_off,
    int64_t n_mem_total, int32_t m_max, const float* keys, const float* values,
    const int32_t* node_off, int32_t n_nodes_total, int32_t t_max, const float* h,
    const int32_t* depth, const int32_t* K, const int32_t* idx, int32_t k_max,
    const float* dh_hat, float* dh, float* dkeys, float* dvalues, const fovea_grads* grads,
    void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace fovea_build_memory_backward needs (0 on bad arguments). */
size_t fovea_build_memory_backward_workspace(const fovea_ctx* ctx, int64_t n_rows);

/* Backward of the memory build (Method, image-specific visual memory; the module is
 * trained end to end): given dL/dkeys and dL/dvalues (e.g. from
 * fovea_retrieve_fuse_backward) for n_rows visual tokens V, the gradients of the
 * projections and the memory LayerNorm, and optionally of V.  fp32 context and
 * arithmetic; deterministic.
 *   params    the raw fp32 weights (W_K, W_U, mem_ln_g, mem_ln_b are read).
 *   V         [n_rows, d_v]; dkeys, dvalues [n_rows, d_m] (fp32, device).
 * Outputs (fp32, device, overwritten): dW_K, dW_U [d_m, d_v], dmem_ln_g, dmem_ln_b [d_v],
 *   dV [n_rows, d_v] or NULL.
 * workspace: fovea_build_memory_backward_workspace(...) bytes, 256-byte aligned. */
fovea_status fovea_build_memory_backward(fovea_ctx* ctx, const fovea_params* params,
                                         int64_t n_rows, const float* V, const float* dkeys,
                                         const float* dvalues, float* dW_K, float* dW_U,
                                         float* dmem_ln_g, float* dmem_ln_b, float* dV,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream);

/* Limits of the candidate extraction below. */
#define FOVEA_LM_MAX_K 16             /* candidates per row */
#define FOVEA_LM_MAX_VOCAB (1 << 24)  /* vocabulary size */
#define FOVEA_LM_MAX_ROWS (1 << 20)   /* rows per call */

/* Bytes of workspace fovea_lm_topk needs for these sizes (0 on bad arguments). */
size_t fovea_lm_topk_workspace(const fovea_ctx* ctx, int32_t n_rows, int32_t vocab, int32_t k);

/* Draft candidates of every corrected state (Eq. hidden_correction's z_n = W_LM h_hat_n
 * and Algorithm 1's expansion step, which adds each node's K_c most likely tokens to the
 * draft tree; K_c = 6 in the experiments):
 *   z_n = W_LM h[n]  over the whole vocabulary, then the k largest entries of z_n.
 *   h        [n_rows, d] storage dtype, device (typically fovea_retrieve_fuse's h_out).
 *   W_LM     [vocab, d] storage dtype, device: the language-model head, [out, in].  Read
 *            in place, not copied; the caller keeps it alive until the call has run.
 *   k        1 <= k <= min(vocab, FOVEA_LM_MAX_K).
 * Outputs (device):
 *   idx_out   [n_rows, k] int32: token ids by descending logit, equal logits by
 *             ascending id.  A NaN logit is never chosen; a slot with nothing left to
 *             choose (every remaining logit NaN) holds -1.
 *   logit_out [n_rows, k] float32 or NULL: the chosen logits (-inf where idx is -1).
 * The logits are accumulated in fp32 and never written to memory.
 * workspace: device memory of at least fovea_lm_topk_workspace(...) bytes, 256-byte
 * aligned, clobbered.  Outputs must not overlap the workspace or each other. */
fovea_status fovea_lm_topk(fovea_ctx* ctx, int32_t n_rows, const void* h, const void* W_LM,
                           int32_t vocab, int32_t k, int32_t* idx_out, float* logit_out,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Synchronise `stream`, read and clear the context's sticky device-data error bits.
 * Returns FOVEA_ERR_DATA if any bit was set (the bits go to *bits if non-NULL),
 * FOVEA_ERR_DEVICE on a HIP error, else FOVEA_OK. */
fovea_status fovea_last_error(fovea_ctx* ctx, hipStream_t stream, uint32_t* bits);

/* Diagnostics: per-kernel timing with HIP events.  While enabled, every kernel that
 * fovea_retrieve_fuse, fovea_build_memory or fovea_lm_topk launches is bracketed by two HIP events on
 * the call's stream (this adds event packets between the kernels, so time whole calls
 * with profiling off).  fovea_profile_read waits for the recorded events, writes up to
 * max_kernels entries (kernel name, summed milliseconds, launch count; names are
 * static strings owned by the library) and forgets what it read.  Returns the number
 * of entries written, or -1 on an error. */
fovea_status fovea_profile(fovea_ctx* ctx, int32_t enable);
int32_t fovea_profile_read(fovea_ctx* ctx, int32_t max_kernels, const char** names,
                           float* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* FOVEA_H_ */
