"""Seeded synthetic workloads shaped like the paper's LLaVA- and Qwen-VL-class draft steps.

No trained weights, images or benchmark items are used or reproduced: every array is
drawn from a NumPy PCG64 generator in float64 and rounded once to the storage dtype,
and both the oracle and the library consume exactly those rounded values.

Recipe (per workload):
  * weights ~ N(0, 1/fan_in); LayerNorm gains 1 and biases 0 ("unit" affine) or
    gains 1 + N(0, 0.1^2) and biases N(0, 0.1^2) ("random" affine, used by parity
    tests to exercise every term); E_dep ~ N(0, 0.25); correction biases 0 (or
    N(0, 0.1^2)), gate output bias -2; RMSNorm weight 1 (or 1 + N(0, 0.1^2)).
  * hidden states h ~ N(0, 1).
  * depth of node j in a request follows a draft tree of width 6: the root at depth 0,
    the next six nodes at depth 1, the rest spread evenly over depths 2..6.
  * memory keys k_i = a_b * beta_i * (mu_{c(i)} + eps_i) and values
    u_i = nu_{c(i)} + eta_i: cluster centres carry ``cluster_share`` of the per-element
    variance 1/d_m, the noise the rest; a fraction of entries gets a norm boost beta_i;
    a_b is the per-request key scale, which plays the role of the query temperature
    (LayerNorm cancels any scale on h).  Clusters are 4x4 spatial blocks of the patch
    grid when M is a square, shared across frames (with jitter) for multi-frame
    memories, and random otherwise.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np

__all__ = ["Workload", "Case", "WORKLOADS", "make_weights", "make_case", "make_memory_case",
           "round_to"]


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                      # storage dtype: "f32" or "bf16"
    B: int                          # requests
    T: int                          # draft-tree nodes per request
    M: int                          # memory entries per request (upper bound if ragged)
    d: int                          # drafter hidden size
    d_m: int                        # key / value width
    k_max: int
    tau: float                      # mass threshold (lower bound if tau_hi is set)
    seed: int
    M_lo: int | None = None         # ragged memories: M_b ~ U{M_lo..M}
    tau_hi: float | None = None     # tau_b ~ U[tau, tau_hi]
    k_min: int = 1
    d_c: int = 512                  # correction / gate hidden width
    n_depth: int = 7                # depths 0..6
    n_clusters: int = 16
    cluster_share: float = 0.5
    key_scale: tuple = (1.0, 1.0)   # per-request key scale a_b, log-uniform in [lo, hi]
    key_scale_split: tuple | None = None  # (flat, peaked): first half / second half of requests
    boost_frac: float = 0.0
    boost: float = 1.0
    frames: int = 1
    valid_frac: float = 1.0         # fraction of memory entries marked valid (1: no mask)
    description: str = ""

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS: dict[str, Workload] = {
    "tiny_f32": Workload(
        name="tiny_f32", dtype="f32", B=1, T=4, M=64, d=256, d_m=128, k_max=16, tau=0.9,
        seed=20260000, n_clusters=4, key_scale=(30.0, 30.0),
        description="tiny oracle case: B=1, T=4, M=64, d=256, d_m=128, fp32"),
    "llava_b1": Workload(
        name="llava_b1", dtype="bf16", B=1, T=60, M=576, d=4096, d_m=1024, k_max=64, tau=0.8,
        seed=20260001, key_scale=(60.0, 60.0), boost_frac=0.10, boost=2.0,
        description="LLaVA-1.5-7B shape: B=1, T=60, M=576 (24x24), d=4096, d_m=1024"),
    "batched_b32": Workload(
        name="batched_b32", dtype="bf16", B=32, T=60, M=576, d=4096, d_m=1024, k_max=64,
        tau=0.6, tau_hi=0.95, seed=20260002, key_scale=(35.0, 250.0), boost_frac=0.10,
        boost=1.5,
        description="batched serving: B=32, T=60, M=576 each, d=4096, d_m=1024"),
    "qwen_ragged": Workload(
        name="qwen_ragged", dtype="bf16", B=16, T=48, M=4096, M_lo=256, d=3584, d_m=896,
        k_max=128, tau=0.85, seed=20260003, key_scale=(70.0, 70.0), boost_frac=0.10,
        boost=2.0,
        description="Qwen2.5-VL-7B shape, ragged: B=16, M_b in 256..4096, d=3584, d_m=896, T=48"),
    "stress_video": Workload(
        name="stress_video", dtype="bf16", B=8, T=64, M=16384, d=5120, d_m=1280, k_max=256,
        tau=0.9, seed=20260004, key_scale_split=(8.0, 2000.0), frames=16,
        description="high-res / video stress: B=8, M=16384 (16 frames x 1024), d=5120, d_m=1280"),
    # the paper's own cardinality settings (Method: tau = 0.8, K_min = 32, K_max = 256,
    # key/value width equal to the hidden size) and its fixed-K ablation (K_r = 16)
    "paper_llava": Workload(
        name="paper_llava", dtype="bf16", B=1, T=60, M=576, d=4096, d_m=4096, k_min=32,
        k_max=256, tau=0.8, seed=20260005, key_scale=(80.0, 80.0), boost_frac=0.10,
        boost=2.0,
        description="paper preset on the LLaVA-1.5-7B shape: tau=0.8, K_min=32, K_max=256, "
                    "d_m=d=4096, B=1, T=60, M=576"),
    "fixed16_b32": Workload(
        name="fixed16_b32", dtype="bf16", B=32, T=60, M=576, d=4096, d_m=1024, k_min=16,
        k_max=16, tau=0.6, tau_hi=0.95, seed=20260006, key_scale=(35.0, 250.0),
        boost_frac=0.10, boost=1.5,
        description="fixed cardinality K=16 on the batched shape: B=32, T=60, M=576, "
                    "d=4096, d_m=1024"),
}


@dataclass
class Case:
    workload: Workload
    weights: dict
    mem_off: np.ndarray     # int64 [B+1]
    keys: np.ndarray        # [n_mem, d_m] fp64 holding dtype-exact values
    values: np.ndarray
    valid: np.ndarray | None  # bool [n_mem] or None (all valid)
    node_off: np.ndarray    # int32 [B+1]
    h: np.ndarray           # [n, d]
    depth: np.ndarray       # int32 [n]
    tau: np.ndarray         # fp64 [B], float32-exact
    k_min: int
    k_max: int

    @property
    def n_nodes(self) -> int:
        return int(self.node_off[-1])

    @property
    def n_mem(self) -> int:
        return int(self.mem_off[-1])

    @property
    def m_max(self) -> int:
        return int(np.max(np.diff(self.mem_off))) if len(self.mem_off) > 1 else 0

    @property
    def t_max(self) -> int:
        return int(np.max(np.diff(self.node_off))) if len(self.node_off) > 1 else 0


def round_to(x, dtype: str) -> np.ndarray:
    """Round float64 values once to the storage dtype and return them as float64."""
    x = np.asarray(x, np.float64)
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        import torch

        t = torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16)
        return t.to(torch.float64).numpy()
    raise ValueError(dtype)


def _normal(rng, shape, std, dtype):
    return round_to(rng.standard_normal(shape) * std, dtype)


def make_weights(wl: Workload, seed: int | None = None, affine: str = "unit") -> dict:
    """All parameters of the retrieval + correction path and of the memory build."""
    rng = np.random.Generator(np.random.PCG64(wl.seed + 7919 if seed is None else seed))
    d, d_m, d_c, dt = wl.d, wl.d_m, wl.d_c, wl.dtype
    rnd = affine == "random"

    def gain(n):
        return round_to(1.0 + 0.1 * rng.standard_normal(n), dt) if rnd else np.ones(n)

    def bias(n):
        return _normal(rng, n, 0.1, dt) if rnd else np.zeros(n)

    W = dict(
        q_ln_g=gain(d), q_ln_b=bias(d),
        E_dep=_normal(rng, (wl.n_depth, d), 0.5, dt),
        W_Q=_normal(rng, (d_m, d), 1.0 / math.sqrt(d), dt),
        W_c1=_normal(rng, (d_c, d + d_m), 1.0 / math.sqrt(d + d_m), dt), b_c1=bias(d_c),
        W_c2=_normal(rng, (d, d_c), 1.0 / math.sqrt(d_c), dt), b_c2=bias(d),
        W_g1=_normal(rng, (d_c, d + d_m), 1.0 / math.sqrt(d + d_m), dt), b_g1=bias(d_c),
        w_g2=_normal(rng, d_c, 1.0 / math.sqrt(d_c), dt),
        b_g2=float(np.float32(-2.0)),
        rms_w=gain(d),
        mem_ln_g=gain(d), mem_ln_b=bias(d),
        W_K=_normal(rng, (d_m, d), 1.0 / math.sqrt(d), dt),
        W_U=_normal(rng, (d_m, d), 1.0 / math.sqrt(d), dt),
        ln_eps=1e-5, rms_eps=1e-6,
    )
    return W


def _depths(T: int) -> np.ndarray:
    j = np.arange(T)
    dep = np.where(j == 0, 0, 1)
    if T > 7:
        rest = j >= 7
        dep = np.where(rest, 2 + ((j - 7) * 5) // max(T - 7, 1), dep)
    return dep.astype(np.int32)


def _clusters(rng, M: int, n_clusters: int, frames: int) -> np.ndarray:
    per = M // frames
    side = int(round(math.sqrt(per)))
    if side * side == per and n_clusters == 16 and side % 4 == 0:
        i = np.arange(per)
        row, col = i // side, i % side
        c = (row * 4 // side) * 4 + (col * 4 // side)
        return np.tile(c, frames)
    if frames == 1:
        return np.arange(M) % n_clusters if n_clusters < 8 else rng.integers(0, n_clusters, M)
    return np.tile(rng.integers(0, n_clusters, per), frames)


def make_case(wl: Workload, seed: int | None = None, affine: str = "unit",
              weights: dict | None = None) -> Case:
    """One seeded draft-step batch for workload ``wl``."""
    seed = wl.seed if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    W = make_weights(wl, seed + 7919, affine) if weights is None else weights
    B, T, d, d_m, dt = wl.B, wl.T, wl.d, wl.d_m, wl.dtype

    if wl.M_lo is None:
        Ms = np.full(B, wl.M, np.int64)
    else:
        Ms = rng.integers(wl.M_lo, wl.M + 1, B).astype(np.int64)
    mem_off = np.concatenate([[0], np.cumsum(Ms)]).astype(np.int64)
    node_off = (np.arange(B + 1) * T).astype(np.int32)

    if wl.key_scale_split is not None:
        flat, peaked = wl.key_scale_split
        scales = np.where(np.arange(B) < (B + 1) // 2, flat, peaked).astype(np.float64)
    else:
        lo, hi = wl.key_scale
        scales = np.exp(rng.uniform(math.log(lo), math.log(hi), B))
    if wl.tau_hi is None:
        tau = np.full(B, wl.tau)
    else:
        tau = rng.uniform(wl.tau, wl.tau_hi, B)
    tau = tau.astype(np.float32).astype(np.float64)

    keys, values = [], []
    sc = math.sqrt(wl.cluster_share / d_m)
    sn = math.sqrt((1.0 - wl.cluster_share) / d_m)
    for b in range(B):
        M = int(Ms[b])
        c = _clusters(rng, M, wl.n_clusters, wl.frames)
        mu = rng.standard_normal((wl.n_clusters, d_m)) * sc
        nu = rng.standard_normal((wl.n_clusters, d_m)) * sc
        kb = mu[c] + rng.standard_normal((M, d_m)) * sn
        ub = nu[c] + rng.standard_normal((M, d_m)) * sn
        if wl.frames > 1:  # per-frame jitter of the shared centres
            f = np.repeat(np.arange(wl.frames), M // wl.frames)
            jit = rng.standard_normal((wl.frames, wl.n_clusters, d_m)) * (0.3 * sc)
            kb += jit[f, c]
        beta = np.ones(M)
        if wl.boost_frac > 0:
            beta[rng.random(M) < wl.boost_frac] = wl.boost
        keys.append(kb * (scales[b] * beta)[:, None])
        values.append(ub)
    keys = round_to(np.concatenate(keys) if keys else np.zeros((0, d_m)), dt)
    values = round_to(np.concatenate(values) if values else np.zeros((0, d_m)), dt)
    valid = None
    if wl.valid_frac < 1.0:
        valid = rng.random(int(mem_off[-1])) < wl.valid_frac

    h = _normal(rng, (B * T, d), 1.0, dt)
    depth = np.tile(_depths(T), B)
    return Case(workload=wl, weights=W, mem_off=mem_off, keys=keys, values=values, valid=valid,
                node_off=node_off, h=h, depth=depth, tau=tau, k_min=wl.k_min, k_max=wl.k_max)


def make_memory_case(wl: Workload, n_rows: int, seed: int | None = None, affine: str = "unit",
                     weights: dict | None = None):
    """Projected visual tokens V ~ N(0, 1) of width d for the one-off memory build."""
    seed = wl.seed + 104729 if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    W = make_weights(wl, seed + 7919, affine) if weights is None else weights
    V = _normal(rng, (n_rows, wl.d), 1.0, wl.dtype)
    return V, W


# Language-model heads of the drafters the paper evaluates: LLaVA-NeXT-7B's Vicuna head
# (vocabulary 32000, hidden 4096) and Qwen2.5-VL-7B's (vocabulary 152064, hidden 3584).
LM_HEADS = {
    "vicuna7b": dict(vocab=32000, d=4096),
    "qwen2_5_7b": dict(vocab=152064, d=3584),
}


def make_lm_case(n: int, d: int, vocab: int, dtype: str, seed: int):
    """Corrected states h ~ N(0, 1) (unit RMS, as after the RMSNorm) and a head
    W_LM ~ N(0, 1/d), so that logits are of unit scale.  Both rounded once to the
    storage dtype; returned as float64."""
    rng = np.random.Generator(np.random.PCG64(seed))
    h = _normal(rng, (n, d), 1.0, dtype)
    W = _normal(rng, (vocab, d), 1.0 / math.sqrt(d), dtype)
    return h, W


def make_output_grad(n: int, d: int, seed: int) -> np.ndarray:
    """dL/dh_hat for the backward: N(0, 1), fp32-exact, returned as float64."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return round_to(rng.standard_normal((n, d)), "f32")
