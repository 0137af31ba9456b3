"""GPU parity on planted exact score ties and on closed-form score profiles.

The rank order breaks equal scores by ascending memory index, so a node's selected set
is unique even when many keys score the same; these cases make the library's tie code
run and check it against the oracle and against closed forms:
  * all keys equal: every score is the same, so K = ceil(tau M) (clamped) and the
    selected entries are the first K indices;
  * a key row duplicated so that its copies straddle the k_max boundary of one node:
    the copies with the lowest indices are kept;
  * geometric scores s_i = -i ln 2 (after a permutation of the entries): the prefix
    masses are (1 - 2^-k) / (1 - 2^-M), so K_raw = ceil(log2(1 / (1 - tau (1 - 2^-M)))).
Each runs through both selection kernels (one wave per node: memories of at most 1024
entries and k_max <= 256; block-wide: larger memories, or k_max above 256), in fp32 and
in bf16 storage.
"""

import math

import numpy as np
import pytest
import torch

import oracle
from parity import compare, dims_of, gpu_outputs, run_oracle, to_device
from synth import WORKLOADS, make_case
from synth.workloads import round_to

pytestmark = pytest.mark.gpu

H_TOL = {"f32": 1e-5, "bf16": 2e-2}

# (memory size, k_max) per selection path
PATHS = {"wave": (200, 64), "wave-kmax256": (300, 256), "block": (1500, 64),
         "block-kmax300": (1500, 300)}


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22883_amd as lib

    assert torch.cuda.is_available()
    return lib


def _base(dtype, **kw):
    base = WORKLOADS["tiny_f32"] if dtype == "f32" else WORKLOADS["llava_b1"].with_(d=512, d_m=256)
    return base.with_(**kw)


def _run(lib, case):
    wl = case.workload
    fv = lib.Fovea(dims_of(wl, case.weights, 1 if wl.dtype == "bf16" else 0), case.weights, device="cuda")
    inp = to_device(case, wl.dtype)
    print(f"[gpu] ties {wl.name}/{wl.dtype}: B={wl.B} n={case.n_nodes} m_max={case.m_max} "
          f"k_max={case.k_max}", flush=True)
    out = fv.retrieve_fuse(inp)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    g = gpu_outputs(out)
    fv.close()
    assert st == 0, f"data error bits {bits:#x}"
    return g


def _exact(case, g, ref, label):
    """Planted ties: the library's sets and order equal the oracle's exactly."""
    rep = {}
    compare(case, g, ref, H_TOL[case.workload.dtype], rep, label=label)
    assert rep["exempt"] == 0 and rep["swapped"] == 0, rep
    assert np.array_equal(g["K"], ref["K"])
    for node in range(case.n_nodes):
        K = int(ref["K"][node])
        assert np.array_equal(g["idx"][node, :K], ref["idx"][node, :K]), node


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("path", list(PATHS))
def test_all_keys_equal(lib, dtype, path):
    """Every key of a request is the same row: K = min(k_max, ceil(tau M)) and the first
    K indices, for a tau below k_max / M and one above it (the threshold itself tied)."""
    M, k_max = PATHS[path]
    taus = np.array([(0.3 * k_max - 0.26) / M, min(0.97, 1.5 * k_max / M + 0.0037)])
    wl = _base(dtype, B=2, T=6, M=M, k_max=k_max, tau=0.5)
    case = make_case(wl, affine="random")
    keys = case.keys.copy()
    for b in range(2):
        m0, m1 = int(case.mem_off[b]), int(case.mem_off[b + 1])
        keys[m0:m1] = keys[m0]
    case.keys = keys
    case.tau = taus.astype(np.float32).astype(np.float64)
    ref = run_oracle(case)
    g = _run(lib, case)
    for b in range(2):
        K = min(k_max, math.ceil(case.tau[b] * M))
        nodes = slice(int(case.node_off[b]), int(case.node_off[b + 1]))
        assert (ref["K"][nodes] == K).all() and (g["K"][nodes] == K).all(), (b, K)
        assert (g["idx"][nodes, :K] == np.arange(K)[None, :]).all()
    _exact(case, g, ref, f"ties: all equal {path} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("path", list(PATHS))
def test_duplicates_straddle_kmax(lib, dtype, path):
    """Copies of one key row sit at ranks k_max - 3 .. k_max + 2 of node 0 (tau high, so
    K = k_max): the tied copies with the lowest indices fill the last places."""
    M, k_max = PATHS[path]
    wl = _base(dtype, B=1, T=4, M=M, k_max=k_max, tau=0.999, key_scale=(4.0, 4.0))
    case = make_case(wl, affine="random")
    q0 = run_oracle(case)["q"][0]
    s0 = oracle.scores(q0[None, :], case.keys)[0]
    order = np.argsort(-s0, kind="stable")
    src = int(order[k_max - 3])
    # six copies at spread indices drawn from entries ranked below k_max + 3
    rng = np.random.default_rng(7)
    pool = order[k_max + 3:]
    dst = rng.choice(pool, size=5, replace=False)
    keys = case.keys.copy()
    keys[dst] = keys[src]
    case.keys = keys
    ref = run_oracle(case)
    s0 = ref["records"][0]["s"]
    order = ref["records"][0]["order"]
    copies = np.sort(np.concatenate([[src], dst]))
    ranks = np.flatnonzero(np.isin(order, copies))
    assert len(ranks) == 6 and ranks[0] < k_max <= ranks[-1], ranks   # the group straddles k_max
    assert np.array_equal(order[ranks], copies)                       # ties by ascending index
    g = _run(lib, case)
    assert g["K"][0] == k_max == ref["K"][0]
    kept = copies[: k_max - ranks[0]]
    assert np.isin(kept, g["idx"][0, :k_max]).all() and not np.isin(copies[len(kept):], g["idx"][0]).any()
    _exact(case, g, ref, f"ties: duplicates at k_max {path} {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("path", ["wave", "block"])
def test_geometric_profile(lib, dtype, path):
    """Scores -i ln 2 over a permutation of the entries; the query is the same for every
    node (zero LayerNorm gain, no depth embedding), so K follows the closed form."""
    M, k_max = PATHS[path]
    M = min(M, 1100) if path == "block" else 64
    wl = _base(dtype, B=1, T=3, M=M, k_max=k_max, tau=0.5)
    case = make_case(wl, affine="random")
    W = dict(case.weights)
    W["q_ln_g"] = np.zeros(wl.d)
    W["E_dep"] = np.zeros_like(W["E_dep"])
    case.weights = W
    q = run_oracle(case)["q"][0]
    perm = np.random.default_rng(11).permutation(M)   # entry perm[i] gets rank i
    target = np.zeros(M)
    target[perm] = -np.arange(M) * math.log(2.0)
    keys = round_to(target[:, None] * math.sqrt(wl.d_m) * q[None, :] / float(q @ q), dtype)
    case.keys = keys
    taus = [0.3, 0.9, 0.999]
    for tau in taus:
        case.tau = np.array([tau], np.float32).astype(np.float64)
        ref = run_oracle(case)
        K_closed = math.ceil(math.log2(1.0 / (1.0 - tau * (1.0 - 2.0 ** -M))))
        assert (ref["K"] == K_closed).all(), (tau, ref["K"], K_closed)
        g = _run(lib, case)
        assert (g["K"] == K_closed).all(), (tau, g["K"])
        assert (g["idx"][:, :K_closed] == perm[None, :K_closed]).all()
        rep = {}
        compare(case, g, ref, H_TOL[dtype], rep, label=f"ties: geometric {path} {dtype} tau={tau}")
        assert rep["exempt"] == 0
