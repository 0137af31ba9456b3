"""GPU parity of the HIP library against the fp64 oracle, through the C ABI.

Every BASELINE workload shape runs at full size with the oracle on the same rounded
inputs; special cases cover the method's degenerate regimes and the error paths.
"""

import math

import numpy as np
import pytest
import torch

from parity import compare, dims_of, gpu_outputs, run_oracle, to_device
from synth import WORKLOADS, make_case, make_memory_case

pytestmark = pytest.mark.gpu

H_TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22883_amd as lib

    assert torch.cuda.is_available()
    return lib


def _ctx(lib, wl, W):
    return lib.Fovea(dims_of(wl, W, 1 if wl.dtype == "bf16" else 0), W, device="cuda")


def _run(lib, case, W=None, fv=None):
    wl = case.workload
    W = case.weights if W is None else W
    own = fv is None
    if own:
        fv = _ctx(lib, wl, W)
    inp = to_device(case, wl.dtype)
    print(f"[gpu] {wl.name}: B={wl.B} n={case.n_nodes} m_max={case.m_max} k_max={case.k_max}", flush=True)
    out = fv.retrieve_fuse(inp)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    g = gpu_outputs(out)
    if own:
        fv.close()
    return g, st, bits


@pytest.mark.parametrize("name,affine", [
    ("tiny_f32", "unit"), ("tiny_f32", "random"), ("llava_b1", "unit"), ("llava_b1", "random"),
    ("batched_b32", "unit"), ("qwen_ragged", "unit"), ("stress_video", "unit"),
    ("paper_llava", "unit"), ("fixed16_b32", "unit")])
def test_workload_parity(lib, name, affine):
    wl = WORKLOADS[name]
    case = make_case(wl, affine=affine)
    g, st, bits = _run(lib, case)
    assert st == 0, f"data error bits {bits:#x}"
    ref = run_oracle(case)
    rep = {}
    compare(case, g, ref, H_TOL[wl.dtype], rep, label=f"{name}/{affine}")
    print(f"[gpu] {name}/{affine}: {rep}", flush=True)
    assert rep["exempt"] <= rep["admissible"]


def _small(dtype="f32", **kw):
    base = WORKLOADS["tiny_f32"] if dtype == "f32" else WORKLOADS["llava_b1"].with_(d=512, d_m=256, T=12, M=200)
    return base.with_(**kw)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_dense_tau_one(lib, dtype):
    wl = _small(dtype, tau=1.0, k_max=256, M=200, key_scale=(3.0, 3.0))
    case = make_case(wl, affine="random")
    g, st, _ = _run(lib, case)
    ref = run_oracle(case)
    assert (g["K"] == 200).all() and (ref["K"] == 200).all()
    compare(case, g, ref, H_TOL[dtype], label=f"dense tau=1 {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_peaked_argmax_exact(lib, dtype):
    wl = _small(dtype, T=5, M=48)
    case = make_case(wl)
    ref0 = run_oracle(case)
    q = ref0["q"]
    target = 11
    direction = q.sum(0) / np.linalg.norm(q.sum(0))
    from synth.workloads import round_to
    keys = case.keys.copy()
    keys[target] = round_to(direction * 4000.0 / math.sqrt(np.abs(direction).max() * len(direction)), dtype)
    case.keys = keys
    case.tau[:] = 0.99
    ref = run_oracle(case)
    assert (ref["K"] == 1).all()
    g, _, _ = _run(lib, case)
    assert (g["K"] == 1).all() and (g["idx"][:, 0] == target).all()
    assert np.array_equal(g["r"], np.repeat(case.values[target][None], case.n_nodes, 0))
    assert np.all(g["mass"] > 0.999)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gate_zero_returns_h_exactly(lib, dtype):
    wl = _small(dtype)
    case = make_case(wl, affine="random")
    W = dict(case.weights, b_g2=-math.inf)
    W.pop("rms_w")
    W["rms_w"] = None
    g, st, _ = _run(lib, case, W=W)
    assert st == 0
    assert (g["gate"] == 0).all()
    assert np.array_equal(g["h_out"], case.h)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [256, 8256])
def test_small_batch_layer2_and_rmsnorm(lib, dtype, d):
    """A few nodes run layer 2 split-K; with the RMSNorm, rows up to 8192 wide take the
    one-pass combine + RMSNorm kernel and wider rows the combine and RMSNorm launches."""
    wl = _small(dtype, d=d)
    case = make_case(wl, affine="random")
    g, st, _ = _run(lib, case)
    assert st == 0
    compare(case, g, run_oracle(case), H_TOL[dtype], label=f"small-batch layer 2 {dtype} d={d}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gate_one_without_rmsnorm(lib, dtype):
    wl = _small(dtype)
    case = make_case(wl, affine="random")
    W = dict(case.weights, b_g2=math.inf, rms_w=None)
    g, st, _ = _run(lib, case, W=W)
    ref = run_oracle(case, weights=W)
    assert (g["gate"] == 1).all()
    compare(case, g, ref, H_TOL[dtype], weights=W, label=f"gate one, no RMSNorm {dtype}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("k_min,k_max", [(16, 16), (32, 256), (0, 1), (3, 7)])
def test_cardinality_bounds(lib, dtype, k_min, k_max):
    wl = _small(dtype, k_min=k_min, k_max=k_max, M=300, tau=0.8)
    case = make_case(wl, affine="random")
    g, _, _ = _run(lib, case)
    ref = run_oracle(case)
    compare(case, g, ref, H_TOL[dtype], label=f"cardinality k_min={k_min} k_max={k_max} {dtype}")
    assert (g["K"] <= k_max).all() and (g["K"] >= min(k_min, 300)).all()


# The header's limits: request memories of FOVEA_MAX_M entries and k_max = FOVEA_MAX_KMAX
# (block-wide selection, candidate sort past 256); the key scale puts K anywhere from a
# few dozen entries to the full k_max.
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_maximum_sizes(lib, dtype):
    max_m, max_k = lib.FOVEA_MAX_M, lib.FOVEA_MAX_KMAX
    wl = WORKLOADS["llava_b1"].with_(dtype=dtype, d=512, d_m=256, B=2, T=6, M=max_m, k_min=0,
                                     k_max=max_k, tau=0.3, tau_hi=0.95, key_scale=(20.0, 20.0))
    case = make_case(wl, affine="random")
    assert case.m_max == max_m
    g, st, bits = _run(lib, case)
    assert st == 0, f"data error bits {bits:#x}"
    ref = run_oracle(case)
    rep = {}
    compare(case, g, ref, H_TOL[dtype], rep, label=f"maximum sizes {dtype}")
    print(f"[gpu] maximum sizes {dtype}: K max {int(g['K'].max())} {rep}", flush=True)
    assert rep["exempt"] <= rep["admissible"]
    assert int(ref["K"].max()) == max_k and int(ref["K"].min()) < 256


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_masked_and_ragged_and_empty(lib, dtype):
    wl = _small(dtype, B=5, M=150, M_lo=1, T=6, valid_frac=0.6, tau=0.9)
    case = make_case(wl, affine="random")
    # request 1: empty memory; request 3: no nodes
    Ms = np.diff(case.mem_off)
    Ms[1] = 0
    keep = np.concatenate([np.arange(case.mem_off[b], case.mem_off[b] + Ms[b]) for b in range(wl.B)])
    case.keys, case.values, case.valid = case.keys[keep], case.values[keep], case.valid[keep]
    case.mem_off = np.concatenate([[0], np.cumsum(Ms)])
    Ts = np.diff(case.node_off)
    Ts[3] = 0
    nkeep = np.concatenate([np.arange(case.node_off[b], case.node_off[b] + Ts[b]) for b in range(wl.B)])
    case.h, case.depth = case.h[nkeep], case.depth[nkeep]
    case.node_off = np.concatenate([[0], np.cumsum(Ts)]).astype(np.int32)
    g, st, bits = _run(lib, case)
    assert st == 0, bits
    ref = run_oracle(case)
    compare(case, g, ref, H_TOL[dtype], label=f"masked, ragged, empty {dtype}")
    b1 = slice(case.node_off[1], case.node_off[2])
    assert (g["K"][b1] == 0).all() and (g["r"][b1] == 0).all()
    for node in range(case.n_nodes):
        b = np.searchsorted(case.node_off, node, side="right") - 1
        sel = g["idx"][node, :g["K"][node]]
        assert case.valid[case.mem_off[b] + sel].all()


# No draft nodes at all (every request's node range empty): the call succeeds and
# launches nothing; a later call on the same context is unaffected.
def test_no_nodes_at_all(lib):
    wl = _small("bf16", B=2, T=3)
    case = make_case(wl)
    fv = _ctx(lib, wl, case.weights)
    inp = to_device(case, "bf16")
    empty = dict(inp, node_off=torch.zeros(wl.B + 1, dtype=torch.int32, device="cuda"),
                 h=inp["h"][:0].contiguous(), depth=inp["depth"][:0].contiguous())
    out = fv.retrieve_fuse(empty)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    assert st == 0, bits
    assert out.h_out.shape[0] == 0
    g, st, bits = _run(lib, case, fv=fv)
    assert st == 0, bits
    compare(case, g, run_oracle(case), H_TOL["bf16"], label="after an empty call")
    fv.close()


@pytest.mark.parametrize("dtype,rows", [("f32", 333), ("bf16", 333), ("bf16", 16400)])
def test_build_memory(lib, dtype, rows):
    # 333 rows: 128-row tiles; 16400 bf16 rows with d_m = 256: 65 x 4 tiles of 256 rows, the last
    # row tile ragged
    wl = _small(dtype)
    V, W = make_memory_case(wl, rows, affine="random")
    import oracle
    fv = _ctx(lib, wl, W)
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    Vt = torch.tensor(V, dtype=dt, device="cuda")
    keys, values = fv.build_memory(Vt)
    torch.cuda.synchronize()
    fv.close()
    kr, vr = oracle.build_memory(V, W["mem_ln_g"], W["mem_ln_b"], W["W_K"], W["W_U"], W["ln_eps"],
                                 gain_rounding="bf16" if dtype == "bf16" else None)
    tol = 1e-5 if dtype == "f32" else 1e-2
    for got, ref in ((keys, kr), (values, vr)):
        got = got.double().cpu().numpy()
        rel = np.linalg.norm(got - ref, axis=1) / np.linalg.norm(ref, axis=1)
        assert rel.max() <= tol, rel.max()


# Repeated calls give bit-identical outputs on every path: split-K GEMMs with their
# combines (one request), whole-tile GEMMs and two nodes per selection block (batched),
# the block-wide selection (ragged memories of up to 4096 rows), the bitonic candidate
# sort (k_max 256) and the fixed-cardinality path.  Every output is compared, and the
# workspace is reused between the calls (its contents need no initialisation).
@pytest.mark.parametrize("name", ["llava_b1", "batched_b32", "qwen_ragged", "paper_llava", "fixed16_b32"])
def test_determinism(lib, name):
    wl = WORKLOADS[name]
    case = make_case(wl)
    fv = _ctx(lib, wl, case.weights)
    inp = to_device(case, wl.dtype)
    first = fv.retrieve_fuse(inp)
    ref = {f: getattr(first, f).clone() for f in ("h_out", "k", "idx", "gate", "mass", "r")}
    for _ in range(2):
        again = fv.retrieve_fuse(inp)
        torch.cuda.synchronize()
        for f, v in ref.items():
            assert torch.equal(v, getattr(again, f)), (name, f)
    fv.close()


def test_data_errors_flag_and_nan(lib):
    wl = _small("f32", B=3, T=4, M=40)
    case = make_case(wl)
    fv = _ctx(lib, wl, case.weights)
    inp = to_device(case, "f32")
    inp["depth"][1] = 99          # bad depth on node 1
    inp["tau"][2] = 1.5           # bad tau on request 2
    out = fv.retrieve_fuse(inp)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    assert st == lib.FOVEA_ERR_DATA
    assert bits & lib.FOVEA_DATA_BAD_DEPTH and bits & lib.FOVEA_DATA_BAD_TAU
    h = out.h_out.cpu()
    assert torch.isnan(h[1]).all() and torch.isnan(h[8:12]).all()
    assert torch.isfinite(h[0]).all() and torch.isfinite(h[4:8]).all()
    st, bits = lib.fovea_last_error(fv.ctx)
    assert st == 0 and bits == 0   # read clears
    # bad memory offsets: request 1 claims more than m_max entries
    inp = to_device(case, "f32")
    inp["mem_off"][2] = inp["mem_off"][3]
    inp["m_max"] = 40
    out = fv.retrieve_fuse(inp)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    assert st == lib.FOVEA_ERR_DATA and bits & lib.FOVEA_DATA_BAD_MEM_OFFSETS
    fv.close()


def test_host_argument_errors(lib):
    wl = _small("f32")
    case = make_case(wl)
    fv = _ctx(lib, wl, case.weights)
    inp = to_device(case, "f32")
    with pytest.raises(lib.FoveaError) as e:
        fv.retrieve_fuse(dict(inp, k_min=5, k_max=4))
    assert e.value.status == lib.FOVEA_ERR_INVALID_ARG
    with pytest.raises(lib.FoveaError) as e:
        fv.retrieve_fuse(dict(inp, k_max=2048))
    assert e.value.status == lib.FOVEA_ERR_UNSUPPORTED
    out = fv.alloc_outputs(case.n_nodes, case.k_max, wl.d, wl.d_m)
    ws = fv.ensure_workspace(case.workload.B, case.n_nodes, case.n_mem, case.m_max, case.k_max)
    with pytest.raises(lib.FoveaError) as e:   # workspace too small
        lib.fovea_retrieve_fuse(fv.ctx, 1, inp["mem_off"], case.n_mem, case.m_max, inp["keys"],
                                inp["values"], None, inp["node_off"], case.n_nodes, case.t_max,
                                inp["h"], inp["depth"], inp["tau"], 1, 16, out.h_out,
                                workspace=ws[:256])
    assert e.value.status == lib.FOVEA_ERR_WORKSPACE
    with pytest.raises(lib.FoveaError) as e:   # output aliases the input
        lib.fovea_retrieve_fuse(fv.ctx, 1, inp["mem_off"], case.n_mem, case.m_max, inp["keys"],
                                inp["values"], None, inp["node_off"], case.n_nodes, case.t_max,
                                inp["h"], inp["depth"], inp["tau"], 1, 16, inp["h"], workspace=ws)
    assert e.value.status == lib.FOVEA_ERR_INVALID_ARG
    fv.close()


@pytest.mark.parametrize("B,M,d_m,M_lo", [(32, 576, 1024, None), (40, 576, 1024, None),
                                          (3, 130, 384, None), (5, 700, 896, None),
                                          (2, 576, 1024, None), (2, 576, 1024, 64)],
                         ids=["80-key-blocks", "96-key-blocks", "fallback-d384", "64-key-blocks-d896",
                              "2-k-slices", "k-slices-ragged-spread"])
def test_score_tilings(lib, B, M, d_m, M_lo):
    """Each score-kernel tiling (keys per block chosen from the grid size), the
    unpipelined fallback, d_m split in k slices (two requests: 72 blocks, two slices)
    and, for ragged memories, tiles spread over the XCDs agree with the oracle."""
    extra = {} if M_lo is None else dict(M_lo=M_lo)
    wl = WORKLOADS["llava_b1"].with_(B=B, M=M, d=512, d_m=d_m, T=5, tau=0.7, tau_hi=0.95,
                                     key_scale=(40.0, 200.0), **extra)
    case = make_case(wl, affine="random")
    g, st, _ = _run(lib, case)
    assert st == 0
    compare(case, g, run_oracle(case), H_TOL["bf16"], label=f"score tiling B={B} M={M} d_m={d_m}")
