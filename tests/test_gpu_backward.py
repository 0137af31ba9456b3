"""GPU parity of the backward (fovea_retrieve_fuse_backward) against the fp64 oracle's
retrieve_fuse_backward, through the C ABI.  The selection both sides hold fixed is the
oracle forward's own (an input of the backward)."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
from parity import dims_of, to_device
from synth import WORKLOADS, make_case, make_output_grad

pytestmark = pytest.mark.gpu

GRADS = ["dh", "dkeys", "dvalues", "dW_Q", "dq_ln_g", "dq_ln_b", "dE_dep", "dW_c1", "db_c1",
         "dW_c2", "db_c2", "dW_g1", "db_g1", "dw_g2", "db_g2", "drms_w"]
TOL = 2e-4  # fp32 recompute + fp32 GEMMs (K <= 4096 or the node count) against fp64


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22883_amd as lib

    assert torch.cuda.is_available()
    return lib


def _wl(name, **kw):
    return WORKLOADS[name].with_(dtype="f32", **kw)


def _run(lib, case, no_rms=False):
    wl = case.workload
    W = dict(case.weights)
    if no_rms:
        W.pop("rms_w")
    ref_f = oracle.retrieve_fuse(W, case.mem_off, case.keys, case.values, case.valid,
                                 case.node_off, case.h, case.depth, case.tau, case.k_min,
                                 case.k_max)
    dh_hat = make_output_grad(case.n_nodes, wl.d, wl.seed + 17)
    ref = oracle.retrieve_fuse_backward(W, case.mem_off, case.keys, case.values, case.node_off,
                                        case.h, case.depth, ref_f["idx"], ref_f["K"], dh_hat)
    fv = lib.Fovea(dims_of(wl, W, 0), W, device="cuda")
    inp = to_device(case, "f32")
    K = torch.tensor(ref_f["K"], dtype=torch.int32, device="cuda")
    idx = torch.tensor(ref_f["idx"], dtype=torch.int32, device="cuda")
    print(f"[gpu] backward {wl.name}: B={wl.B} n={case.n_nodes} m_max={case.m_max} "
          f"k_max={case.k_max} d={wl.d} d_m={wl.d_m}", flush=True)
    g = fv.retrieve_fuse_backward(inp, K, idx, torch.tensor(dh_hat, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    fv.close()
    out = {k: v.double().cpu().numpy() for k, v in g.items()}
    if "db_g2" in out:
        out["db_g2"] = out["db_g2"][0]
    return out, ref, st, bits, ref_f


def _compare(out, ref, tol=TOL):
    for k in GRADS:
        if ref.get(k) is None:
            assert k not in out, k
            continue
        r = np.asarray(ref[k])
        o = np.asarray(out[k]).reshape(r.shape)
        scale = max(float(np.abs(r).max()), 1e-30)
        err = float(np.abs(o - r).max()) / scale
        assert err <= tol, f"{k}: max error {err:.2e} of max |ref| {scale:.3e}"


@pytest.mark.parametrize("name,kw,affine", [
    ("tiny_f32", {}, "random"),
    ("qwen_ragged", dict(B=4, T=16, M=300, M_lo=64, d=512, d_m=256, k_max=32), "random"),
    ("llava_b1", {}, "unit"),
    ("fixed16_b32", dict(B=3, T=20), "random"),  # the paper trains with K_r fixed at 16
])
def test_backward_parity(lib, name, kw, affine):
    case = make_case(_wl(name, **kw), affine=affine)
    out, ref, st, bits, ref_f = _run(lib, case)
    assert st == 0, f"data error bits {bits:#x}"
    assert ref_f["K"].max() > 1
    _compare(out, ref)


def test_backward_many_depths(lib):
    # 27 depths: the depth-embedding sums take four column-sum jobs of at most eight depths,
    # and the backward's column sums more jobs than one launch carries
    case = make_case(_wl("tiny_f32", B=2, T=60, n_depth=27), affine="random")
    case.depth = ((np.arange(case.n_nodes) * 5) % 27).astype(np.int32)
    out, ref, st, bits, _ = _run(lib, case)
    assert st == 0, f"data error bits {bits:#x}"
    assert np.count_nonzero(np.abs(ref["dE_dep"]).sum(axis=1)) == 27
    _compare(out, ref)


def test_backward_memory_rows_outside_every_request(lib):
    # 5 memory rows before the first request and 3 after the last: their gradients are zero
    case = make_case(_wl("tiny_f32", B=2, T=9, M=100), affine="random")
    rng = np.random.default_rng(5)

    def pad(x):
        lead = rng.standard_normal((5, x.shape[1])).astype(np.float32).astype(np.float64)
        tail = rng.standard_normal((3, x.shape[1])).astype(np.float32).astype(np.float64)
        return np.concatenate([lead, x, tail])

    case = dataclasses.replace(case, keys=pad(case.keys), values=pad(case.values),
                               mem_off=case.mem_off + 5)
    # NaN-filled blocks of the outputs' size, freed so that the outputs likely reuse them
    junk = [torch.full((case.keys.shape[0], case.workload.d_m), float("nan"), device="cuda")
            for _ in range(4)]
    del junk
    out, ref, st, bits, _ = _run(lib, case)
    assert st == 0, f"data error bits {bits:#x}"
    for k in ("dkeys", "dvalues"):
        assert np.all(out[k][:5] == 0) and np.all(out[k][-3:] == 0), k
    _compare(out, ref)


def test_backward_without_rmsnorm(lib):
    case = make_case(_wl("tiny_f32", T=9, M=100), affine="random")
    out, ref, st, bits, _ = _run(lib, case, no_rms=True)
    assert st == 0
    assert ref["drms_w"] is None
    _compare(out, ref)


def test_backward_bad_selection_flags_and_skips_the_node(lib):
    case = make_case(_wl("tiny_f32", T=6), affine="unit")
    wl = case.workload
    W = case.weights
    ref_f = oracle.retrieve_fuse(W, case.mem_off, case.keys, case.values, case.valid,
                                 case.node_off, case.h, case.depth, case.tau, case.k_min,
                                 case.k_max)
    idx = ref_f["idx"].copy()
    idx[2, 0] = case.m_max + 5  # outside the request's memory
    fv = lib.Fovea(dims_of(wl, W, 0), W, device="cuda")
    inp = to_device(case, "f32")
    dh_hat = torch.tensor(make_output_grad(case.n_nodes, wl.d, 3), dtype=torch.float32, device="cuda")
    print(f"[gpu] backward bad selection n={case.n_nodes}", flush=True)
    g = fv.retrieve_fuse_backward(inp, torch.tensor(ref_f["K"], dtype=torch.int32, device="cuda"),
                                  torch.tensor(idx, dtype=torch.int32, device="cuda"), dh_hat)
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    fv.close()
    assert st == lib.FOVEA_ERR_DATA and bits & lib.FOVEA_DATA_BAD_SELECTION
    dh = g["dh"].cpu().numpy()
    assert np.all(np.isnan(dh[2])) and np.all(np.isfinite(np.delete(dh, 2, axis=0)))
    for k, v in g.items():
        if k != "dh":
            assert torch.isfinite(v).all(), k


def test_backward_host_errors(lib):
    wl = WORKLOADS["tiny_f32"]
    case = make_case(wl)
    fvb = lib.Fovea(dims_of(wl, case.weights, 1), case.weights, device="cuda")  # bf16 context
    inp = to_device(case, "f32")
    n = case.n_nodes
    K = torch.ones(n, dtype=torch.int32, device="cuda")
    idx = torch.zeros(n, case.k_max, dtype=torch.int32, device="cuda")
    dh_hat = torch.zeros(n, wl.d, dtype=torch.float32, device="cuda")
    print("[gpu] backward host errors", flush=True)
    p32 = {k: v.float() for k, v in fvb.params.items()}
    shapes = dict(W_Q=(wl.d_m, wl.d), q_ln_g=(wl.d,), q_ln_b=(wl.d,), E_dep=(wl.n_depth, wl.d),
                  W_c1=(wl.d_c, wl.d + wl.d_m), b_c1=(wl.d_c,), W_c2=(wl.d, wl.d_c), b_c2=(wl.d,),
                  W_g1=(wl.d_c, wl.d + wl.d_m), b_g1=(wl.d_c,), w_g2=(wl.d_c,), b_g2=(1,),
                  rms_w=(wl.d,))
    grads = {k: torch.empty(v, dtype=torch.float32, device="cuda") for k, v in shapes.items()}
    n_mem = case.n_mem
    out = [torch.empty(n, wl.d, device="cuda"), torch.empty(n_mem, wl.d_m, device="cuda"),
           torch.empty(n_mem, wl.d_m, device="cuda")]
    ws = torch.empty(1 << 24, dtype=torch.uint8, device="cuda")

    def call(ctx, **over):
        a = dict(params=p32, grads=grads)
        a.update(over)
        lib.fovea_retrieve_fuse_backward(
            ctx, a["params"], -2.0, 1, inp["mem_off"], n_mem, case.m_max, inp["keys"],
            inp["values"], inp["node_off"], n, case.t_max, inp["h"], inp["depth"], K, idx,
            case.k_max, dh_hat, *out, a["grads"], ws)

    with pytest.raises(lib.FoveaError) as e:  # the backward needs an fp32 context
        call(fvb.ctx)
    assert e.value.status == lib.FOVEA_ERR_UNSUPPORTED
    fvb.close()
    fv = lib.Fovea(dims_of(wl, case.weights, 0), case.weights, device="cuda")
    for bad in (dict(grads={k: v for k, v in grads.items() if k != "W_c2"}),  # a missing output
                dict(grads={k: v for k, v in grads.items() if k != "rms_w"})):  # rms_w mismatch
        with pytest.raises(lib.FoveaError) as e:
            call(fv.ctx, **bad)
        assert e.value.status == lib.FOVEA_ERR_INVALID_ARG
    with pytest.raises(lib.FoveaError) as e:  # workspace too small
        lib.fovea_retrieve_fuse_backward(
            fv.ctx, p32, -2.0, 1, inp["mem_off"], n_mem, case.m_max, inp["keys"], inp["values"],
            inp["node_off"], n, case.t_max, inp["h"], inp["depth"], K, idx, case.k_max, dh_hat,
            *out, grads, ws[:1024])
    assert e.value.status == lib.FOVEA_ERR_WORKSPACE
    fv.close()
    assert lib.fovea_retrieve_fuse_backward_workspace(None, 1, n, case.m_max, case.k_max) == 0


def test_backward_no_nodes_gives_zero_gradients(lib):
    wl = _wl("tiny_f32")
    case = make_case(wl)
    fv = lib.Fovea(dims_of(wl, case.weights, 0), case.weights, device="cuda")
    inp = to_device(case, "f32")
    inp["h"] = inp["h"][:0]
    inp["node_off"] = torch.zeros_like(inp["node_off"])
    print("[gpu] backward with no nodes", flush=True)
    g = fv.retrieve_fuse_backward(inp, torch.zeros(0, dtype=torch.int32, device="cuda"),
                                  torch.zeros(0, case.k_max, dtype=torch.int32, device="cuda"),
                                  torch.zeros(0, wl.d, dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    fv.close()
    for k, v in g.items():
        assert v.numel() == 0 or float(v.abs().max()) == 0.0, k


@pytest.mark.parametrize("name,n_rows,affine", [("tiny_f32", 64, "random"), ("llava_b1", 576, "random"),
                                               ("tiny_f32", 130, "unit")])
def test_memory_backward_parity(lib, name, n_rows, affine):
    from synth import make_memory_case

    wl = _wl(name)
    V, W = make_memory_case(wl, n_rows, affine=affine)
    dk = make_output_grad(n_rows, wl.d_m, wl.seed + 5)
    du = make_output_grad(n_rows, wl.d_m, wl.seed + 6)
    ref = oracle.build_memory_backward(V, W["mem_ln_g"], W["mem_ln_b"], W["W_K"], W["W_U"],
                                       W["ln_eps"], dk, du)
    fv = lib.Fovea(dims_of(wl, W, 0), W, device="cuda")
    t = lambda x: torch.tensor(x, dtype=torch.float32, device="cuda")  # noqa: E731
    print(f"[gpu] memory backward {name}: rows={n_rows} d_v={wl.d} d_m={wl.d_m}", flush=True)
    g = fv.build_memory_backward(t(V), t(dk), t(du))
    torch.cuda.synchronize()
    st, bits = lib.fovea_last_error(fv.ctx)
    fv.close()
    assert st == 0, f"data error bits {bits:#x}"
    for k in ("dW_K", "dW_U", "dmem_ln_g", "dmem_ln_b", "dV"):
        r = np.asarray(ref[k])
        o = g[k].double().cpu().numpy().reshape(r.shape)
        err = float(np.abs(o - r).max()) / max(float(np.abs(r).max()), 1e-30)
        assert err <= TOL, f"{k}: max error {err:.2e}"
