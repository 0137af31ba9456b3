"""GPU parity of the LM head + draft-candidate extraction (fovea_lm_topk) against the
fp64 oracle, through the C ABI.

The logits are compared at the chosen ids; the chosen ids must be the oracle's exactly
wherever the oracle's ranking is decided by more than the tolerance, and elsewhere the
q-th chosen logit must equal the oracle's q-th largest within the tolerance.
"""

import numpy as np
import pytest
import torch

import oracle
from parity import dims_of
from synth import LM_HEADS, WORKLOADS, make_lm_case, make_weights

pytestmark = pytest.mark.gpu

# fp32 accumulation of dtype-exact products over d <= 4096 terms of unit-scale logits
Z_TOL = 1e-4


@pytest.fixture(scope="module")
def lib():
    import paper_2608_22883_amd as lib

    assert torch.cuda.is_available()
    return lib


_CTX = {}


def _ctx(lib, dtype: str, d: int):
    """A context whose hidden size is d (the head only uses the context's dtype and d)."""
    key = (dtype, d)
    if key not in _CTX:
        wl = WORKLOADS["tiny_f32"] if dtype == "f32" else WORKLOADS["llava_b1"]
        import dataclasses

        wl = dataclasses.replace(wl, d=d, d_m=64, dtype=dtype)
        W = make_weights(wl, seed=5)
        _CTX[key] = lib.Fovea(dims_of(wl, W, 1 if dtype == "bf16" else 0), W, device="cuda")
    return _CTX[key]


def _tensor(x, dtype):
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to(torch.bfloat16 if dtype == "bf16" else torch.float32).cuda().contiguous()


def _run(lib, h, W, k, dtype):
    fv = _ctx(lib, dtype, h.shape[1])
    print(f"[gpu] lm_topk n={h.shape[0]} d={h.shape[1]} vocab={W.shape[0]} k={k} {dtype}", flush=True)
    idx, val = fv.lm_topk(_tensor(h, dtype), _tensor(W, dtype), k)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), val.cpu().numpy().astype(np.float64)


def check_topk(idx, val, z, k, tol=Z_TOL):
    """idx/val: GPU [n, k]; z: oracle logits [n, vocab] (fp64).  Returns the fraction of
    ranks whose id had to match exactly."""
    n, vocab = z.shape
    ref_idx, ref_val = oracle.lm_topk_from_logits(z, k)
    decided = 0
    for r in range(n):
        assert len(set(idx[r].tolist())) == k, (r, idx[r])
        assert np.all((idx[r] >= 0) & (idx[r] < vocab)), (r, idx[r])
        zr = z[r, idx[r]]
        np.testing.assert_allclose(val[r], zr, rtol=0, atol=tol * max(1.0, np.abs(zr).max()))
        # rank by rank, the chosen logit is the q-th largest within the tolerance
        np.testing.assert_allclose(zr, ref_val[r], rtol=0, atol=2 * tol)
        # exact ids where the oracle's order is decided by more than the tolerance
        top = np.append(np.sort(z[r])[::-1][: k + 1], -np.inf)  # k = vocab has no (k+1)-th
        for q in range(k):
            lo = top[q] - top[q + 1]
            hi = top[q - 1] - top[q] if q > 0 else np.inf
            if min(lo, hi) > 4 * tol:
                assert idx[r, q] == ref_idx[r, q], (r, q, idx[r], ref_idx[r])
                decided += 1
    return decided / (n * k)


@pytest.mark.parametrize("dtype,n,d,vocab,k", [
    ("f32", 5, 128, 1000, 6),      # one row tile, ragged last column tile (1000 = 7 * 128 + 104)
    ("f32", 130, 256, 777, 16),    # three 64-row tiles ... two 128-row tiles, k at its limit
    ("bf16", 65, 512, 4099, 1),    # arg-max, first row past one 64-row tile
    ("bf16", 7, 64, 100, 16),      # vocabulary inside one partial tile
    ("bf16", 3, 64, 16, 16),       # k = vocab: the full sort
    ("f32", 800, 128, 1000, 6),    # 256-row tiles, the last one ragged (800 = 3 * 256 + 32)
    ("bf16", 777, 256, 2000, 16),  # 256-row tiles, k at its limit
])
def test_lm_topk_small(lib, dtype, n, d, vocab, k):
    h, W = make_lm_case(n, d, vocab, dtype, seed=n * 1000 + vocab)
    idx, val = _run(lib, h, W, k, dtype)
    z = oracle.lm_logits(h, W)
    assert check_topk(idx, val, z, k) > 0.9


@pytest.mark.parametrize("head,n", [("vicuna7b", 60), ("vicuna7b", 1920), ("qwen2_5_7b", 60)])
def test_lm_topk_paper_heads(lib, head, n):
    """Full-size heads: one request's 60-node tree, 32 requests' trees, K_c = 6."""
    cfg = LM_HEADS[head]
    h, W = make_lm_case(n, cfg["d"], cfg["vocab"], "bf16", seed=77 + n)
    idx, val = _run(lib, h, W, 6, "bf16")
    z = oracle.lm_logits(h, W)
    assert check_topk(idx, val, z, 6) > 0.9


def test_lm_topk_exact_ties(lib):
    """Duplicated head rows give bit-identical logits on both sides: ids ascend."""
    h, W = make_lm_case(20, 256, 3000, "bf16", seed=11)
    z0 = oracle.lm_logits(h, W)
    # copy each row's top token into higher ids of other column tiles
    for r in range(4):
        j = int(np.argmax(z0[r]))
        for dst in (j + 129 + r, j + 1000 + r, 2999 - r):
            if dst < 3000 and dst != j:
                W[dst] = W[j]
    idx, val = _run(lib, h, W, 8, "bf16")
    z = oracle.lm_logits(h, W)
    ref_idx, _ = oracle.lm_topk_from_logits(z, 8)
    for r in range(4):
        j = ref_idx[r, 0]
        ties = np.flatnonzero(z[r] == z[r, j])
        assert ties.size >= 2
        assert idx[r, : ties.size].tolist() == sorted(ties.tolist())
        assert np.all(val[r, : ties.size] == val[r, 0])
    check_topk(idx, val, z, 8)


def test_lm_topk_nan_rows(lib):
    h, W = make_lm_case(6, 128, 500, "f32", seed=3)
    h[2] = np.nan
    idx, val = _run(lib, h, W, 4, "f32")
    assert idx[2].tolist() == [-1, -1, -1, -1] and np.all(val[2] == -np.inf)
    keep = [0, 1, 3, 4, 5]
    check_topk(idx[keep], val[keep], oracle.lm_logits(h[keep], W), 4)


def test_lm_topk_without_logits_and_repeat(lib):
    h, W = make_lm_case(70, 256, 2000, "bf16", seed=9)
    fv = _ctx(lib, "bf16", 256)
    ht, Wt = _tensor(h, "bf16"), _tensor(W, "bf16")
    a, _ = fv.lm_topk(ht, Wt, 6, want_logits=False)
    b, lb = fv.lm_topk(ht, Wt, 6)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    check_topk(b.cpu().numpy(), lb.cpu().numpy().astype(np.float64), oracle.lm_logits(h, W), 6)


def test_lm_topk_host_errors(lib):
    fv = _ctx(lib, "bf16", 128)
    h = torch.zeros(4, 128, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(300, 128, dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(4, 16, dtype=torch.int32, device="cuda")
    ws = torch.empty(1 << 20, dtype=torch.uint8, device="cuda")
    f = lib.fovea_lm_topk
    for k, st in ((0, lib.FOVEA_ERR_INVALID_ARG), (17, lib.FOVEA_ERR_UNSUPPORTED)):
        with pytest.raises(lib.FoveaError) as e:
            f(fv.ctx, 4, h, W, 300, k, idx, None, ws)
        assert e.value.status == st
    with pytest.raises(lib.FoveaError) as e:   # vocab < k
        f(fv.ctx, 4, h, W, 5, 6, idx, None, ws)
    assert e.value.status == lib.FOVEA_ERR_INVALID_ARG
    with pytest.raises(lib.FoveaError) as e:   # workspace too small
        f(fv.ctx, 4, h, W, 300, 6, idx, None, ws[:64])
    assert e.value.status == lib.FOVEA_ERR_WORKSPACE
    with pytest.raises(lib.FoveaError) as e:   # misaligned workspace
        f(fv.ctx, 4, h, W, 300, 6, idx, None, ws[1:])
    assert e.value.status == lib.FOVEA_ERR_WORKSPACE
    with pytest.raises(lib.FoveaError) as e:   # output inside the workspace
        f(fv.ctx, 4, h, W, 300, 6, ws[:4 * 16 * 4].view(torch.int32).view(4, 16), None, ws)
    assert e.value.status == lib.FOVEA_ERR_INVALID_ARG
    assert lib.fovea_lm_topk_workspace(fv.ctx, 4, 300, 17) == 0
    f(fv.ctx, 0, h, W, 300, 6, idx, None, ws)   # no rows: nothing to do
