"""Pins of the oracle's backward (retrieve_fuse_backward) on the CPU: central finite
differences of the forward in fp64, an independent autograd derivation in torch (fp64),
and the special cases where whole branches have zero gradient."""

import numpy as np
import pytest
import torch

import oracle

PARAMS = ["W_Q", "q_ln_g", "q_ln_b", "E_dep", "W_c1", "b_c1", "W_c2", "b_c2", "W_g1", "b_g1",
          "w_g2", "rms_w"]


def _case(seed=0, d=16, d_m=8, d_c=12, n_depth=4, B=2, T=(3, 2), M=(7, 5), tau=0.7, k_max=4,
          rms=True):
    rng = np.random.default_rng(seed)
    W = dict(
        W_Q=rng.standard_normal((d_m, d)) / np.sqrt(d), q_ln_g=1 + 0.2 * rng.standard_normal(d),
        q_ln_b=0.2 * rng.standard_normal(d), E_dep=0.5 * rng.standard_normal((n_depth, d)),
        W_c1=rng.standard_normal((d_c, d + d_m)) / np.sqrt(d + d_m),
        b_c1=0.1 * rng.standard_normal(d_c),
        W_c2=rng.standard_normal((d, d_c)) / np.sqrt(d_c), b_c2=0.1 * rng.standard_normal(d),
        W_g1=rng.standard_normal((d_c, d + d_m)) / np.sqrt(d + d_m),
        b_g1=0.1 * rng.standard_normal(d_c), w_g2=rng.standard_normal(d_c) / np.sqrt(d_c),
        b_g2=0.3, rms_w=(1 + 0.2 * rng.standard_normal(d)) if rms else None,
        ln_eps=1e-5, rms_eps=1e-6)
    mem_off = np.concatenate([[0], np.cumsum(M)]).astype(np.int64)
    node_off = np.concatenate([[0], np.cumsum(T)]).astype(np.int64)
    n, n_mem = int(node_off[-1]), int(mem_off[-1])
    keys = 2.0 * rng.standard_normal((n_mem, d_m))
    values = rng.standard_normal((n_mem, d_m))
    h = rng.standard_normal((n, d))
    depth = rng.integers(0, n_depth, n)
    tau_b = np.full(B, tau)
    fwd = oracle.retrieve_fuse(W, mem_off, keys, values, None, node_off, h, depth, tau_b, 1, k_max)
    dh_hat = rng.standard_normal((n, d))
    return dict(W=W, mem_off=mem_off, node_off=node_off, keys=keys, values=values, h=h,
                depth=depth, idx=fwd["idx"], K=fwd["K"], dh_hat=dh_hat)


def _loss(c, W=None, h=None, keys=None, values=None):
    """sum(dh_hat * h_hat) with the selection held fixed, from the oracle's forward pieces."""
    W = c["W"] if W is None else W
    h = c["h"] if h is None else h
    keys = c["keys"] if keys is None else keys
    values = c["values"] if values is None else values
    q = oracle.query(h, c["depth"], W["q_ln_g"], W["q_ln_b"], W["E_dep"], W["W_Q"], W["ln_eps"])
    n = h.shape[0]
    r = np.zeros((n, keys.shape[1]))
    for b in range(len(c["node_off"]) - 1):
        m0, m1 = c["mem_off"][b], c["mem_off"][b + 1]
        for i in range(c["node_off"][b], c["node_off"][b + 1]):
            s = oracle.scores(q[i:i + 1], keys[m0:m1])[0]
            r[i], _ = oracle.readout(s, c["idx"][i, : c["K"][i]], values[m0:m1])
    cc, g = oracle.correction(h, r, W["W_c1"], W["b_c1"], W["W_c2"], W["b_c2"], W["W_g1"],
                              W["b_g1"], W["w_g2"], W["b_g2"])
    return float((c["dh_hat"] * oracle.fuse(h, g, cc, W.get("rms_w"), W["rms_eps"])).sum())


def _grads(c):
    return oracle.retrieve_fuse_backward(c["W"], c["mem_off"], c["keys"], c["values"],
                                         c["node_off"], c["h"], c["depth"], c["idx"], c["K"],
                                         c["dh_hat"])


def _fd(f, x, entries, eps=1e-6):
    out = []
    for e in entries:
        x0 = x[e]
        x[e] = x0 + eps
        lp = f()
        x[e] = x0 - eps
        lm = f()
        x[e] = x0
        out.append((lp - lm) / (2 * eps))
    return np.array(out)


def _entries(shape, rng, k=6):
    flat = rng.choice(int(np.prod(shape)), size=min(k, int(np.prod(shape))), replace=False)
    return [np.unravel_index(i, shape) for i in flat]


@pytest.mark.parametrize("seed,rms", [(0, True), (1, True), (2, False)])
def test_backward_matches_finite_differences(seed, rms):
    c = _case(seed, rms=rms)
    assert c["K"].min() >= 1 and c["K"].max() >= 2  # softmax over several entries somewhere
    G = _grads(c)
    rng = np.random.default_rng(100 + seed)
    checks = [("dh", c["h"], lambda: _loss(c))]
    checks += [("dkeys", c["keys"], lambda: _loss(c)), ("dvalues", c["values"], lambda: _loss(c))]
    for name, x, f in checks:
        ent = _entries(x.shape, rng, 10)
        if name != "dh":  # include selected rows, where the gradient is non-zero
            rows = c["mem_off"][0] + c["idx"][0, : c["K"][0]]
            ent += [(int(rows[0]), j) for j in range(3)]
        np.testing.assert_allclose(G[name][tuple(np.array(ent).T)], _fd(f, x, ent), rtol=1e-6,
                                   atol=1e-8, err_msg=name)
    for p in PARAMS:
        if p == "rms_w" and not rms:
            assert G["drms_w"] is None
            continue
        x = c["W"][p]
        ent = _entries(x.shape, rng, 8)
        np.testing.assert_allclose(G["d" + p][tuple(np.array(ent).T)], _fd(lambda: _loss(c), x, ent),
                                   rtol=1e-6, atol=1e-8, err_msg=p)
    # the scalar gate bias
    W2 = dict(c["W"])
    e = 1e-6
    W2["b_g2"] = c["W"]["b_g2"] + e
    lp = _loss(c, W=W2)
    W2["b_g2"] = c["W"]["b_g2"] - e
    lm = _loss(c, W=W2)
    np.testing.assert_allclose(G["db_g2"], (lp - lm) / (2 * e), rtol=1e-6, atol=1e-9)


def _torch_grads(c):
    """The same forward written with torch ops and differentiated by autograd."""
    t = lambda x: torch.tensor(np.asarray(x, np.float64), requires_grad=True)  # noqa: E731
    W = {p: t(c["W"][p]) for p in PARAMS if c["W"].get(p) is not None}
    b_g2 = t(c["W"]["b_g2"])
    h, keys, values = t(c["h"]), t(c["keys"]), t(c["values"])
    depth = torch.tensor(c["depth"])
    x = torch.nn.functional.layer_norm(h, (h.shape[1],), W["q_ln_g"], W["q_ln_b"], c["W"]["ln_eps"])
    q = (x + W["E_dep"][depth]) @ W["W_Q"].T
    rs = []
    for b in range(len(c["node_off"]) - 1):
        m0 = int(c["mem_off"][b])
        for i in range(int(c["node_off"][b]), int(c["node_off"][b + 1])):
            rows = torch.tensor(m0 + c["idx"][i, : c["K"][i]])
            a = torch.softmax(keys[rows] @ q[i] / keys.shape[1] ** 0.5, 0)
            rs.append(a @ values[rows])
    y = torch.cat([h, torch.stack(rs)], 1)
    cc = torch.nn.functional.silu(y @ W["W_c1"].T + W["b_c1"]) @ W["W_c2"].T + W["b_c2"]
    g = torch.sigmoid(torch.nn.functional.silu(y @ W["W_g1"].T + W["b_g1"]) @ W["w_g2"] + b_g2)
    hp = h + g[:, None] * cc
    out = hp
    if "rms_w" in W:
        out = hp * torch.rsqrt((hp * hp).mean(1, keepdim=True) + c["W"]["rms_eps"]) * W["rms_w"]
    (out * torch.tensor(c["dh_hat"])).sum().backward()
    res = {"d" + p: W[p].grad.numpy() for p in W}
    res.update(dh=h.grad.numpy(), dkeys=keys.grad.numpy(), dvalues=values.grad.numpy(),
               db_g2=b_g2.grad.numpy())
    return res


@pytest.mark.parametrize("seed,rms", [(3, True), (4, False)])
def test_backward_matches_torch_autograd(seed, rms):
    c = _case(seed, d=32, d_m=16, d_c=24, B=3, T=(4, 1, 3), M=(9, 6, 11), rms=rms)
    G, R = _grads(c), _torch_grads(c)
    for k, v in R.items():
        np.testing.assert_allclose(G[k], v, rtol=1e-10, atol=1e-12, err_msg=k)


def test_backward_closed_gate():
    """g = 0 (b_g2 = -inf): h_hat = RMSNorm(h), so nothing before the residual gets a
    gradient and dh is RMSNorm's own backward."""
    c = _case(5)
    c["W"]["b_g2"] = -np.inf
    G = _grads(c)
    for k in ("dkeys", "dvalues", "dW_Q", "dE_dep", "dW_c1", "db_c1", "dW_c2", "db_c2", "dW_g1",
              "db_g1", "dw_g2", "dq_ln_g", "dq_ln_b"):
        assert np.all(G[k] == 0), k
    h = torch.tensor(c["h"], requires_grad=True)
    w = torch.tensor(c["W"]["rms_w"])
    (h * torch.rsqrt((h * h).mean(1, keepdim=True) + 1e-6) * w * torch.tensor(c["dh_hat"])).sum().backward()
    np.testing.assert_allclose(G["dh"], h.grad.numpy(), rtol=1e-12, atol=1e-12)


def _mem_case(seed=0, n=7, d_v=16, d_m=8):
    rng = np.random.default_rng(seed)
    return dict(V=2.0 * rng.standard_normal((n, d_v)) + 0.5,
                g=1 + 0.2 * rng.standard_normal(d_v), b=0.2 * rng.standard_normal(d_v),
                W_K=rng.standard_normal((d_m, d_v)) / np.sqrt(d_v),
                W_U=rng.standard_normal((d_m, d_v)) / np.sqrt(d_v),
                dk=rng.standard_normal((n, d_m)), du=rng.standard_normal((n, d_m)), eps=1e-5)


def _mem_loss(c):
    k, u = oracle.build_memory(c["V"], c["g"], c["b"], c["W_K"], c["W_U"], c["eps"])
    return float((c["dk"] * k).sum() + (c["du"] * u).sum())


def _mem_grads(c):
    return oracle.build_memory_backward(c["V"], c["g"], c["b"], c["W_K"], c["W_U"], c["eps"],
                                        c["dk"], c["du"])


@pytest.mark.parametrize("seed", [0, 1])
def test_memory_backward_matches_finite_differences(seed):
    c = _mem_case(seed)
    G = _mem_grads(c)
    rng = np.random.default_rng(200 + seed)
    for name, key in (("dV", "V"), ("dW_K", "W_K"), ("dW_U", "W_U"), ("dmem_ln_g", "g"),
                      ("dmem_ln_b", "b")):
        x = c[key]
        ent = _entries(x.shape, rng, 8)
        np.testing.assert_allclose(G[name][tuple(np.array(ent).T)], _fd(lambda: _mem_loss(c), x, ent),
                                   rtol=1e-6, atol=1e-8, err_msg=name)


def test_memory_backward_matches_torch_autograd():
    c = _mem_case(3, n=11, d_v=32, d_m=12)
    t = {k: torch.tensor(c[k], requires_grad=True) for k in ("V", "g", "b", "W_K", "W_U")}
    x = torch.nn.functional.layer_norm(t["V"], (32,), t["g"], t["b"], c["eps"])
    ((x @ t["W_K"].T) * torch.tensor(c["dk"]) + (x @ t["W_U"].T) * torch.tensor(c["du"])).sum().backward()
    G = _mem_grads(c)
    for name, key in (("dV", "V"), ("dW_K", "W_K"), ("dW_U", "W_U"), ("dmem_ln_g", "g"),
                      ("dmem_ln_b", "b")):
        np.testing.assert_allclose(G[name], t[key].grad.numpy(), rtol=1e-10, atol=1e-12, err_msg=name)
