"""Plain fp64 reference of FOVEA's per-draft-step retrieval and fusion.

TEST INFRASTRUCTURE: imported only by tests, the smoke check and the benchmark's
CPU-baseline leg.  It shares no code with the HIP library.

Sources (paper section / equation):
  * Method, "Image-specific visual memory": k_i = W_K LN(v_i), u_i = W_U LN(v_i),
    with a validity mask m_i.
  * Method, "State-conditioned top-K retrieval": q_n = W_Q(LN(h_n) + E_dep[l_n]),
    s_{n,i} = q_n . k_i / sqrt(d_k); global softmax over valid keys; descending rank
    pi_n; cardinality equation K_r (raw cardinality = smallest prefix whose normalised
    mass reaches rho, clamped by K_min, K_max and |V|); renormalised readout over
    the selected set.
  * Method, "Cache-friendly hidden-vector correction" and the appendix paragraph
    "Visual correction module": c_n = f([h_n; r_n]), g_n = sigmoid(g([h_n; r_n])), both
    nets two biased linear layers with a 512-wide SiLU hidden layer; the scalar gate is
    broadcast over the hidden size; h_hat = RMSNorm(h_n + g_n c_n) (Eq. hidden_correction).
  * Algorithm 1 orders the per-node steps the same way.
  * Training the module (Method, training objective; appendix, draft model training):
    ``retrieve_fuse_backward`` takes dL/dh_hat and returns the gradients of the states,
    the memory and every per-step weight, by the chain rule through RMSNorm, the gated
    residual, both nets, the renormalised softmax over the selected set and the query;
    the selected set itself is held fixed (it is a discrete choice);
    ``build_memory_backward`` carries dL/dkeys and dL/dvalues into W_K, W_U, the
    memory LayerNorm and the visual tokens.
  * Eq. hidden_correction's z_n = W_LM h_hat_n and Algorithm 1's tree expansion, which
    adds each node's K_c highest-scoring tokens (K_c = 6 in the experimental setup):
    ``lm_topk``.

Readings where the paper is silent (each one is listed with its reason in the design notes):
  * ties in the descending rank are broken by ascending memory index;
  * if the prefix mass never reaches rho, the raw cardinality is |V| (so rho = 1 means
    dense retrieval);
  * d_k is the key width actually used (d_m);
  * |V| = 0 gives K = 0 and a zero readout; the correction is still applied;
  * LayerNorm is affine with biased variance; RMSNorm has a weight (optional: None
    returns h + g c unnormalised, the reading used for the "gate = 0 returns h" check);
  * the concatenation is [h; r] with h first; W_Q, W_K, W_U have no bias;
  * the K_c candidates of a node are its K_c largest logits, equal logits by ascending
    token id; a NaN logit is never a candidate, and a slot left without one holds -1.

Parity pins (tests/test_oracle.py): brute-force subset enumeration, closed forms for
uniform and geometric score profiles, the dense special case against PyTorch's
scaled-dot-product attention, LayerNorm/RMSNorm/linear against torch.nn.functional,
the peaked case (K = 1, readout equals the value row exactly), gate = 0 and gate = 1
special cases, invariants (mass, clamps, permutation equivariance, masking); for
``lm_topk``, pure-Python brute force (dot products and repeated arg-max scans),
exact ties from duplicated head rows, and the k = vocab case as a full sort; for
``retrieve_fuse_backward``, central finite differences of the forward in fp64, an
autograd re-derivation in torch (fp64, CPU), and the gate-closed and no-RMSNorm cases.  The
correction MLPs at random weights have no independent numeric fixture in the paper:
they are pinned through the gate special cases and the torch cross-check of each
linear layer, not through a printed example.
"""

from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_round",
    "fold_gain",
    "layer_norm",
    "rms_norm",
    "sigmoid",
    "silu",
    "projected_layer_norm",
    "build_memory",
    "query",
    "scores",
    "select_cumulative_mass",
    "readout",
    "correction",
    "fuse",
    "retrieve_fuse",
    "retrieve_fuse_backward",
    "build_memory_backward",
    "lm_logits",
    "lm_topk",
    "lm_topk_from_logits",
]


# --------------------------------------------------------------------------------------
# elementary pieces
# --------------------------------------------------------------------------------------


def bf16_round(x) -> np.ndarray:
    """Round to the nearest bfloat16 value, ties to even.

    Only defined here for inputs that are exactly representable in float32 (e.g. the
    product of two bf16 numbers), so that there is a single rounding step.
    """
    x = np.asarray(x, dtype=np.float64)
    f = x.astype(np.float32)
    if not np.array_equal(f.astype(np.float64), x, equal_nan=True):
        raise ValueError("bf16_round expects float32-representable inputs")
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    u = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def fold_gain(W, gain, rounding: str | None):
    """W diag(gain): a LayerNorm gain folded into the projection that follows it.

    For bf16 storage the library keeps the folded weight in bf16, one rounding per
    element of an exactly computed product; ``rounding="bf16"`` applies that same
    rounding so both sides contract the same weight.  With a unit gain it is exact.
    """
    Wg = np.asarray(W, np.float64) * np.asarray(gain, np.float64)[None, :]
    if rounding is None:
        return Wg
    if rounding == "bf16":
        return bf16_round(Wg)
    raise ValueError(f"unknown rounding {rounding!r}")


def layer_norm(x, gain, bias, eps):
    """LayerNorm over the last axis: biased variance, affine gain and bias."""
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * gain + bias


def rms_norm(x, weight, eps):
    """RMSNorm over the last axis with a weight."""
    x = np.asarray(x, np.float64)
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * weight


def sigmoid(x):
    x = np.asarray(x, np.float64)
    out = np.empty_like(x)
    pos = x >= 0
    out[pos] = 1.0 / (1.0 + np.exp(-x[pos]))
    ex = np.exp(x[~pos])
    out[~pos] = ex / (1.0 + ex)
    return out


def silu(x):
    x = np.asarray(x, np.float64)
    return x * sigmoid(x)


def projected_layer_norm(x, gain, bias, W, eps, gain_rounding=None):
    """W LN(x) for each row of x.

    With ``gain_rounding=None`` this is literally ``LN(x) @ W.T``.  With "bf16" the
    LayerNorm gain is folded into W and rounded once (``fold_gain``); the bias term
    stays exact: W LN(x) = (W diag(g)) xhat + W b, where xhat = (x - mu)/sqrt(var + eps).
    """
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    if gain_rounding is None:
        return layer_norm(x, gain, bias, eps) @ W.T
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    xhat = (x - mu) / np.sqrt(var + eps)
    return xhat @ fold_gain(W, gain, gain_rounding).T + (W @ np.asarray(bias, np.float64))[None, :]


# --------------------------------------------------------------------------------------
# the method
# --------------------------------------------------------------------------------------


def build_memory(V, ln_g, ln_b, W_K, W_U, eps, gain_rounding=None):
    """Per-image visual memory (Method, image-specific visual memory): keys and values
    are the LayerNormed visual tokens projected by W_K and W_U (no bias)."""
    keys = projected_layer_norm(V, ln_g, ln_b, W_K, eps, gain_rounding)
    values = projected_layer_norm(V, ln_g, ln_b, W_U, eps, gain_rounding)
    return keys, values


def query(h, depth, ln_g, ln_b, E_dep, W_Q, eps, gain_rounding=None):
    """State-conditioned query q_n = W_Q (LN(h_n) + E_dep[l_n]) (Method, retrieval)."""
    depth = np.asarray(depth, np.int64)
    E = np.asarray(E_dep, np.float64)[depth]
    W_Q = np.asarray(W_Q, np.float64)
    return projected_layer_norm(h, ln_g, ln_b, W_Q, eps, gain_rounding) + E @ W_Q.T


def scores(q, keys):
    """s_{n,i} = q_n . k_i / sqrt(d_k), with d_k the key width (Method, retrieval)."""
    keys = np.asarray(keys, np.float64)
    return np.asarray(q, np.float64) @ keys.T / np.sqrt(keys.shape[1])


def select_cumulative_mass(s, valid, tau, k_min, k_max):
    """Cumulative-mass cardinality rule for one node (Method, cardinality equation K_r).

    s: scores over the request's memory (local indices); valid: boolean mask.
    Returns a dict with K, the selected local indices in rank order, the selected mass
    C_K, K_raw, and the full descending order and prefix masses for diagnostics.
    """
    s = np.asarray(s, np.float64)
    valid = np.ones(s.shape, bool) if valid is None else np.asarray(valid, bool)
    V = np.flatnonzero(valid)  # ascending local index
    nV = V.size
    if nV == 0:
        return dict(K=0, K_raw=0, idx=np.zeros(0, np.int64), mass=0.0, n_valid=0,
                    order=np.zeros(0, np.int64), prefix=np.zeros(0), alpha_tilde=np.zeros(0))
    sv = s[V]
    # global softmax over the valid keys
    e = np.exp(sv - sv.max())
    alpha_tilde = e / e.sum()
    # descending rank; a stable sort of -s keeps ascending index among equal scores
    rank = np.argsort(-sv, kind="stable")
    order = V[rank]
    prefix = np.cumsum(alpha_tilde[rank])
    reached = np.flatnonzero(prefix >= tau)
    K_raw = int(reached[0]) + 1 if reached.size else nV
    K = min(nV, int(k_max), max(int(k_min), K_raw))
    return dict(K=K, K_raw=K_raw, idx=order[:K].copy(), mass=float(prefix[K - 1]) if K else 0.0,
                n_valid=nV, order=order, prefix=prefix, alpha_tilde=alpha_tilde)


def readout(s, idx, values):
    """Renormalised readout over the selected set (Method, readout equation):
    alpha_i = exp(s_i) / sum_{j in I} exp(s_j); r = sum_i alpha_i u_i."""
    values = np.asarray(values, np.float64)
    idx = np.asarray(idx, np.int64)
    if idx.size == 0:
        return np.zeros(values.shape[1]), np.zeros(0)
    sI = np.asarray(s, np.float64)[idx]
    e = np.exp(sI - sI.max())
    alpha = e / e.sum()
    return alpha @ values[idx], alpha


def correction(h, r, W_c1, b_c1, W_c2, b_c2, W_g1, b_g1, w_g2, b_g2):
    """c = f([h; r]) and g = sigmoid(g_net([h; r])) (Method, correction; appendix,
    visual correction module): each net is Linear -> SiLU -> Linear, biased."""
    y = np.concatenate([np.atleast_2d(h), np.atleast_2d(r)], axis=-1)
    a_c = silu(y @ np.asarray(W_c1, np.float64).T + b_c1)
    c = a_c @ np.asarray(W_c2, np.float64).T + b_c2
    a_g = silu(y @ np.asarray(W_g1, np.float64).T + b_g1)
    g = sigmoid(a_g @ np.asarray(w_g2, np.float64) + b_g2)
    return c, g


def fuse(h, g, c, rms_w, eps):
    """h_hat = RMSNorm(h + g c) (Eq. hidden_correction); rms_w=None returns h + g c."""
    hp = np.atleast_2d(h) + np.asarray(g, np.float64)[:, None] * c
    return hp if rms_w is None else rms_norm(hp, rms_w, eps)


def retrieve_fuse(W, mem_off, keys, values, valid, node_off, h, depth, tau, k_min, k_max,
                  gain_rounding=None):
    """One draft step over a ragged batch of requests (Algorithm 1's inner loop).

    W: dict of weights (q_ln_g, q_ln_b, E_dep, W_Q, W_c1, b_c1, W_c2, b_c2, W_g1, b_g1,
    w_g2, b_g2, rms_w or None, ln_eps, rms_eps).  Request b owns memory rows
    mem_off[b]:mem_off[b+1] and nodes node_off[b]:node_off[b+1].
    Returns h_out, K, idx (local indices in rank order, -1 padded to k_max), gate,
    mass (C_K), r, q, and per-node selection records.
    """
    h = np.asarray(h, np.float64)
    n, d = h.shape
    keys = np.asarray(keys, np.float64)
    values = np.asarray(values, np.float64)
    d_m = keys.shape[1]
    B = len(node_off) - 1
    q = query(h, depth, W["q_ln_g"], W["q_ln_b"], W["E_dep"], W["W_Q"], W["ln_eps"], gain_rounding)
    K = np.zeros(n, np.int64)
    idx = np.full((n, k_max), -1, np.int64)
    mass = np.zeros(n)
    r = np.zeros((n, d_m))
    records = [None] * n
    for b in range(B):
        m0, m1 = int(mem_off[b]), int(mem_off[b + 1])
        kb, ub = keys[m0:m1], values[m0:m1]
        vb = None if valid is None else np.asarray(valid[m0:m1], bool)
        t0, t1 = int(node_off[b]), int(node_off[b + 1])
        if t1 == t0:
            continue
        sb = scores(q[t0:t1], kb) if m1 > m0 else np.zeros((t1 - t0, 0))
        for j in range(t1 - t0):
            sel = select_cumulative_mass(sb[j], vb, float(tau[b]), k_min, k_max)
            nid = t0 + j
            K[nid] = sel["K"]
            idx[nid, : sel["K"]] = sel["idx"]
            mass[nid] = sel["mass"]
            r[nid], _ = readout(sb[j], sel["idx"], ub)
            sel["s"] = sb[j]
            records[nid] = sel
    c, g = correction(h, r, W["W_c1"], W["b_c1"], W["W_c2"], W["b_c2"], W["W_g1"], W["b_g1"],
                      W["w_g2"], W["b_g2"])
    h_out = fuse(h, g, c, W.get("rms_w"), W["rms_eps"])
    return dict(h_out=h_out, K=K, idx=idx, gate=g, mass=mass, r=r, q=q, records=records)


def lm_logits(h, W_LM):
    """z_n = W_LM h_n for every row (Eq. hidden_correction), in fp64."""
    return np.asarray(h, np.float64) @ np.asarray(W_LM, np.float64).T


def lm_topk(h, W_LM, k):
    """The k draft candidates of every row (Algorithm 1, tree expansion): token ids of
    the k largest logits, descending, equal logits by ascending id; NaN logits are
    skipped and an unfilled slot holds id -1 and logit -inf.  Returns (idx, logits)."""
    return lm_topk_from_logits(lm_logits(h, W_LM), k)


def lm_topk_from_logits(z, k):
    """The candidate rule of ``lm_topk`` applied to given logits [n, vocab]."""
    z = np.asarray(z, np.float64)
    n, vocab = z.shape
    idx = np.full((n, k), -1, np.int64)
    val = np.full((n, k), -np.inf)
    ids = np.arange(vocab)
    for r in range(n):
        ok = ~np.isnan(z[r])
        # lexsort: last key is primary -> by -z, then by id
        order = ids[ok][np.lexsort((ids[ok], -z[r][ok]))][:k]
        idx[r, : order.size] = order
        val[r, : order.size] = z[r][order]
    return idx, val


def retrieve_fuse_backward(W, mem_off, keys, values, node_off, h, depth, idx, K, dh_hat):
    """Gradients of one draft step's output h_hat with respect to its inputs and weights,
    given dL/dh_hat (Method, training objective: the module is trained end to end; the
    selected sets I_n = idx[n, :K[n]] are held fixed, a discrete choice with no
    gradient).  fp64 throughout, no weight rounding.

    Forward (per node n, request b, y = [h; r]):
      x   = LN_q(h),  q = W_Q (x + E_dep[l]),  s_i = q . k_i / sqrt(d_m)  (i in I_n)
      a_i = softmax over I_n of s,  r = sum_i a_i u_i
      z_c = W_c1 y + b_c1,  c = W_c2 SiLU(z_c) + b_c2
      z_g = W_g1 y + b_g1,  g = sigmoid(w_g2 . SiLU(z_g) + b_g2)
      h'  = h + g c,  h_hat = h' rho w  (rho = 1/sqrt(mean(h'^2) + eps); rms_w None: h' )
    Returns a dict with dh [n, d], dkeys and dvalues [n_mem, d_m], and dW_Q, dq_ln_g,
    dq_ln_b, dE_dep, dW_c1, db_c1, dW_c2, db_c2, dW_g1, db_g1, dw_g2, db_g2, drms_w
    (None without RMSNorm), each shaped like its weight."""
    f = np.float64
    h = np.asarray(h, f)
    n, d = h.shape
    keys = np.asarray(keys, f)
    values = np.asarray(values, f)
    d_m = keys.shape[1]
    dh_hat = np.asarray(dh_hat, f)
    depth = np.asarray(depth, np.int64)
    W_Q, E_dep = np.asarray(W["W_Q"], f), np.asarray(W["E_dep"], f)
    g_q, b_q = np.asarray(W["q_ln_g"], f), np.asarray(W["q_ln_b"], f)
    W_c1, b_c1 = np.asarray(W["W_c1"], f), np.asarray(W["b_c1"], f)
    W_c2, b_c2 = np.asarray(W["W_c2"], f), np.asarray(W["b_c2"], f)
    W_g1, b_g1 = np.asarray(W["W_g1"], f), np.asarray(W["b_g1"], f)
    w_g2, b_g2 = np.asarray(W["w_g2"], f), float(W["b_g2"])
    rms_w = W.get("rms_w")
    eps_ln, eps_rms = W["ln_eps"], W["rms_eps"]
    scale = 1.0 / np.sqrt(d_m)
    # request of every node, global memory rows of every selected entry
    req = np.zeros(n, np.int64)
    for b in range(len(node_off) - 1):
        req[int(node_off[b]):int(node_off[b + 1])] = b

    # ---- forward, keeping what the chain rule needs
    mu = h.mean(axis=1, keepdims=True)
    rstd = 1.0 / np.sqrt(((h - mu) ** 2).mean(axis=1, keepdims=True) + eps_ln)
    xhat = (h - mu) * rstd
    xe = xhat * g_q + b_q + E_dep[depth]
    q = xe @ W_Q.T
    r = np.zeros((n, d_m))
    sel, alpha = [], []
    for i in range(n):
        rows = int(mem_off[req[i]]) + np.asarray(idx[i][: int(K[i])], np.int64)
        sel.append(rows)
        if rows.size == 0:
            alpha.append(np.zeros(0))
            continue
        s_i = keys[rows] @ q[i] * scale
        e = np.exp(s_i - s_i.max())
        a = e / e.sum()
        alpha.append(a)
        r[i] = a @ values[rows]
    y = np.concatenate([h, r], axis=1)
    z_c = y @ W_c1.T + b_c1
    a_c = silu(z_c)
    c = a_c @ W_c2.T + b_c2
    z_g = y @ W_g1.T + b_g1
    a_g = silu(z_g)
    g = sigmoid(a_g @ w_g2 + b_g2)
    hp = h + g[:, None] * c

    def dsilu(z):  # d/dz z sigmoid(z)
        sg = sigmoid(z)
        return sg * (1.0 + z * (1.0 - sg))

    # ---- RMSNorm: h_hat = h' rho w
    if rms_w is None:
        dhp = dh_hat
        drms = None
    else:
        w = np.asarray(rms_w, f)
        rho = 1.0 / np.sqrt((hp * hp).mean(axis=1, keepdims=True) + eps_rms)
        drms = (dh_hat * hp * rho).sum(axis=0)
        gw = dh_hat * w
        dhp = rho * gw - rho ** 3 * hp * (gw * hp).sum(axis=1, keepdims=True) / d
    # ---- gated residual h' = h + g c
    dh = dhp.copy()
    dc = g[:, None] * dhp
    dg = (dhp * c).sum(axis=1)
    dlogit = dg * g * (1.0 - g)
    # ---- layer 2 and the gate's second layer
    dW_c2 = dc.T @ a_c
    db_c2 = dc.sum(axis=0)
    dz_c = (dc @ W_c2) * dsilu(z_c)
    dw_g2 = a_g.T @ dlogit
    db_g2 = dlogit.sum()
    dz_g = dlogit[:, None] * w_g2[None, :] * dsilu(z_g)
    # ---- first layers over y = [h; r]
    dW_c1 = dz_c.T @ y
    db_c1 = dz_c.sum(axis=0)
    dW_g1 = dz_g.T @ y
    db_g1 = dz_g.sum(axis=0)
    dy = dz_c @ W_c1 + dz_g @ W_g1
    dh += dy[:, :d]
    dr = dy[:, d:]
    # ---- readout r = sum a_i u_i, a = softmax over the selected set of s
    dkeys = np.zeros_like(keys)
    dvalues = np.zeros_like(values)
    dq = np.zeros((n, d_m))
    for i in range(n):
        rows, a = sel[i], alpha[i]
        if rows.size == 0:
            continue
        da = values[rows] @ dr[i]
        ds = a * (da - a @ da)
        np.add.at(dvalues, rows, a[:, None] * dr[i][None, :])
        dq[i] = ds @ keys[rows] * scale
        np.add.at(dkeys, rows, ds[:, None] * q[i][None, :] * scale)
    # ---- query q = W_Q (LN(h) g + b + E_dep[l])
    dW_Q = dq.T @ xe
    dxe = dq @ W_Q
    dE_dep = np.zeros_like(E_dep)
    np.add.at(dE_dep, depth, dxe)
    dq_ln_g = (dxe * xhat).sum(axis=0)
    dq_ln_b = dxe.sum(axis=0)
    dxh = dxe * g_q
    dh += rstd * (dxh - dxh.mean(axis=1, keepdims=True)
                  - xhat * (dxh * xhat).mean(axis=1, keepdims=True))
    return dict(dh=dh, dkeys=dkeys, dvalues=dvalues, dW_Q=dW_Q, dq_ln_g=dq_ln_g,
                dq_ln_b=dq_ln_b, dE_dep=dE_dep, dW_c1=dW_c1, db_c1=db_c1, dW_c2=dW_c2,
                db_c2=db_c2, dW_g1=dW_g1, db_g1=db_g1, dw_g2=dw_g2, db_g2=db_g2,
                drms_w=drms)


def build_memory_backward(V, ln_g, ln_b, W_K, W_U, eps, dkeys, dvalues):
    """Gradients of the memory build k_i = W_K LN(v_i), u_i = W_U LN(v_i) (Method,
    image-specific visual memory) given dL/dkeys and dL/dvalues: returns dW_K, dW_U,
    dmem_ln_g, dmem_ln_b and dV.  fp64, no weight rounding."""
    f = np.float64
    V = np.asarray(V, f)
    g, b = np.asarray(ln_g, f), np.asarray(ln_b, f)
    W_K, W_U = np.asarray(W_K, f), np.asarray(W_U, f)
    dk, du = np.asarray(dkeys, f), np.asarray(dvalues, f)
    mu = V.mean(axis=1, keepdims=True)
    rstd = 1.0 / np.sqrt(((V - mu) ** 2).mean(axis=1, keepdims=True) + eps)
    xhat = (V - mu) * rstd
    xn = xhat * g + b
    dW_K = dk.T @ xn
    dW_U = du.T @ xn
    dxn = dk @ W_K + du @ W_U
    dg = (dxn * xhat).sum(axis=0)
    db = dxn.sum(axis=0)
    dxh = dxn * g
    dV = rstd * (dxh - dxh.mean(axis=1, keepdims=True)
                 - xhat * (dxh * xhat).mean(axis=1, keepdims=True))
    return dict(dW_K=dW_K, dW_U=dW_U, dmem_ln_g=dg, dmem_ln_b=db, dV=dV)
