"""ctypes binding of libfovea.so (the C ABI in include/fovea.h).

Argument marshalling only: torch tensors supply device pointers and torch's current
stream supplies the HIP stream; every step of the computation runs in the library's
HIP kernels.  Importing this module fails loudly if the library has not been built.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libfovea.so")

FOVEA_OK = 0
FOVEA_ERR_INVALID_ARG = 1
FOVEA_ERR_UNSUPPORTED = 2
FOVEA_ERR_WORKSPACE = 3
FOVEA_ERR_DEVICE = 4
FOVEA_ERR_DATA = 5
FOVEA_F32 = 0
FOVEA_BF16 = 1

FOVEA_DATA_BAD_NODE_OFFSETS = 0x1
FOVEA_DATA_BAD_MEM_OFFSETS = 0x2
FOVEA_DATA_BAD_DEPTH = 0x4
FOVEA_DATA_BAD_TAU = 0x8
FOVEA_DATA_BAD_SELECTION = 0x10

FOVEA_MAX_M = 16384
FOVEA_MAX_KMAX = 1024
FOVEA_LM_MAX_K = 16
FOVEA_LM_MAX_VOCAB = 1 << 24
FOVEA_LM_MAX_ROWS = 1 << 20

EXPORTED = [
    "fovea_abi_version", "fovea_status_str", "fovea_create", "fovea_destroy",
    "fovea_build_memory_workspace", "fovea_build_memory", "fovea_retrieve_fuse_workspace",
    "fovea_retrieve_fuse", "fovea_retrieve_fuse_noalloc",
    "fovea_last_error", "fovea_profile", "fovea_profile_read", "fovea_lm_topk_workspace",
    "fovea_lm_topk", "fovea_retrieve_fuse_backward_workspace", "fovea_retrieve_fuse_backward",
    "fovea_build_memory_backward_workspace", "fovea_build_memory_backward",
]


class FoveaError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {fovea_status_str(status)} (status {status})")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("d", ctypes.c_int32), ("d_v", ctypes.c_int32), ("d_m", ctypes.c_int32),
                ("d_c", ctypes.c_int32), ("n_depth", ctypes.c_int32), ("dtype", ctypes.c_int),
                ("ln_eps", ctypes.c_float), ("rms_eps", ctypes.c_float)]


PARAM_TENSORS = ["mem_ln_g", "mem_ln_b", "W_K", "W_U", "q_ln_g", "q_ln_b", "E_dep", "W_Q",
                 "W_c1", "b_c1", "W_c2", "b_c2", "W_g1", "b_g1", "w_g2"]


class Params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in PARAM_TENSORS] + [
        ("b_g2", ctypes.c_float), ("rms_w", ctypes.c_void_p)]


GRAD_TENSORS = ["W_Q", "q_ln_g", "q_ln_b", "E_dep", "W_c1", "b_c1", "W_c2", "b_c2", "W_g1",
                "b_g1", "w_g2", "b_g2", "rms_w"]


class Grads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in GRAD_TENSORS]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.fovea_abi_version.restype = ctypes.c_int
    lib.fovea_abi_version.argtypes = []
    lib.fovea_status_str.restype = ctypes.c_char_p
    lib.fovea_status_str.argtypes = [ctypes.c_int]
    lib.fovea_create.restype = ctypes.c_int
    lib.fovea_create.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(Dims), ctypes.POINTER(Params), vp]
    lib.fovea_destroy.restype = None
    lib.fovea_destroy.argtypes = [vp]
    lib.fovea_build_memory_workspace.restype = sz
    lib.fovea_build_memory_workspace.argtypes = [vp, i64]
    lib.fovea_build_memory.restype = ctypes.c_int
    lib.fovea_build_memory.argtypes = [vp, i64, vp, vp, vp, vp, sz, vp]
    lib.fovea_retrieve_fuse_workspace.restype = sz
    lib.fovea_retrieve_fuse_workspace.argtypes = [vp, i32, i32, i64, i32, i32]
    lib.fovea_retrieve_fuse.restype = ctypes.c_int
    lib.fovea_retrieve_fuse.argtypes = [
        vp, i32, vp, i64, i32, vp, vp, vp, vp, i32, i32, vp, vp, vp, i32, i32,
        vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.fovea_retrieve_fuse_noalloc.restype = ctypes.c_int
    lib.fovea_retrieve_fuse_noalloc.argtypes = [
        vp, i32, vp, i64, i32, vp, vp, vp, vp, i32, i32, vp, vp, vp, i32, i32,
        vp, vp, vp, vp, vp, vp, vp]
    lib.fovea_last_error.restype = ctypes.c_int
    lib.fovea_last_error.argtypes = [vp, vp, ctypes.POINTER(ctypes.c_uint32)]
    lib.fovea_profile.restype = ctypes.c_int
    lib.fovea_profile.argtypes = [vp, i32]
    lib.fovea_profile_read.restype = i32
    lib.fovea_profile_read.argtypes = [vp, i32, ctypes.POINTER(ctypes.c_char_p),
                                       ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32)]
    lib.fovea_retrieve_fuse_backward_workspace.restype = sz
    lib.fovea_retrieve_fuse_backward_workspace.argtypes = [vp, i32, i32, i32, i32]
    lib.fovea_retrieve_fuse_backward.restype = ctypes.c_int
    lib.fovea_retrieve_fuse_backward.argtypes = [
        vp, ctypes.POINTER(Params), i32, vp, i64, i32, vp, vp, vp, i32, i32, vp, vp, vp, vp, i32,
        vp, vp, vp, vp, ctypes.POINTER(Grads), vp, sz, vp]
    lib.fovea_build_memory_backward_workspace.restype = sz
    lib.fovea_build_memory_backward_workspace.argtypes = [vp, i64]
    lib.fovea_build_memory_backward.restype = ctypes.c_int
    lib.fovea_build_memory_backward.argtypes = [vp, ctypes.POINTER(Params), i64, vp, vp, vp, vp, vp,
                                                vp, vp, vp, vp, sz, vp]
    lib.fovea_lm_topk_workspace.restype = sz
    lib.fovea_lm_topk_workspace.argtypes = [vp, i32, i32, i32]
    lib.fovea_lm_topk.restype = ctypes.c_int
    lib.fovea_lm_topk.argtypes = [vp, i32, vp, vp, i32, i32, vp, vp, vp, sz, vp]
    return lib


lib = _load()


def fovea_abi_version() -> int:
    return lib.fovea_abi_version()


def fovea_status_str(status: int) -> str:
    return lib.fovea_status_str(status).decode()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _ptr(t: torch.Tensor | None, dtype=None, name: str = "") -> int | None:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _check(status: int, where: str):
    if status != FOVEA_OK:
        raise FoveaError(status, where)


def storage_dtype(dtype: int) -> torch.dtype:
    return torch.bfloat16 if dtype == FOVEA_BF16 else torch.float32


def fovea_create(dims: Dims, params: dict, b_g2: float, stream=None) -> int:
    """params: the PARAM_TENSORS (and optional "rms_w") as device tensors in the storage
    dtype.  Returns the opaque context handle."""
    dt = storage_dtype(dims.dtype)
    P = Params()
    for n in PARAM_TENSORS:
        setattr(P, n, _ptr(params[n], dt, n))
    P.b_g2 = float(b_g2)
    P.rms_w = _ptr(params.get("rms_w"), dt, "rms_w")
    ctx = ctypes.c_void_p()
    _check(lib.fovea_create(ctypes.byref(ctx), ctypes.byref(dims), ctypes.byref(P), _stream(stream)),
           "fovea_create")
    return ctx.value


def fovea_destroy(ctx: int) -> None:
    lib.fovea_destroy(ctx)


def fovea_build_memory_workspace(ctx: int, n_rows: int) -> int:
    return lib.fovea_build_memory_workspace(ctx, n_rows)


def fovea_build_memory(ctx: int, V: torch.Tensor, keys: torch.Tensor, values: torch.Tensor,
                       workspace=None, stream=None) -> None:
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.fovea_build_memory(ctx, V.shape[0], _ptr(V, None, "V"), _ptr(keys, V.dtype, "keys"),
                                  _ptr(values, V.dtype, "values"), _ptr(workspace, None, "workspace"),
                                  ws_bytes, _stream(stream)),
           "fovea_build_memory")


def fovea_retrieve_fuse_workspace(ctx: int, B: int, n_nodes_total: int, n_mem_total: int,
                                  m_max: int, k_max: int) -> int:
    return lib.fovea_retrieve_fuse_workspace(ctx, B, n_nodes_total, n_mem_total, m_max, k_max)


def fovea_retrieve_fuse(ctx: int, B: int, mem_off, n_mem_total: int, m_max: int, keys, values,
                        valid, node_off, n_nodes_total: int, t_max: int, h, depth, tau,
                        k_min: int, k_max: int, h_out, k_out=None, idx_out=None, gate_out=None,
                        mass_out=None, r_out=None, workspace=None, stream=None) -> None:
    """Same arguments as the C entry point; tensors stand for device pointers."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.fovea_retrieve_fuse(
        ctx, B, _ptr(mem_off, torch.int64, "mem_off"), n_mem_total, m_max,
        _ptr(keys, h.dtype, "keys"), _ptr(values, h.dtype, "values"),
        _ptr(valid, torch.uint8, "valid"), _ptr(node_off, torch.int32, "node_off"),
        n_nodes_total, t_max, _ptr(h, None, "h"), _ptr(depth, torch.int32, "depth"),
        _ptr(tau, torch.float32, "tau"), k_min, k_max, _ptr(h_out, h.dtype, "h_out"),
        _ptr(k_out, torch.int32, "k_out"), _ptr(idx_out, torch.int32, "idx_out"),
        _ptr(gate_out, torch.float32, "gate_out"), _ptr(mass_out, torch.float32, "mass_out"),
        _ptr(r_out, torch.float32, "r_out"), _ptr(workspace, None, "workspace"), ws_bytes,
        _stream(stream))
    _check(st, "fovea_retrieve_fuse")


FOVEA_STATIC_WORKSPACE_BYTES = 64 << 20


def fovea_retrieve_fuse_noalloc(ctx: int, B: int, mem_off, n_mem_total: int, m_max: int, keys,
                                values, valid, node_off, n_nodes_total: int, t_max: int, h, depth,
                                tau, k_min: int, k_max: int, h_out, k_out=None, idx_out=None,
                                gate_out=None, mass_out=None, r_out=None, stream=None) -> None:
    """fovea_retrieve_fuse on the library's fixed per-GPU workspace (no allocation)."""
    st = lib.fovea_retrieve_fuse_noalloc(
        ctx, B, _ptr(mem_off, torch.int64, "mem_off"), n_mem_total, m_max,
        _ptr(keys, h.dtype, "keys"), _ptr(values, h.dtype, "values"),
        _ptr(valid, torch.uint8, "valid"), _ptr(node_off, torch.int32, "node_off"),
        n_nodes_total, t_max, _ptr(h, None, "h"), _ptr(depth, torch.int32, "depth"),
        _ptr(tau, torch.float32, "tau"), k_min, k_max, _ptr(h_out, h.dtype, "h_out"),
        _ptr(k_out, torch.int32, "k_out"), _ptr(idx_out, torch.int32, "idx_out"),
        _ptr(gate_out, torch.float32, "gate_out"), _ptr(mass_out, torch.float32, "mass_out"),
        _ptr(r_out, torch.float32, "r_out"), _stream(stream))
    _check(st, "fovea_retrieve_fuse_noalloc")


def fovea_lm_topk_workspace(ctx: int, n_rows: int, vocab: int, k: int) -> int:
    return lib.fovea_lm_topk_workspace(ctx, n_rows, vocab, k)


def fovea_lm_topk(ctx: int, n_rows: int, h, W_LM, vocab: int, k: int, idx_out, logit_out=None,
                  workspace=None, stream=None) -> None:
    """Same arguments as the C entry point; tensors stand for device pointers."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.fovea_lm_topk(
        ctx, n_rows, _ptr(h, None, "h"), _ptr(W_LM, h.dtype, "W_LM"), vocab, k,
        _ptr(idx_out, torch.int32, "idx_out"), _ptr(logit_out, torch.float32, "logit_out"),
        _ptr(workspace, None, "workspace"), ws_bytes, _stream(stream))
    _check(st, "fovea_lm_topk")


def fovea_retrieve_fuse_backward_workspace(ctx: int, B: int, n_nodes_total: int, m_max: int,
                                           k_max: int) -> int:
    return lib.fovea_retrieve_fuse_backward_workspace(ctx, B, n_nodes_total, m_max, k_max)


def fovea_retrieve_fuse_backward(ctx: int, params: dict, b_g2: float, B: int, mem_off,
                                 n_mem_total: int, m_max: int, keys, values, node_off,
                                 n_nodes_total: int, t_max: int, h, depth, K, idx, k_max: int,
                                 dh_hat, dh, dkeys, dvalues, grads: dict, workspace=None,
                                 stream=None) -> None:
    """Same arguments as the C entry point; params / grads: dicts of fp32 device tensors
    named as in PARAM_TENSORS (+ "rms_w") / GRAD_TENSORS."""
    f32 = torch.float32
    P = Params()
    for nme in PARAM_TENSORS:
        setattr(P, nme, _ptr(params.get(nme), f32, nme))
    P.b_g2 = float(b_g2)
    P.rms_w = _ptr(params.get("rms_w"), f32, "rms_w")
    G = Grads()
    for nme in GRAD_TENSORS:
        setattr(G, nme, _ptr(grads.get(nme), f32, "grad " + nme))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.fovea_retrieve_fuse_backward(
        ctx, ctypes.byref(P), B, _ptr(mem_off, torch.int64, "mem_off"), n_mem_total, m_max,
        _ptr(keys, f32, "keys"), _ptr(values, f32, "values"), _ptr(node_off, torch.int32, "node_off"),
        n_nodes_total, t_max, _ptr(h, f32, "h"), _ptr(depth, torch.int32, "depth"),
        _ptr(K, torch.int32, "K"), _ptr(idx, torch.int32, "idx"), k_max, _ptr(dh_hat, f32, "dh_hat"),
        _ptr(dh, f32, "dh"), _ptr(dkeys, f32, "dkeys"), _ptr(dvalues, f32, "dvalues"),
        ctypes.byref(G), _ptr(workspace, None, "workspace"), ws_bytes, _stream(stream))
    _check(st, "fovea_retrieve_fuse_backward")


def fovea_build_memory_backward_workspace(ctx: int, n_rows: int) -> int:
    return lib.fovea_build_memory_backward_workspace(ctx, n_rows)


def fovea_build_memory_backward(ctx: int, params: dict, V, dkeys, dvalues, dW_K, dW_U, dmem_ln_g,
                                dmem_ln_b, dV=None, workspace=None, stream=None) -> None:
    """Same arguments as the C entry point; params: dict of fp32 device tensors."""
    f32 = torch.float32
    P = Params()
    for nme in PARAM_TENSORS:
        setattr(P, nme, _ptr(params.get(nme), f32, nme))
    P.b_g2 = 0.0
    P.rms_w = None
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = lib.fovea_build_memory_backward(
        ctx, ctypes.byref(P), V.shape[0], _ptr(V, f32, "V"), _ptr(dkeys, f32, "dkeys"),
        _ptr(dvalues, f32, "dvalues"), _ptr(dW_K, f32, "dW_K"), _ptr(dW_U, f32, "dW_U"),
        _ptr(dmem_ln_g, f32, "dmem_ln_g"), _ptr(dmem_ln_b, f32, "dmem_ln_b"), _ptr(dV, f32, "dV"),
        _ptr(workspace, None, "workspace"), ws_bytes, _stream(stream))
    _check(st, "fovea_build_memory_backward")


def fovea_last_error(ctx: int, stream=None) -> tuple[int, int]:
    bits = ctypes.c_uint32(0)
    st = lib.fovea_last_error(ctx, _stream(stream), ctypes.byref(bits))
    return st, bits.value


def fovea_profile(ctx: int, enable: bool) -> None:
    _check(lib.fovea_profile(ctx, 1 if enable else 0), "fovea_profile")


def fovea_profile_read(ctx: int, max_kernels: int = 16) -> dict:
    """{kernel name: (total milliseconds, launches)} recorded since the last read."""
    names = (ctypes.c_char_p * max_kernels)()
    ms = (ctypes.c_float * max_kernels)()
    cnt = (ctypes.c_int32 * max_kernels)()
    n = lib.fovea_profile_read(ctx, max_kernels, names, ms, cnt)
    if n < 0:
        raise FoveaError(FOVEA_ERR_DEVICE, "fovea_profile_read")
    return {names[i].decode(): (ms[i], cnt[i]) for i in range(n)}


# ------------------------------------------------------------------------------------
# convenience wrapper used by the tests and the benchmark
# ------------------------------------------------------------------------------------


@dataclass
class Outputs:
    h_out: torch.Tensor
    k: torch.Tensor
    idx: torch.Tensor
    gate: torch.Tensor
    mass: torch.Tensor
    r: torch.Tensor


class Fovea:
    """Owns one context, its device weight copies and a workspace."""

    def __init__(self, dims: dict, weights: dict, device="cuda", stream=None):
        self.dims = Dims(dims["d"], dims["d_v"], dims["d_m"], dims["d_c"], dims["n_depth"],
                         dims["dtype"], dims["ln_eps"], dims["rms_eps"])
        self.dtype = storage_dtype(dims["dtype"])
        self.device = torch.device(device)
        self.params = {}
        for n in PARAM_TENSORS + ["rms_w"]:
            v = weights.get(n)
            if v is None:
                continue
            self.params[n] = torch.as_tensor(v).to(device=self.device, dtype=self.dtype).contiguous()
        self.b_g2 = float(weights["b_g2"])
        self.ctx = fovea_create(self.dims, self.params, self.b_g2, stream)
        self.workspace = None
        self.lm_workspace = None

    def close(self):
        if getattr(self, "ctx", None):
            fovea_destroy(self.ctx)
            self.ctx = None

    __del__ = close

    def ensure_workspace(self, B: int, n_nodes_total: int, n_mem_total: int, m_max: int,
                         k_max: int) -> torch.Tensor:
        need = fovea_retrieve_fuse_workspace(self.ctx, B, n_nodes_total, n_mem_total, m_max, k_max)
        if self.workspace is None or self.workspace.numel() < need:
            self.workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        return self.workspace

    def build_memory(self, V: torch.Tensor, keys: torch.Tensor | None = None,
                     values: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                     stream=None):
        if keys is None:
            keys = torch.empty(V.shape[0], self.dims.d_m, dtype=V.dtype, device=V.device)
        if values is None:
            values = torch.empty_like(keys)
        if workspace is None:
            need = fovea_build_memory_workspace(self.ctx, V.shape[0])
            workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        fovea_build_memory(self.ctx, V, keys, values, workspace, stream)
        return keys, values

    def alloc_outputs(self, n: int, k_max: int, d: int, d_m: int) -> Outputs:
        dev = self.device
        return Outputs(
            h_out=torch.empty(n, d, dtype=self.dtype, device=dev),
            k=torch.empty(n, dtype=torch.int32, device=dev),
            idx=torch.empty(n, k_max, dtype=torch.int32, device=dev),
            gate=torch.empty(n, dtype=torch.float32, device=dev),
            mass=torch.empty(n, dtype=torch.float32, device=dev),
            r=torch.empty(n, d_m, dtype=torch.float32, device=dev))

    def retrieve_fuse(self, inp: dict, out: Outputs | None = None, debug: bool = True,
                      stream=None) -> Outputs:
        """inp: device tensors mem_off, keys, values, valid (or None), node_off, h, depth,
        tau and host ints m_max, t_max, k_min, k_max."""
        n = inp["h"].shape[0]
        k_max = inp["k_max"]
        if out is None:
            out = self.alloc_outputs(n, k_max, self.dims.d, self.dims.d_m)
        ws = self.ensure_workspace(inp["mem_off"].numel() - 1, n, inp["keys"].shape[0], inp["m_max"], k_max)
        fovea_retrieve_fuse(
            self.ctx, inp["mem_off"].numel() - 1, inp["mem_off"], inp["keys"].shape[0],
            inp["m_max"], inp["keys"], inp["values"], inp.get("valid"), inp["node_off"], n,
            inp["t_max"], inp["h"], inp["depth"], inp["tau"], inp["k_min"], k_max, out.h_out,
            out.k if debug else None, out.idx if debug else None, out.gate if debug else None,
            out.mass if debug else None, out.r if debug else None, ws, stream)
        return out

    def lm_topk(self, h: torch.Tensor, W_LM: torch.Tensor, k: int, idx: torch.Tensor | None = None,
                logit: torch.Tensor | None = None, want_logits: bool = True, stream=None):
        """Top-k token ids (and logits) of W_LM h for every row of h ([n, d])."""
        n, vocab = h.shape[0], W_LM.shape[0]
        if idx is None:
            idx = torch.empty(n, k, dtype=torch.int32, device=self.device)
        if logit is None and want_logits:
            logit = torch.empty(n, k, dtype=torch.float32, device=self.device)
        need = fovea_lm_topk_workspace(self.ctx, n, vocab, k)
        if self.lm_workspace is None or self.lm_workspace.numel() < need:
            self.lm_workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        fovea_lm_topk(self.ctx, n, h, W_LM, vocab, k, idx, logit, self.lm_workspace, stream)
        return idx, logit

    def retrieve_fuse_backward(self, inp: dict, K: torch.Tensor, idx: torch.Tensor,
                               dh_hat: torch.Tensor, stream=None) -> dict:
        """Gradients of one step (fp32 context): inp as for retrieve_fuse; K / idx the
        selection to hold fixed.  Returns dh, dkeys, dvalues and "d<weight>" entries."""
        dev, f32 = self.device, torch.float32
        n, d = inp["h"].shape
        d_m, d_c, nd = self.dims.d_m, self.dims.d_c, self.dims.n_depth
        shapes = dict(W_Q=(d_m, d), q_ln_g=(d,), q_ln_b=(d,), E_dep=(nd, d), W_c1=(d_c, d + d_m),
                      b_c1=(d_c,), W_c2=(d, d_c), b_c2=(d,), W_g1=(d_c, d + d_m), b_g1=(d_c,),
                      w_g2=(d_c,), b_g2=(1,), rms_w=(d,))
        grads = {k: torch.empty(v, dtype=f32, device=dev) for k, v in shapes.items()
                 if k != "rms_w" or "rms_w" in self.params}
        n_mem = inp["keys"].shape[0]
        dh = torch.empty(n, d, dtype=f32, device=dev)
        dkeys = torch.empty(n_mem, d_m, dtype=f32, device=dev)
        dvalues = torch.empty(n_mem, d_m, dtype=f32, device=dev)
        B = inp["mem_off"].numel() - 1
        need = fovea_retrieve_fuse_backward_workspace(self.ctx, B, n, inp["m_max"], idx.shape[1])
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
        fovea_retrieve_fuse_backward(
            self.ctx, self.params, self.b_g2, B, inp["mem_off"], n_mem, inp["m_max"], inp["keys"],
            inp["values"], inp["node_off"], n, inp["t_max"], inp["h"], inp["depth"], K, idx,
            idx.shape[1], dh_hat, dh, dkeys, dvalues, grads, ws, stream)
        out = {"d" + k: v for k, v in grads.items()}
        out.update(dh=dh, dkeys=dkeys, dvalues=dvalues)
        return out


    def build_memory_backward(self, V: torch.Tensor, dkeys: torch.Tensor, dvalues: torch.Tensor,
                              want_dV: bool = True, stream=None) -> dict:
        """Gradients of the memory build (fp32 context): dW_K, dW_U, dmem_ln_g, dmem_ln_b
        and (optionally) dV."""
        dev, f32 = self.device, torch.float32
        d_m, d_v = self.dims.d_m, self.dims.d_v
        out = dict(dW_K=torch.empty(d_m, d_v, dtype=f32, device=dev),
                   dW_U=torch.empty(d_m, d_v, dtype=f32, device=dev),
                   dmem_ln_g=torch.empty(d_v, dtype=f32, device=dev),
                   dmem_ln_b=torch.empty(d_v, dtype=f32, device=dev))
        dV = torch.empty(V.shape[0], d_v, dtype=f32, device=dev) if want_dV else None
        ws = torch.empty(max(fovea_build_memory_backward_workspace(self.ctx, V.shape[0]), 256),
                         dtype=torch.uint8, device=dev)
        fovea_build_memory_backward(self.ctx, self.params, V, dkeys, dvalues, out["dW_K"], out["dW_U"],
                                    out["dmem_ln_g"], out["dmem_ln_b"], dV, ws, stream)
        if dV is not None:
            out["dV"] = dV
        return out
