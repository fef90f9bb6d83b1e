"""Python binding of libkvd (include/kvd.h): argument marshalling only.

Each function has the name of the C entry point it calls, takes torch tensors
that live on the GPU, checks their device / dtype / layout, passes raw pointers
and torch's current HIP stream through ctypes, and raises KvdError on a non-OK
status.  Every step of the computation runs in the HIP kernels of libkvd; there
is no fallback.  Importing this module fails loudly if libkvd.so is not built.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import re
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libkvd.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "kvd.h")

KVD_OK, KVD_ERR_NULL, KVD_ERR_SHAPE, KVD_ERR_UNSUPPORTED, KVD_ERR_WORKSPACE, KVD_ERR_ALIGN, KVD_ERR_DEVICE = range(7)
KVD_F32, KVD_BF16 = 0, 1
KVD_W_ROWMAJOR, KVD_W_PACKED, KVD_W_PACKED_GAMMA = 0, 1, 2
KVD_OP_DECODE_ATTN, KVD_OP_CACHED_ATTN, KVD_OP_FUSED = 0, 1, 2
KVD_FUSED_SPLIT = -128  # kvd_set_fused_tokens: the split engine, 128-token chunks
KVD_FUSED_SPLIT64 = -64  # the split engine, 64-token chunks
KVD_FUSED_PAIR = -2  # two KV heads per 128-token tile (bf16, head_dim 128, even n_kv_heads)

_DTYPES = {KVD_F32: torch.float32, KVD_BF16: torch.bfloat16}


class KvdError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{status_str(status)}: {msg}")
        self.status = status


class AttnShape(ctypes.Structure):
    _fields_ = [
        ("d_model", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("rms_eps", ctypes.c_float),
        ("rope_theta", ctypes.c_double),
        ("dtype", ctypes.c_int32),
        ("w_layout", ctypes.c_int32),
    ]


class KvView(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("t_cap", ctypes.c_int32), ("t_off", ctypes.c_int32)]


class BlockWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("gamma_attn", "w_q", "w_k", "w_v", "w_o", "gamma_mlp", "w_gate",
                                               "w_up", "w_down")] + [("d_ff", ctypes.c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2603_19664_amd.build` "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_size_t, ctypes.c_void_p
    S, V = P(AttnShape), P(KvView)
    sig = {
        "kvd_recompute_kv": [S, VP, I32, VP, VP, VP, VP, I32, I32, V, VP],
        "kvd_project_qkv": [S, VP, VP, VP, VP, VP, VP, I32, VP, V, VP],
        "kvd_project_q": [S, VP, VP, VP, VP, I32, VP, VP],
        "kvd_decode_attn": [S, VP, V, I32, I32, VP, VP, SZ, VP],
        "kvd_cached_attn": [S, VP, V, I32, I32, VP, VP, SZ, VP],
        "kvd_fused_recompute_attn": [S, VP, VP, I32, VP, VP, VP, VP, I32, I32, V, I32, VP, VP, SZ, V, VP],
        "kvd_fused_window_attn": [S, VP, VP, I32, VP, VP, VP, I32, I32, V, I32, I32, VP, VP, SZ, VP],
        "kvd_fused_recompute_attn_noalloc": [S, VP, VP, I32, VP, VP, VP, VP, I32, I32, V, I32, VP, VP],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    lib.kvd_store_residual.argtypes = [S, VP, VP, I32, I32, I32, VP]
    lib.kvd_store_residual.restype = ctypes.c_int
    lib.kvd_pack_weights.argtypes = [S, VP, I32, VP, VP]
    lib.kvd_pack_weights.restype = ctypes.c_int
    lib.kvd_pack_weights_gamma.argtypes = [S, VP, VP, I32, VP, VP]
    lib.kvd_pack_weights_gamma.restype = ctypes.c_int
    lib.kvd_pack_matrix.argtypes = [VP, I32, I32, VP, VP]
    lib.kvd_pack_matrix.restype = ctypes.c_int
    lib.kvd_block_forward.argtypes = [S, P(BlockWeights), VP, VP, VP, I32, I32, VP, SZ, VP]
    lib.kvd_block_forward.restype = ctypes.c_int
    lib.kvd_block_workspace_bytes.argtypes = [S, I32, I32, I32]
    lib.kvd_block_workspace_bytes.restype = SZ
    lib.kvd_combine.argtypes = [S, I32, I32, VP, SZ, VP, VP]
    lib.kvd_combine.restype = ctypes.c_int
    lib.kvd_workspace_bytes.argtypes = [S, I32, I32, I32, I32]
    lib.kvd_workspace_bytes.restype = SZ
    lib.kvd_num_splits.argtypes = [S, I32, I32, I32, I32]
    lib.kvd_num_splits.restype = I32
    lib.kvd_set_attn_workgroups.argtypes = [I32]
    lib.kvd_set_attn_workgroups.restype = I32
    lib.kvd_set_fused_tokens.argtypes = [I32]
    lib.kvd_set_fused_tokens.restype = I32
    lib.kvd_status_str.argtypes = [ctypes.c_int]
    lib.kvd_status_str.restype = ctypes.c_char_p
    lib.kvd_last_error.argtypes = []
    lib.kvd_last_error.restype = ctypes.c_char_p
    lib.kvd_abi_version.argtypes = []
    lib.kvd_abi_version.restype = ctypes.c_int
    return lib


lib = _load()


def header_symbols(path: str = HEADER_PATH) -> list:
    """Names of the functions include/kvd.h declares."""
    with open(path) as f:
        src = f.read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(kvd_[a-z_]+)\s*\(", src)))


def status_str(status: int) -> str:
    return lib.kvd_status_str(status).decode()


def last_error() -> str:
    return lib.kvd_last_error().decode()


def abi_version() -> int:
    return lib.kvd_abi_version()


@dataclass(frozen=True)
class Shape:
    """One attention layer's shape (kvd_attn_shape)."""
    d_model: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rms_eps: float
    rope_theta: float
    dtype: int
    w_layout: int = KVD_W_ROWMAJOR

    @property
    def torch_dtype(self) -> torch.dtype:
        return _DTYPES[self.dtype]

    def c(self) -> AttnShape:
        return AttnShape(self.d_model, self.n_q_heads, self.n_kv_heads, self.head_dim, self.rms_eps,
                         self.rope_theta, self.dtype, self.w_layout)

    def packed(self) -> "Shape":
        """The same shape with weights in the packed MFMA layout (kvd_pack_weights)."""
        return dataclasses.replace(self, w_layout=KVD_W_PACKED)

    def packed_gamma(self) -> "Shape":
        """The same shape with gamma folded into packed weights (kvd_pack_weights_gamma)."""
        return dataclasses.replace(self, w_layout=KVD_W_PACKED_GAMMA)


def shape_of(wl) -> Shape:
    """The Shape of a configs.Workload."""
    return Shape(wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.rms_eps, wl.rope_theta,
                 KVD_BF16 if wl.dtype == "bf16" else KVD_F32)


def _check(st: int):
    if st != KVD_OK:
        raise KvdError(st, last_error())


def _ptr(t, name, dtype=None, ndim=None):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name} must be a torch tensor on the GPU")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} has {t.dim()} dims, expected {ndim}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _extent(t, name, want):
    """ValueError unless tensor t (if given) has exactly the extents `want` (a tuple); checked
    before any pointer is taken, so a mismatched tensor never reaches a kernel."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a torch tensor")
    if tuple(t.shape) != tuple(want):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(want)}")


def _kv_extent(k, v, name, B, shape: "Shape", min_rows: int, t_off: int, ring: bool = False):
    """k, v: [B, n_kv, t_cap, head_dim] with rows t_off .. t_off + min_rows - 1 inside t_cap
    (ring: the rows wrap modulo t_cap, so t_off < t_cap and min_rows <= t_cap)."""
    if k is None and v is None:
        return
    if k is None or v is None or k.dim() != 4:
        raise ValueError(f"{name}: k and v must both be [B, n_kv, t_cap, head_dim] tensors")
    t_cap = k.shape[2]
    _extent(k, name + "_k", (B, shape.n_kv_heads, t_cap, shape.head_dim))
    _extent(v, name + "_v", (B, shape.n_kv_heads, t_cap, shape.head_dim))
    if ring:
        if t_off < 0 or t_off >= t_cap or min_rows > t_cap:
            raise ValueError(f"{name}: {min_rows} rows from slot {t_off} do not fit a ring of {t_cap} slots")
    elif t_off < 0 or t_off + min_rows > t_cap:
        raise ValueError(f"{name}: rows {t_off} .. {t_off + min_rows - 1} exceed t_cap {t_cap}")


def _weights_extent(shape: "Shape", **mats):
    """gamma [d]; w_q [n_q*hd, d]; w_k, w_v [n_kv*hd, d] (packed weights keep these extents).
    With gamma folded into the weights (KVD_W_PACKED_GAMMA) gamma may be None."""
    d, hd = shape.d_model, shape.head_dim
    want = {"gamma": (d,), "w_q": (shape.n_q_heads * hd, d), "w_k": (shape.n_kv_heads * hd, d),
            "w_v": (shape.n_kv_heads * hd, d)}
    for name, t in mats.items():
        if name == "gamma" and t is None and shape.w_layout == KVD_W_PACKED_GAMMA:
            continue
        _extent(t, name, want[name])


def _pos_extent(pos, name, B):
    if pos is None:
        raise ValueError(f"{name} is required")
    _extent(pos, name, (B,))


def _qo_extent(t, name, B, shape: "Shape"):
    _extent(t, name, (B, shape.n_q_heads, shape.head_dim))


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _view(k, v, t_off, name, dt):
    if k is None and v is None:
        return None
    if k is None or v is None or k.shape != v.shape or k.dim() != 4:
        raise ValueError(f"{name}: k and v must both be [B, n_kv, t_cap, head_dim] tensors")
    return KvView(_ptr(k, name + "_k", dt), _ptr(v, name + "_v", dt), k.shape[2], t_off)


def kvd_workspace_bytes(shape: Shape, op: int, B: int, T_main: int, T_tail: int = 0) -> int:
    return lib.kvd_workspace_bytes(ctypes.byref(shape.c()), op, B, T_main, T_tail)


def kvd_num_splits(shape: Shape, op: int, B: int, T_main: int, T_tail: int = 0) -> int:
    return lib.kvd_num_splits(ctypes.byref(shape.c()), op, B, T_main, T_tail)


def kvd_set_attn_workgroups(target: int) -> int:
    """Workgroup target of the bf16 stored-K/V attention's split policy (0: the default);
    returns the previous value.  Process-wide; size workspaces after setting it."""
    return lib.kvd_set_attn_workgroups(int(target))


def kvd_set_fused_tokens(tokens: int) -> int:
    """Recomputed tokens per workgroup of the fused calls: 0 chooses per call, 128 the
    wide engine where it exists, KVD_FUSED_PAIR the pair engine (two KV heads per tile)
    where it exists, KVD_FUSED_SPLIT the split engine where a call can use it, 64 the
    64-token tiles; returns the previous setting."""
    return lib.kvd_set_fused_tokens(int(tokens))


def workspace(shape: Shape, op: int, B: int, T_main: int, T_tail: int = 0, device="cuda") -> torch.Tensor:
    """A zero-filled device buffer of kvd_workspace_bytes bytes (torch allocations are
    256-byte aligned; the split counters at its start must be zero before first use)."""
    n = kvd_workspace_bytes(shape, op, B, T_main, T_tail)
    return torch.zeros(max(n, 256), dtype=torch.uint8, device=device)


def _ws(ws):
    if not isinstance(ws, torch.Tensor):
        raise ValueError("ws must be a torch tensor")
    return _ptr(ws, "ws"), ws.numel() * ws.element_size()


def kvd_recompute_kv(shape: Shape, h, gamma, w_k, w_v, pos0, T: int, k_out, v_out, t_off: int = 0):
    """K/V of residual rows 0..T-1 of h [B, h_ld, d] into k_out/v_out [B, n_kv, t_cap, hd] at rows t_off.."""
    dt = shape.torch_dtype
    if not isinstance(h, torch.Tensor) or h.dim() != 3:
        raise ValueError("h must be a [B, h_ld, d_model] tensor")
    B, h_ld = h.shape[0], h.shape[1]
    _extent(h, "h", (B, h_ld, shape.d_model))
    _weights_extent(shape, gamma=gamma, w_k=w_k, w_v=w_v)
    _pos_extent(pos0, "pos0", B)
    _kv_extent(k_out, v_out, "out", B, shape, T, t_off)
    view = _view(k_out, v_out, t_off, "out", dt)
    _check(lib.kvd_recompute_kv(ctypes.byref(shape.c()), _ptr(h, "h", dt, 3), h_ld, _ptr(gamma, "gamma", dt),
                                _ptr(w_k, "w_k", dt), _ptr(w_v, "w_v", dt), _ptr(pos0, "pos0", torch.int32), B, T,
                                ctypes.byref(view) if view is not None else None, _stream()))


def kvd_project_qkv(shape: Shape, h_new, gamma, w_q, w_k, w_v, pos, q_out, k_out=None, v_out=None, t_off: int = 0):
    """q (and, if k_out/v_out are given, the token's K/V at row t_off) of h_new [B, d]."""
    dt = shape.torch_dtype
    if not isinstance(h_new, torch.Tensor) or h_new.dim() != 2:
        raise ValueError("h_new must be a [B, d_model] tensor")
    B = h_new.shape[0]
    _extent(h_new, "h_new", (B, shape.d_model))
    _weights_extent(shape, gamma=gamma, w_q=w_q, w_k=w_k, w_v=w_v)
    _pos_extent(pos, "pos", B)
    _qo_extent(q_out, "q_out", B, shape)
    _kv_extent(k_out, v_out, "kv_out", B, shape, 1, t_off)
    view = _view(k_out, v_out, t_off, "kv_out", dt)
    _check(lib.kvd_project_qkv(ctypes.byref(shape.c()), _ptr(h_new, "h_new", dt, 2), _ptr(gamma, "gamma", dt),
                               _ptr(w_q, "w_q", dt), _ptr(w_k, "w_k", dt), _ptr(w_v, "w_v", dt),
                               _ptr(pos, "pos", torch.int32), B, _ptr(q_out, "q_out", dt, 3),
                               ctypes.byref(view) if view is not None else None, _stream()))


def kvd_project_q(shape: Shape, h_new, gamma, w_q, pos, q_out):
    """q = RoPE(RMSNorm(h_new) W_q^T, pos) of h_new [B, d] into q_out [B, n_q, hd]."""
    dt = shape.torch_dtype
    if not isinstance(h_new, torch.Tensor) or h_new.dim() != 2:
        raise ValueError("h_new must be a [B, d_model] tensor")
    B = h_new.shape[0]
    _extent(h_new, "h_new", (B, shape.d_model))
    _weights_extent(shape, gamma=gamma, w_q=w_q)
    _pos_extent(pos, "pos", B)
    _qo_extent(q_out, "q_out", B, shape)
    _check(lib.kvd_project_q(ctypes.byref(shape.c()), _ptr(h_new, "h_new", dt, 2), _ptr(gamma, "gamma", dt),
                             _ptr(w_q, "w_q", dt), _ptr(pos, "pos", torch.int32), B, _ptr(q_out, "q_out", dt, 3),
                             _stream()))


def _attn(fn, shape, q, k, v, T, out, ws, t_off):
    dt = shape.torch_dtype
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a [B, n_q, head_dim] tensor")
    B = q.shape[0]
    _qo_extent(q, "q", B, shape)
    _qo_extent(out, "out", B, shape)
    _kv_extent(k, v, "kv", B, shape, T, t_off)
    if k is None:
        raise ValueError("kv: k and v are required")
    view = _view(k, v, t_off, "kv", dt)
    wp, wb = _ws(ws)
    _check(fn(ctypes.byref(shape.c()), _ptr(q, "q", dt, 3), ctypes.byref(view), B, T,
              _ptr(out, "out", dt, 3), wp, wb, _stream()))


def kvd_store_residual(shape: Shape, h_new, ckpt, row: int):
    """STORE_RESIDUAL: ckpt[b, row] = h_new[b] for every sequence (h_new [B, d], ckpt [B, c_ld, d])."""
    dt = shape.torch_dtype
    if not isinstance(h_new, torch.Tensor) or h_new.dim() != 2:
        raise ValueError("h_new must be a [B, d_model] tensor")
    B = h_new.shape[0]
    _extent(h_new, "h_new", (B, shape.d_model))
    if not isinstance(ckpt, torch.Tensor) or ckpt.dim() != 3:
        raise ValueError("ckpt must be a [B, c_ld, d_model] tensor")
    _extent(ckpt, "ckpt", (B, ckpt.shape[1], shape.d_model))
    _check(lib.kvd_store_residual(ctypes.byref(shape.c()), _ptr(h_new, "h_new", dt, 2), _ptr(ckpt, "ckpt", dt, 3),
                                  ckpt.shape[1], row, B, _stream()))


def kvd_pack_weights(shape: Shape, w):
    """A packed copy (MFMA operand order) of a row-major [rows, d_model] bf16 weight matrix."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2 or w.shape[1] != shape.d_model:
        raise ValueError(f"w must be a [rows, d_model={shape.d_model}] tensor")
    out = torch.empty_like(w)
    _check(lib.kvd_pack_weights(ctypes.byref(shape.c()), _ptr(w, "w", torch.bfloat16, 2), w.shape[0],
                                _ptr(out, "packed", torch.bfloat16, 2), _stream()))
    return out


def kvd_pack_weights_gamma(shape: Shape, w, gamma):
    """A packed copy of W diag(gamma) (bf16(w * gamma) per element) for the KVD_W_PACKED_GAMMA layout."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2 or w.shape[1] != shape.d_model:
        raise ValueError(f"w must be a [rows, d_model={shape.d_model}] tensor")
    _extent(gamma, "gamma", (shape.d_model,))
    out = torch.empty_like(w)
    _check(lib.kvd_pack_weights_gamma(ctypes.byref(shape.c()), _ptr(w, "w", torch.bfloat16, 2),
                                      _ptr(gamma, "gamma", torch.bfloat16, 1), w.shape[0],
                                      _ptr(out, "packed", torch.bfloat16, 2), _stream()))
    return out


def kvd_combine(shape: Shape, B: int, S: int, ws, out):
    """Merge the S split-K partials an attention call (with out=None) left in ws into out."""
    _qo_extent(out, "out", B, shape)
    wp, wb = _ws(ws)
    _check(lib.kvd_combine(ctypes.byref(shape.c()), B, S, wp, wb, _ptr(out, "out", shape.torch_dtype, 3), _stream()))


def kvd_decode_attn(shape: Shape, q, k, v, T: int, out, ws, t_off: int = 0):
    """Decode attention of q [B, n_q, hd] over stored K/V rows t_off..t_off+T-1 into out
    (out=None: partials only, merged later by kvd_combine)."""
    _attn(lib.kvd_decode_attn, shape, q, k, v, T, out, ws, t_off)


def kvd_cached_attn(shape: Shape, q, k, v, T: int, out, ws, t_off: int = 0):
    """The cached-K/V baseline (bf16 cache): same as kvd_decode_attn."""
    _attn(lib.kvd_cached_attn, shape, q, k, v, T, out, ws, t_off)


def _fused_extents(shape, q, h, T_rec, gamma, w_k, w_v, out, tail_k, tail_v, T_tail, tail_t_off):
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a [B, n_q, head_dim] tensor")
    B = q.shape[0]
    _qo_extent(q, "q", B, shape)
    _qo_extent(out, "out", B, shape)
    if T_rec > 0:
        if not isinstance(h, torch.Tensor) or h.dim() != 3:
            raise ValueError("h must be a [B, h_ld, d_model] tensor")
        _extent(h, "h", (B, h.shape[1], shape.d_model))
        _weights_extent(shape, gamma=gamma, w_k=w_k, w_v=w_v)
    if T_tail > 0 and tail_k is None:
        raise ValueError("tail_k / tail_v are required when T_tail > 0")
    _kv_extent(tail_k, tail_v, "tail", B, shape, T_tail, tail_t_off, ring=True)
    return B


def kvd_fused_recompute_attn(shape: Shape, q, h, T_rec: int, gamma, w_k, w_v, pos0, out, ws,
                             tail_k=None, tail_v=None, T_tail: int = 0, tail_t_off: int = 0,
                             dbg_k=None, dbg_v=None, dbg_t_off: int = 0):
    """Attention of q over K/V recomputed from h rows 0..T_rec-1, followed by T_tail stored tail rows
    (out=None: partials only, merged later by kvd_combine)."""
    dt = shape.torch_dtype
    B = _fused_extents(shape, q, h, T_rec, gamma, w_k, w_v, out, tail_k, tail_v, T_tail, tail_t_off)
    if T_rec > 0:
        _pos_extent(pos0, "pos0", B)
        _kv_extent(dbg_k, dbg_v, "kv_debug", B, shape, T_rec, dbg_t_off)
    tail = _view(tail_k, tail_v, tail_t_off, "tail", dt)
    dbg = _view(dbg_k, dbg_v, dbg_t_off, "kv_debug", dt)
    wp, wb = _ws(ws)
    _check(lib.kvd_fused_recompute_attn(
        ctypes.byref(shape.c()), _ptr(q, "q", dt, 3), _ptr(h, "h", dt, 3), h.shape[1] if h is not None else 0,
        _ptr(gamma, "gamma", dt),
        _ptr(w_k, "w_k", dt), _ptr(w_v, "w_v", dt), _ptr(pos0, "pos0", torch.int32), B, T_rec,
        ctypes.byref(tail) if tail is not None else None, T_tail, _ptr(out, "out", dt, 3) if out is not None else None,
        wp, wb, ctypes.byref(dbg) if dbg is not None else None, _stream()))


def kvd_fused_recompute_attn_noalloc(shape: Shape, q, h, T_rec: int, gamma, w_k, w_v, pos0, out,
                                     tail_k=None, tail_v=None, T_tail: int = 0, tail_t_off: int = 0):
    """kvd_fused_recompute_attn with the library's static per-device scratch as its workspace
    (allocates nothing; calls on one GPU must not overlap)."""
    dt = shape.torch_dtype
    B = _fused_extents(shape, q, h, T_rec, gamma, w_k, w_v, out, tail_k, tail_v, T_tail, tail_t_off)
    if out is None:
        raise ValueError("out is required")
    if T_rec > 0:
        _pos_extent(pos0, "pos0", B)
    tail = _view(tail_k, tail_v, tail_t_off, "tail", dt)
    _check(lib.kvd_fused_recompute_attn_noalloc(
        ctypes.byref(shape.c()), _ptr(q, "q", dt, 3), _ptr(h, "h", dt, 3), h.shape[1] if h is not None else 0,
        _ptr(gamma, "gamma", dt), _ptr(w_k, "w_k", dt), _ptr(w_v, "w_v", dt), _ptr(pos0, "pos0", torch.int32), B,
        T_rec, ctypes.byref(tail) if tail is not None else None, T_tail, _ptr(out, "out", dt, 3), _stream()))


def kvd_fused_window_attn(shape: Shape, q, h, T_rec: int, gamma, w_k, w_v, window: int, out, ws,
                          tail_k=None, tail_v=None, T_tail: int = 0, tail_t_off: int = 0):
    """Sliding-window attention of q over the newest `window` of [h rows 0..T_rec-1 recomputed || T_tail stored
    tail rows], each kept key rotated by its index inside the window (out=None: partials only)."""
    dt = shape.torch_dtype
    B = _fused_extents(shape, q, h, T_rec, gamma, w_k, w_v, out, tail_k, tail_v, T_tail, tail_t_off)
    tail = _view(tail_k, tail_v, tail_t_off, "tail", dt)
    wp, wb = _ws(ws)
    _check(lib.kvd_fused_window_attn(
        ctypes.byref(shape.c()), _ptr(q, "q", dt, 3), _ptr(h, "h", dt, 3), h.shape[1] if h is not None else 0,
        _ptr(gamma, "gamma", dt), _ptr(w_k, "w_k", dt), _ptr(w_v, "w_v", dt), B, T_rec,
        ctypes.byref(tail) if tail is not None else None, T_tail, window,
        _ptr(out, "out", dt, 3) if out is not None else None, wp, wb, _stream()))


def kvd_pack_matrix(w):
    """A packed copy (MFMA operand order) of a row-major [rows, cols] bf16 matrix."""
    if not isinstance(w, torch.Tensor) or w.dim() != 2:
        raise ValueError("w must be a [rows, cols] tensor")
    out = torch.empty_like(w)
    _check(lib.kvd_pack_matrix(_ptr(w, "w", torch.bfloat16, 2), w.shape[0], w.shape[1],
                               _ptr(out, "packed", torch.bfloat16, 2), _stream()))
    return out


def kvd_block_workspace_bytes(shape: Shape, d_ff: int, B: int, T: int) -> int:
    return lib.kvd_block_workspace_bytes(ctypes.byref(shape.c()), d_ff, B, T)


def block_weights(gamma_attn, w_q, w_k, w_v, w_o, gamma_mlp, w_gate, w_up, w_down, shape: Shape = None) -> BlockWeights:
    """The kvd_block_weights of one block (device bf16 tensors, kept alive by the caller).  With `shape`,
    every extent is checked against it: gammas [d], W_q [n_q*hd, d], W_k/W_v [n_kv*hd, d], W_o [d, n_q*hd],
    W_gate/W_up [d_ff, d], W_down [d, d_ff]."""
    ts = (gamma_attn, w_q, w_k, w_v, w_o, gamma_mlp, w_gate, w_up, w_down)
    names = ("gamma_attn", "w_q", "w_k", "w_v", "w_o", "gamma_mlp", "w_gate", "w_up", "w_down")
    if not isinstance(w_gate, torch.Tensor) or w_gate.dim() != 2:
        raise ValueError("w_gate must be a [d_ff, d_model] tensor")
    d_ff = w_gate.shape[0]
    if shape is not None:
        d, qd, kd = shape.d_model, shape.n_q_heads * shape.head_dim, shape.n_kv_heads * shape.head_dim
        want = ((d,), (qd, d), (kd, d), (kd, d), (d, qd), (d,), (d_ff, d), (d_ff, d), (d, d_ff))
        for t, n, wsh in zip(ts, names, want):
            _extent(t, n, wsh)
    ptrs = [_ptr(t, n, torch.bfloat16) for t, n in zip(ts, names)]
    bw = BlockWeights(*ptrs, d_ff)
    bw._extents = tuple(tuple(t.shape) for t in ts)  # checked against the shape by kvd_block_forward
    return bw


def kvd_block_forward(shape: Shape, weights: BlockWeights, h_in, h_out, pos0, ws):
    """h_out [B, T, d] = one pre-norm transformer block over every position of h_in [B, T, d]."""
    if not isinstance(h_in, torch.Tensor) or h_in.dim() != 3:
        raise ValueError("h_in must be a [B, T, d_model] tensor")
    B, T = h_in.shape[0], h_in.shape[1]
    _extent(h_in, "h_in", (B, T, shape.d_model))
    _extent(h_out, "h_out", (B, T, shape.d_model))
    _pos_extent(pos0, "pos0", B)
    ext = getattr(weights, "_extents", None)
    if ext is not None:
        d, qd, kd, d_ff = shape.d_model, shape.n_q_heads * shape.head_dim, shape.n_kv_heads * shape.head_dim, \
            weights.d_ff
        want = ((d,), (qd, d), (kd, d), (kd, d), (d, qd), (d,), (d_ff, d), (d_ff, d), (d, d_ff))
        names = ("gamma_attn", "w_q", "w_k", "w_v", "w_o", "gamma_mlp", "w_gate", "w_up", "w_down")
        for e, wsh, n in zip(ext, want, names):
            if tuple(e) != wsh:
                raise ValueError(f"{n} has shape {tuple(e)}, expected {wsh}")
    wp, wb = _ws(ws)
    _check(lib.kvd_block_forward(ctypes.byref(shape.c()), ctypes.byref(weights), _ptr(h_in, "h_in", torch.bfloat16, 3),
                                 _ptr(h_out, "h_out", torch.bfloat16, 3), _ptr(pos0, "pos0", torch.int32), B, T,
                                 wp, wb, _stream()))
