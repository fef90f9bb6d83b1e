"""Shared helpers of the GPU tests: seeded device inputs for one layer, the
library calls of one decode step, and the oracle's answer on the same values."""
from __future__ import annotations

import dataclasses
import sys

import numpy as np
import torch

import oracle as O
from paper_2603_19664_amd import inputs
from paper_2603_19664_amd import kvd

TOL = {kvd.KVD_F32: 1e-5, kvd.KVD_BF16: 2e-2}


def note(msg: str):
    print(msg, file=sys.__stderr__, flush=True)


def err(x, ref) -> float:
    """max |x - ref| / max |ref| over the tensor."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.max(np.abs(x - ref)) / max(np.max(np.abs(ref)), 1e-300))


def f64(t):
    return inputs.to_f64(t)


@dataclasses.dataclass
class Layer:
    wl: object
    shape: kvd.Shape
    B: int
    T: int            # checkpointed context rows (recomputed)
    h: torch.Tensor   # [B, T, d]
    h_new: torch.Tensor
    gamma: torch.Tensor
    w_q: torch.Tensor
    w_k: torch.Tensor
    w_v: torch.Tensor
    pos0: torch.Tensor      # [B] int32 (device)
    pos_new: torch.Tensor   # [B] int32 (device) = pos0 + T
    lw_q: torch.Tensor = None   # the weights as the library receives them (packed or row-major)
    lw_k: torch.Tensor = None
    lw_v: torch.Tensor = None


def make_layer(wl, B, T, seed=0, layer=0, w_q_std=None, pos0=None, t_cap=None, packed=None, **over) -> Layer:
    """Seeded inputs of one layer.  bf16 weights go to the library in the packed MFMA
    layout unless packed=False; packed="gamma" folds gamma into them
    (kvd_pack_weights_gamma).  The oracle always gets the row-major values and gamma."""
    if over:
        wl = dataclasses.replace(wl, **over)
    dev = "cuda"
    gamma, w_q, w_k, w_v = inputs.weights(wl, layer, seed, dev, w_std=w_q_std)
    h, h_new = inputs.residuals(wl, layer, B, T, seed, dev, t_cap=t_cap)
    p0 = inputs.positions(wl, B, seed) if pos0 is None else torch.as_tensor(pos0, dtype=torch.int32)
    shape = kvd.shape_of(wl)
    if packed is None:
        packed = shape.dtype == kvd.KVD_BF16
    lw = (w_q, w_k, w_v)
    if packed == "gamma":
        shape = shape.packed_gamma()
        lw = tuple(kvd.kvd_pack_weights_gamma(shape, w, gamma) for w in lw)
    elif packed:
        shape = shape.packed()
        lw = tuple(kvd.kvd_pack_weights(shape, w) for w in lw)
    return Layer(wl, shape, B, T, h, h_new, gamma, w_q, w_k, w_v, p0.to(dev), (p0 + T).to(torch.int32).to(dev),
                 *lw)


def empty_kv(L: Layer, t_cap: int):
    s = L.shape
    z = torch.zeros((L.B, s.n_kv_heads, t_cap, s.head_dim), dtype=s.torch_dtype, device="cuda")
    return z, z.clone()


# ------------------------------------------------------------------ library steps

def gpu_recompute(L: Layer, t_cap=None, t_off=0):
    K, V = empty_kv(L, t_cap or (L.T + t_off))
    kvd.kvd_recompute_kv(L.shape, L.h, L.gamma, L.lw_k, L.lw_v, L.pos0, L.T, K, V, t_off)
    return K, V


def gpu_project(L: Layer, kv=None, t_off=0):
    s = L.shape
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    k, v = kv if kv is not None else (None, None)
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, L.pos_new, q, k, v, t_off)
    return q


def gpu_unfused(L: Layer):
    """recompute_kv of the context + project_qkv of the current token into row T, then decode_attn."""
    s = L.shape
    K, V = gpu_recompute(L, t_cap=L.T + 1)
    q = gpu_project(L, (K, V), t_off=L.T)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_DECODE_ATTN, L.B, L.T + 1)
    kvd.kvd_decode_attn(s, q, K, V, L.T + 1, out, ws)
    return q, K, V, out


def gpu_fused(L: Layer, q=None, kv_debug=False, with_current=True):
    """project_qkv (q + the current token's K/V as a one-row tail) + fused recompute-attention."""
    s = L.shape
    tk, tv = empty_kv(L, 1)
    q_ = gpu_project(L, (tk, tv), 0)
    q = q_ if q is None else q
    out = torch.empty_like(q)
    T_tail = 1 if with_current else 0
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, L.T, T_tail)
    dk = dv = None
    if kv_debug:
        dk, dv = empty_kv(L, max(L.T, 1))
    kvd.kvd_fused_recompute_attn(s, q, L.h, L.T, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws,
                                 tk if with_current else None, tv if with_current else None, T_tail, 0, dk, dv, 0)
    return q, (tk, tv), out, (dk, dv)


# ------------------------------------------------------------------ oracle on the same values

def oracle_kv(L: Layer, b_sel=None):
    s = L.shape
    bs = range(L.B) if b_sel is None else b_sel
    h = f64(L.h[list(bs), :L.T])
    pos = f64(L.pos0)[list(bs)][:, None] + np.arange(L.T)[None, :]
    return O.recompute_kv(h, f64(L.gamma), f64(L.w_k), f64(L.w_v), pos, s.n_kv_heads, s.head_dim, s.rms_eps,
                          s.rope_theta)


def oracle_qkv(L: Layer):
    s = L.shape
    return O.project_qkv(f64(L.h_new), f64(L.gamma), f64(L.w_q), f64(L.w_k), f64(L.w_v), f64(L.pos_new),
                         s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps, s.rope_theta)


def oracle_decode(L: Layer, b_sel=None, with_current=True):
    """One decode step of Algorithm 1 at budget 0, from the inputs alone (fp64)."""
    s = L.shape
    bs = list(range(L.B)) if b_sel is None else list(b_sel)
    q, kt, vt = oracle_qkv(L)
    h = f64(L.h[bs, :L.T])
    pos = f64(L.pos0)[bs][:, None] + np.arange(L.T)[None, :]
    tail_k = kt[bs][:, :, None] if with_current else None
    tail_v = vt[bs][:, :, None] if with_current else None
    return O.kv_direct_decode(q[bs], h, f64(L.gamma), f64(L.w_k), f64(L.w_v), pos, tail_k, tail_v,
                              s.n_kv_heads, s.head_dim, s.rms_eps, s.rope_theta)
