"""Seeded synthetic inputs shared by the HIP path's tests/benchmark and the oracle.

This module holds no arithmetic of the method: it only draws random tensors.
Each tensor has its own generator, seeded from (seed, workload id, layer,
tensor id), so draws do not depend on the order in which they are made.
Values are drawn in float32 from torch's generator on the requested device and
rounded (round-to-nearest-even) to the workload dtype; the oracle receives the
rounded values, upcast exactly.
"""
from __future__ import annotations

import numpy as np
import torch

# tensor ids (part of the seed)
T_H, T_HNEW, T_GAMMA, T_WQ, T_WK, T_WV, T_POS, T_SCALE = range(8)
T_WO, T_GAMMA_MLP, T_WGATE, T_WUP, T_WDOWN = range(8, 13)

_DT = {"f32": torch.float32, "bf16": torch.bfloat16}


def torch_dtype(name: str) -> torch.dtype:
    return _DT[name]


def seed_of(*ints: int) -> int:
    """A 63-bit seed derived from a tuple of integers (order-independent draws)."""
    return int(np.random.SeedSequence([int(i) for i in ints]).generate_state(2, np.uint64)[0] >> 1)


def _gen(device, *ints):
    g = torch.Generator(device=device)
    g.manual_seed(seed_of(*ints))
    return g


def normal(shape, std, device, *ids, mean=0.0):
    g = _gen(device, *ids)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        x.mul_(std)
    if mean != 0.0:
        x.add_(mean)
    return x


def uniform(shape, lo, hi, device, *ids):
    g = _gen(device, *ids)
    return torch.rand(shape, generator=g, device=device, dtype=torch.float64) * (hi - lo) + lo


def layer_scale(wl, layer: int, seed: int = 0) -> float:
    """Per-layer residual scale s_l ~ U(lo, hi) (one scalar per layer)."""
    lo, hi = wl.layer_scale
    if lo == hi:
        return float(lo)
    return float(uniform((1,), lo, hi, "cpu", seed, wl.cfg_id, layer, T_SCALE)[0])


def weights(wl, layer: int, seed: int = 0, device="cpu", w_std=None):
    """gamma [d], W_q [n_q*hd, d], W_k / W_v [n_kv*hd, d] in the workload dtype."""
    dt = _DT[wl.dtype]
    d, hd = wl.d_model, wl.head_dim
    std = wl.w_std if w_std is None else w_std
    ids = (seed, wl.cfg_id, layer)
    gamma = normal((d,), wl.gamma_std, device, *ids, T_GAMMA, mean=1.0).to(dt)
    w_q = normal((wl.n_q * hd, d), std, device, *ids, T_WQ).to(dt)
    w_k = normal((wl.n_kv * hd, d), wl.w_std, device, *ids, T_WK).to(dt)
    w_v = normal((wl.n_kv * hd, d), wl.w_std, device, *ids, T_WV).to(dt)
    return gamma, w_q, w_k, w_v


def block_weights(wl, layer: int, d_ff: int, seed: int = 0, device="cpu", w_std=None):
    """The rest of a transformer block's parameters: W_o [d, n_q*hd], gamma_mlp [d],
    W_gate / W_up [d_ff, d], W_down [d, d_ff], in the workload dtype (N(0, w_std^2);
    gamma 1 + N(0, gamma_std^2))."""
    dt = _DT[wl.dtype]
    d, qd = wl.d_model, wl.n_q * wl.head_dim
    std = wl.w_std if w_std is None else w_std
    ids = (seed, wl.cfg_id, layer)
    w_o = normal((d, qd), std, device, *ids, T_WO).to(dt)
    gamma_mlp = normal((d,), wl.gamma_std, device, *ids, T_GAMMA_MLP, mean=1.0).to(dt)
    w_gate = normal((d_ff, d), std, device, *ids, T_WGATE).to(dt)
    w_up = normal((d_ff, d), std, device, *ids, T_WUP).to(dt)
    w_down = normal((d, d_ff), std, device, *ids, T_WDOWN).to(dt)
    return w_o, gamma_mlp, w_gate, w_up, w_down


def residuals(wl, layer: int, B: int, T: int, seed: int = 0, device="cpu", t_cap=None):
    """Checkpointed residuals h [B, t_cap, d] (first T rows drawn) and the new token's h_new [B, d].

    h ~ N(0, 1) * s_l with s_l the per-layer scale.  Rows T..t_cap-1 are zero.
    """
    dt = _DT[wl.dtype]
    t_cap = T if t_cap is None else t_cap
    s = layer_scale(wl, layer, seed)
    ids = (seed, wl.cfg_id, layer, B, T)
    h = torch.zeros((B, t_cap, wl.d_model), device=device, dtype=dt)
    if T > 0:
        h[:, :T] = normal((B, T, wl.d_model), s, device, *ids, T_H).to(dt)
    h_new = normal((B, wl.d_model), s, device, *ids, T_HNEW).to(dt)
    return h, h_new


def positions(wl, B: int, seed: int = 0):
    """pos0[b]: absolute position of each sequence's first checkpointed token (int32, host)."""
    if wl.pos_offset_max <= 0:
        return torch.zeros((B,), dtype=torch.int32)
    g = _gen("cpu", seed, wl.cfg_id, B, T_POS)
    return torch.randint(0, wl.pos_offset_max, (B,), generator=g, dtype=torch.int32)


def to_f64(t: torch.Tensor) -> np.ndarray:
    """Exact upcast of a (possibly bf16, possibly device) tensor to a float64 numpy array."""
    return t.detach().to("cpu").to(torch.float64).numpy()
