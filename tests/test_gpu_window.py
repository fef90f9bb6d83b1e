"""GPU parity of sliding-window layers (Sec. 3.2, the sliding-window boundary and
Eq. sw_error): kvd_fused_window_attn keeps the newest `window` keys and rotates
each by its index inside the window.  Checked against the oracle's
sliding-window decode step, and bit for bit against kvd_fused_recompute_attn
called on the kept rows at positions 0, 1, ... (the same kernel and arithmetic).

Tolerances (max |gpu - oracle| / max |oracle|): 1e-5 fp32, 2e-2 bf16."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import TOL, empty_kv, err, f64, make_layer, note

pytestmark = pytest.mark.gpu

BF, F32 = kvd.KVD_BF16, kvd.KVD_F32


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def _layer(dtype, T, seed):
    if dtype == BF:
        return make_layer(C.GEMMA3_4B, B=2, T=T, seed=seed, d_model=512)
    return make_layer(C.SMOLLM_FP32, B=2, T=T, seed=seed)


def _current(L, local_pos):
    """q and the current token's K/V (one tail row), rotated at window index local_pos."""
    s = L.shape
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    tk, tv = empty_kv(L, 1)
    pos = torch.full((L.B,), local_pos, dtype=torch.int32, device="cuda")
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, pos, q, tk, tv, 0)
    return q, tk, tv


def _oracle(L, window):
    s = L.shape
    return O.sliding_window_decode(f64(L.h_new), f64(L.h[:, :L.T]), f64(L.gamma), f64(L.w_q), f64(L.w_k),
                                   f64(L.w_v), window, s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps,
                                   s.rope_theta)


def _check(name, x, ref, tol):
    e = err(f64(x), ref)
    note(f"    {name}: err {e:.3e} (tol {tol:g})")
    assert e < tol, f"{name}: err {e:.3e} >= {tol:g}"


@pytest.mark.parametrize("dtype", [BF, F32])
@pytest.mark.parametrize("window", [1, 5, 64, 65, 130, 200, 201, 500])
def test_window_vs_oracle(dtype, window):
    # 200 context rows + the current token; the window keeps min(201, window) keys
    T = 200
    L = _layer(dtype, T, seed=60 + window)
    s = L.shape
    n_keep = min(T + 1, window)
    q, tk, tv = _current(L, n_keep - 1)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T, 1)
    kvd.kvd_fused_window_attn(s, q, L.h, T, L.gamma, L.lw_k, L.lw_v, window, out, ws, tk, tv, 1)
    _check(f"window {window} vs oracle", out, _oracle(L, window), TOL[dtype])

    # the same kernel on the kept rows by hand: residual rows T+1-n_keep.. at positions 0, 1, ...
    drop = T + 1 - n_keep
    out2 = torch.empty_like(q)
    zeros = torch.zeros(L.B, dtype=torch.int32, device="cuda")
    ws2 = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T - drop, 1)
    kept = L.h[:, drop:].contiguous()
    kvd.kvd_fused_recompute_attn(s, q, kept, T - drop, L.gamma, L.lw_k, L.lw_v, zeros, out2, ws2, tk, tv, 1)
    assert torch.equal(out.view(torch.int16 if dtype == BF else torch.int32),
                       out2.view(torch.int16 if dtype == BF else torch.int32))


@pytest.mark.parametrize("dtype", [BF, F32])
@pytest.mark.parametrize("T_rec,window", [(100, 50), (100, 101), (100, 150), (0, 30), (130, 201)])
def test_window_over_recomputed_and_stored_rows(dtype, T_rec, window):
    # hybrid budget: rows 0..T_rec-1 recomputed, rows T_rec..T-1 stored (their K/V
    # written by kvd_recompute_kv at window indices), then the current token.  A
    # window shorter than the stored block drops stored rows as well.
    T = 200
    L = _layer(dtype, T, seed=90 + T_rec + window)
    s = L.shape
    n_keep = min(T + 1, window)
    w = T + 1 - n_keep                     # window start (absolute key index)
    K, V = empty_kv(L, T + 1)
    if T > T_rec:
        pos0 = torch.full((L.B,), T_rec - w, dtype=torch.int32, device="cuda")  # window index of row T_rec
        stored = L.h[:, T_rec:].contiguous()
        kvd.kvd_recompute_kv(s, stored, L.gamma, L.lw_k, L.lw_v, pos0, T - T_rec, K, V, T_rec)
    q, tk, tv = _current(L, n_keep - 1)
    K[:, :, T], V[:, :, T] = tk[:, :, 0], tv[:, :, 0]
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T + 1 - T_rec)
    kvd.kvd_fused_window_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, window, out, ws, K, V, T + 1 - T_rec, T_rec)
    _check(f"T_rec {T_rec} window {window} vs oracle", out, _oracle(L, window), TOL[dtype])
    assert torch.isfinite(out.float()).all()


def test_window_workspace_for_kept_rows_suffices():
    # a workspace sized for the kept rows only (fewer splits than the full call)
    T, window = 700, 100
    L = _layer(BF, T, seed=5)
    s = L.shape
    q, tk, tv = _current(L, window - 1)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, window - 1, 1)
    assert ws.numel() < kvd.kvd_workspace_bytes(s, kvd.KVD_OP_FUSED, L.B, T, 1)
    kvd.kvd_fused_window_attn(s, q, L.h, T, L.gamma, L.lw_k, L.lw_v, window, out, ws, tk, tv, 1)
    _check("window 100 of 701, small workspace", out, _oracle(L, window), TOL[BF])
