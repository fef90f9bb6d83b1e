"""GPU parity of the wide fused engine (128 recomputed tokens per workgroup,
8 waves, bf16, head_dim 128 / 256): forced with kvd_set_fused_tokens(128) on
small shapes that span several tiles and a ragged one, and reached by the
automatic policy on a shape with a full round of wide tiles.

- The K/V it recomputes in LDS (dumped through kv_debug) are bit-identical to
  the prefill K/V of kvd_recompute_kv (Prop. reconstruction: the same MFMA
  chain over d per element), row-major or packed weights.
- Its attention output matches the fp64 oracle's decode step (Eqs.
  attn_weights / head_output) and the 64-token tiling to the bf16 tolerance.
- Stored tails (Algorithm 1's bounded cache, also as a wrapped ring), the
  partials-then-kvd_combine path and sliding-window layers go through it too.
  A tail of <= 4 rows (the current token) folds into the last 128-token chunk,
  also a partial one; a longer tail's remainder of <= 4 rows joins its last
  64-row tile.

Tolerance (max |gpu - oracle| / max |oracle|): 2e-2 for bf16 inputs."""
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import (TOL, empty_kv, err, f64, gpu_fused, gpu_recompute, gpu_unfused, make_layer, note,
                       oracle_decode, oracle_kv)

pytestmark = pytest.mark.gpu

BF = kvd.KVD_BF16
TOL_BF = TOL[BF]


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()
    kvd.kvd_set_fused_tokens(0)


def check(name, x, ref, tol=TOL_BF):
    e = err(f64(x) if isinstance(x, torch.Tensor) else x, ref)
    note(f"    {name}: err {e:.3e} (tol {tol:g})")
    assert e < tol, f"{name}: err {e:.3e} >= {tol:g}"


def _bits(t):
    return t.view(torch.int16)


def _layer(hd, T, seed, B=2, packed=False, **kw):
    n_q, n_kv = (8, 4) if hd == 256 else (12, 2)
    base = dict(d_model=512, n_q=n_q, n_kv=n_kv, head_dim=hd)
    base.update(kw)
    wl = C.GEMMA3_4B if hd == 256 else C.QWEN_1_5B
    return make_layer(wl, B=B, T=T, seed=seed, pos0=[3, 700][:B] + [11] * max(0, B - 2), packed=packed, **base)


@pytest.mark.parametrize("hd", [128, 256])
@pytest.mark.parametrize("packed", [False, True])
@pytest.mark.parametrize("T", [128, 300])
def test_wide_kv_bitwise_and_output(hd, packed, T):
    L = _layer(hd, T, seed=80 + T + hd, packed=packed)
    s = L.shape
    Kp, Vp = gpu_recompute(L)
    kvd.kvd_set_fused_tokens(128)
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T, 1) == -(-T // 128)  # the current token folds
    q, _, out, (dk, dv) = gpu_fused(L, kv_debug=True)
    assert torch.equal(_bits(dk), _bits(Kp)) and torch.equal(_bits(dv), _bits(Vp))
    check("wide fused vs oracle", out, oracle_decode(L))
    kvd.kvd_set_fused_tokens(64)
    _, _, out64, (dk64, dv64) = gpu_fused(L, q=q, kv_debug=True)
    assert torch.equal(_bits(dk64), _bits(dk)) and torch.equal(_bits(dv64), _bits(dv))
    check("wide vs 64-token tiles", out, f64(out64))


def _tail_tiles(n_rec, T_tail):
    if n_rec > 0 and 0 < T_tail <= 4:
        return 0  # folded into the last recomputed chunk
    return T_tail // 64 if T_tail > 64 and 0 < T_tail % 64 <= 4 else -(-T_tail // 64)


@pytest.mark.parametrize("T_rec,T", [(130, 430), (128, 131), (256, 262), (300, 300), (1, 70), (128, 320),
                                     (300, 302)])
def test_wide_stored_tail(T_rec, T):
    # recompute the oldest T_rec context rows, read the rest and the current
    # token as a stored tail: folded into the last chunk when it has <= 4 rows
    # (after a full chunk (128, 131), over a partial one (300, 300), (300, 302)),
    # else 64-row tiles of its own, a remainder of <= 4 rows joining the last
    # of them (128, 320)
    L = _layer(256, T, seed=90 + T_rec)
    s = L.shape
    q, K, V, out_u = gpu_unfused(L)
    T_tail = T - T_rec + 1
    kvd.kvd_set_fused_tokens(128)

    def fused(out, ws):
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)

    S = kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    assert S == -(-T_rec // 128) + _tail_tiles(-(-T_rec // 128), T_tail)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    out = torch.empty_like(q)
    fused(out, ws)
    check("wide hybrid vs oracle", out, oracle_decode(L))
    check("wide hybrid vs unfused", out, f64(out_u))
    out2 = torch.empty_like(q)
    fused(out2, ws)  # the counters were left zero
    assert torch.equal(_bits(out), _bits(out2))
    fused(None, ws)  # partials only, merged by kvd_combine
    out3 = torch.empty_like(q)
    kvd.kvd_combine(s, L.B, S, ws, out3)
    assert torch.equal(_bits(out), _bits(out3))
    ctr_bytes = -(-L.B * s.n_kv_heads * 8 // 256) * 256
    assert int(torch.count_nonzero(ws[:ctr_bytes])) == 0


def test_wide_ring_tail():
    # Algorithm 1's bounded cache as a ring: the 40 newest context rows and the
    # current token in a ring of 41 slots whose oldest slot is 25, so the tail
    # view wraps; the older 260 rows are recomputed on the wide engine
    T, n_tail, off = 300, 41, 25
    L = _layer(256, T, seed=97)
    s = L.shape
    q, K, V, _ = gpu_unfused(L)   # K/V rows 0..T-1 the context, row T the current token
    T_rec = T + 1 - n_tail
    ring_k, ring_v = empty_kv(L, n_tail)
    for i in range(n_tail):
        ring_k[:, :, (off + i) % n_tail] = K[:, :, T_rec + i]
        ring_v[:, :, (off + i) % n_tail] = V[:, :, T_rec + i]
    kvd.kvd_set_fused_tokens(128)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, n_tail)
    kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, ring_k, ring_v, n_tail,
                                 off)
    check("wide ring tail vs oracle", out, oracle_decode(L))


def test_wide_by_policy_on_a_full_round():
    # 4 sequences x 8 KV heads x 8 tiles of 128 = 256 wide tiles: the automatic
    # policy takes the wide engine
    L = make_layer(C.QWEN_1_5B, B=4, T=1024, seed=99, d_model=512, n_q=16, n_kv=8, head_dim=128,
                   pos0=[0, 300, 17, 900])
    s = L.shape
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 8
    q, _, out, _ = gpu_fused(L)
    check("auto wide vs oracle (sequences 0, 3)", out[[0, 3]], oracle_decode(L, b_sel=[0, 3]))
    kvd.kvd_set_fused_tokens(128)
    _, _, out128, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(out128))
    kvd.kvd_set_fused_tokens(64)
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 16
    _, _, out64, _ = gpu_fused(L, q=q)
    check("auto wide vs 64-token tiles", out, f64(out64))


@pytest.mark.parametrize("window", [130, 201, 500])
def test_wide_window(window):
    T = 200
    L = _layer(256, T, seed=70 + window)
    s = L.shape
    n_keep = min(T + 1, window)
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    tk, tv = empty_kv(L, 1)
    pos = torch.full((L.B,), n_keep - 1, dtype=torch.int32, device="cuda")
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, pos, q, tk, tv, 0)
    kvd.kvd_set_fused_tokens(128)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T, 1)
    kvd.kvd_fused_window_attn(s, q, L.h, T, L.gamma, L.lw_k, L.lw_v, window, out, ws, tk, tv, 1)
    ref = O.sliding_window_decode(f64(L.h_new), f64(L.h[:, :L.T]), f64(L.gamma), f64(L.w_q), f64(L.w_k),
                                  f64(L.w_v), window, s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps,
                                  s.rope_theta)
    check(f"wide window {window} vs oracle", out, ref)


@pytest.mark.parametrize("hd", [128, 256])
def test_wide_prefill_full_round(hd):
    # kvd_recompute_kv on a call with a full round of 128-token tiles (4 sequences
    # x 8 KV heads x 8 tiles = 256) runs on WideTile's tiles of both halves: its
    # K/V equal, bit for bit, the fused kernel's recomputed K/V (64-token tiles)
    # and the oracle's within the bf16 tolerance
    L = make_layer(C.QWEN_1_5B if hd == 128 else C.GEMMA3_4B, B=4, T=1000, seed=123 + hd, d_model=512, n_q=16,
                   n_kv=8, head_dim=hd, pos0=[0, 300, 17, 900])
    K, V = gpu_recompute(L)
    kvd.kvd_set_fused_tokens(64)
    _, _, _, (dk, dv) = gpu_fused(L, kv_debug=True)
    assert torch.equal(_bits(K), _bits(dk)) and torch.equal(_bits(V), _bits(dv))
    ok, ov = oracle_kv(L, b_sel=[0, 3])
    check("wide prefill K vs oracle", K[[0, 3]], ok)
    check("wide prefill V vs oracle", V[[0, 3]], ov)
