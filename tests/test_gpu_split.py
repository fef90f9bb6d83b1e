"""GPU parity of the split fused engine (bf16, head_dim 128 / 256): each
128-token chunk runs as two workgroups, one recomputing the K rows and taking
the scores and softmax, one recomputing the V rows and taking P V once the
first has published the probabilities, with 128- or 64-token chunks.  Forced with
kvd_set_fused_tokens(KVD_FUSED_SPLIT / KVD_FUSED_SPLIT64) on small shapes that
span several chunks and a ragged one, and on the Gemma-3-4B layer shape; the
64-token chunks are also reached by the automatic policy on small grids.

- The K/V each role recomputes (dumped through kv_debug) are bit-identical to
  the prefill K/V of kvd_recompute_kv (Prop. reconstruction: the same MFMA
  chain over d per element), for row-major, packed and gamma-folded weights.
- The attention output matches the fp64 oracle's decode step (Eqs.
  attn_weights / head_output) and the 64-token tiling to the bf16 tolerance.
- A stored tail of up to 4 rows (the current token, or a small bounded cache,
  also wrapped as a ring) folds into the last chunk; the partials-then-
  kvd_combine path, repeated calls on one workspace (the completion words are
  cleared by the merging workgroup) and sliding-window layers go through it.

Tolerance (max |gpu - oracle| / max |oracle|): 2e-2 for bf16 inputs."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import TOL, empty_kv, err, f64, gpu_fused, gpu_recompute, gpu_unfused, make_layer, note, oracle_decode

pytestmark = pytest.mark.gpu

BF = kvd.KVD_BF16
TOL_BF = TOL[BF]
SPLIT = kvd.KVD_FUSED_SPLIT
MODES = [(kvd.KVD_FUSED_SPLIT, 128), (kvd.KVD_FUSED_SPLIT64, 64)]


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


def _counters_clear(ws, L):
    s = L.shape
    up = lambda x: -(-x // 256) * 256  # noqa: E731
    n = up(L.B * s.n_kv_heads * 8) + up(L.B * s.n_kv_heads * 4 * 8)  # split counters, completion words
    assert int(torch.count_nonzero(ws[:n])) == 0


@pytest.mark.parametrize("mode,mt", MODES)
@pytest.mark.parametrize("hd", [128, 256])
@pytest.mark.parametrize("packed", [False, True, "gamma"])
@pytest.mark.parametrize("T", [1, 128, 300])
def test_split_kv_bitwise_and_output(mode, mt, hd, packed, T):
    L = _layer(hd, T, seed=180 + T + hd, packed=packed)
    s = L.shape
    Kp, Vp = gpu_recompute(L)
    kvd.kvd_set_fused_tokens(mode)
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T, 1) == -(-T // mt)
    q, _, out, (dk, dv) = gpu_fused(L, kv_debug=True)
    assert torch.equal(_bits(dk), _bits(Kp)) and torch.equal(_bits(dv), _bits(Vp))
    check("split fused vs oracle", out, oracle_decode(L))
    kvd.kvd_set_fused_tokens(64)
    _, _, out64, (dk64, dv64) = gpu_fused(L, q=q, kv_debug=True)
    assert torch.equal(_bits(dk64), _bits(dk)) and torch.equal(_bits(dv64), _bits(dv))
    check("split vs 64-token tiles", out, f64(out64))


@pytest.mark.parametrize("mode,mt", MODES)
@pytest.mark.parametrize("hd", [128, 256])
@pytest.mark.parametrize("T_rec,T", [(130, 133), (128, 131), (256, 257), (300, 302), (1, 4), (64, 67)])
def test_split_folded_stored_tail(mode, mt, hd, T_rec, T):
    # recompute the oldest T_rec context rows; the newer context rows and the
    # current token (T + 1 - T_rec <= 4 rows) are a stored tail folded into the
    # last chunk, also when that chunk is partial (its rows move down in LDS)
    L = _layer(hd, T, seed=190 + T_rec + hd)
    s = L.shape
    q, K, V, out_u = gpu_unfused(L)
    T_tail = T - T_rec + 1
    assert T_tail <= 4
    kvd.kvd_set_fused_tokens(mode)

    def fused(out, ws):
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)

    S = kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    assert S == -(-T_rec // mt)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    out = torch.empty_like(q)
    fused(out, ws)
    check("split folded tail vs oracle", out, oracle_decode(L))
    check("split folded tail vs unfused", out, f64(out_u))
    _counters_clear(ws, L)
    out2 = torch.empty_like(q)
    fused(out2, ws)  # the counters and completion words were left zero
    assert torch.equal(_bits(out), _bits(out2))
    fused(None, ws)  # partials only, merged by kvd_combine
    out3 = torch.empty_like(q)
    kvd.kvd_combine(s, L.B, S, ws, out3)
    assert torch.equal(_bits(out), _bits(out3))
    _counters_clear(ws, L)


@pytest.mark.parametrize("mode", [m for m, _ in MODES])
def test_split_ring_tail(mode):
    # Algorithm 1's bounded cache as a ring: the 2 newest context rows and the
    # current token in a ring of 3 slots whose oldest slot is 2, so the tail
    # view wraps; the older 298 rows are recomputed on the split engine
    T, n_tail, off = 300, 3, 2
    L = _layer(256, T, seed=197)
    s = L.shape
    q, K, V, _ = gpu_unfused(L)
    T_rec = T + 1 - n_tail
    ring_k, ring_v = empty_kv(L, n_tail)
    for i in range(n_tail):
        ring_k[:, :, (off + i) % n_tail] = K[:, :, T_rec + i]
        ring_v[:, :, (off + i) % n_tail] = V[:, :, T_rec + i]
    kvd.kvd_set_fused_tokens(mode)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, n_tail)
    kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, ring_k, ring_v, n_tail,
                                 off)
    check("split ring tail vs oracle", out, oracle_decode(L))


def test_split_shared_workspace_across_lengths():
    # one workspace sized for the longest call serves calls of every length, on
    # every engine, in any order: the completion words of one call never leak
    # into the next
    L = _layer(256, 700, seed=201)
    s = L.shape
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, L.T, 1)
    tk, tv = empty_kv(L, 1)
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, L.pos_new, q, tk, tv, 0)
    for mode, T_rec in [(SPLIT, 700), (64, 700), (kvd.KVD_FUSED_SPLIT64, 300), (128, 650), (SPLIT, 129),
                        (kvd.KVD_FUSED_SPLIT64, 700), (SPLIT, 700)]:
        kvd.kvd_set_fused_tokens(mode)
        out = torch.empty_like(q)
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, tk, tv, 1)
        kvd.kvd_set_fused_tokens(0)
        # oracle over the first T_rec rows plus the current token (projected at position T)
        qr, ktr, vtr = O.project_qkv(f64(L.h_new), f64(L.gamma), f64(L.w_q), f64(L.w_k), f64(L.w_v),
                                     f64(L.pos_new), s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps, s.rope_theta)
        pos = f64(L.pos0)[:, None] + np.arange(T_rec)[None, :]
        ref = O.kv_direct_decode(qr, f64(L.h[:, :T_rec]), f64(L.gamma), f64(L.w_k), f64(L.w_v), pos,
                                 ktr[:, :, None], vtr[:, :, None], s.n_kv_heads, s.head_dim, s.rms_eps,
                                 s.rope_theta)
        check(f"engine {mode}, T_rec {T_rec} vs oracle", out, ref)
        _counters_clear(ws, L)


def test_split_gemma_shape_ctx1000():
    # the Gemma-3-4B layer shape (d 2560, 8 query / 4 KV heads, head_dim 256): 8
    # chunks, the last one ragged, with the current token folded
    L = make_layer(C.GEMMA3_4B, B=1, T=1000, seed=203, pos0=[123])
    s = L.shape
    kvd.kvd_set_fused_tokens(SPLIT)
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 8
    q, _, out, _ = gpu_fused(L)
    check("split vs oracle", out, oracle_decode(L))
    kvd.kvd_set_fused_tokens(0)
    _, _, out64, _ = gpu_fused(L, q=q)
    check("split vs the default engine", out, f64(out64))


@pytest.mark.parametrize("mode", [m for m, _ in MODES])
@pytest.mark.parametrize("window", [130, 201, 500])
def test_split_window(mode, window):
    T = 200
    L = _layer(256, T, seed=170 + window)
    s = L.shape
    n_keep = min(T + 1, window)
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    tk, tv = empty_kv(L, 1)
    pos = torch.full((L.B,), n_keep - 1, dtype=torch.int32, device="cuda")
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, pos, q, tk, tv, 0)
    kvd.kvd_set_fused_tokens(mode)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T, 1)
    kvd.kvd_fused_window_attn(s, q, L.h, T, L.gamma, L.lw_k, L.lw_v, window, out, ws, tk, tv, 1)
    ref = O.sliding_window_decode(f64(L.h_new), f64(L.h[:, :L.T]), f64(L.gamma), f64(L.w_q), f64(L.w_k),
                                  f64(L.w_v), window, s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps,
                                  s.rope_theta)
    check(f"split window {window} vs oracle", out, ref)


def test_split64_by_policy_on_small_grids():
    # a Gemma-3-4B layer at B = 1 with 1000 keys: 4 KV heads x 16 tiles of 64 = 64
    # <= 128, so the automatic policy takes the split engine with 64-token chunks
    L = make_layer(C.GEMMA3_4B, B=1, T=1000, seed=207, pos0=[31])
    s = L.shape
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 16
    q, _, out, (dk, dv) = gpu_fused(L, kv_debug=True)
    check("auto split64 vs oracle", out, oracle_decode(L))
    Kp, Vp = gpu_recompute(L)
    assert torch.equal(_bits(dk), _bits(Kp)) and torch.equal(_bits(dv), _bits(Vp))
    kvd.kvd_set_fused_tokens(kvd.KVD_FUSED_SPLIT64)
    _, _, out_s, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(out_s))
    kvd.kvd_set_fused_tokens(64)
    _, _, out64, _ = gpu_fused(L, q=q)
    check("auto split64 vs 64-token tiles", out, f64(out64))
