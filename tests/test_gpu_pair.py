"""GPU parity of the pair fused engine (bf16, head_dim 128, two KV heads per
128-token tile on the head_dim 256 wave layout): forced with
kvd_set_fused_tokens(KVD_FUSED_PAIR) on small shapes that span several tiles
and a ragged one, and reached by the automatic policy on a shape with a full
round of pair tiles.

- The K/V it recomputes in LDS (dumped through kv_debug) are bit-identical to
  the prefill K/V of kvd_recompute_kv (Prop. reconstruction: the same MFMA
  chain over d per element, the same 1/rms and RoPE epilogue), for every
  weight layout.
- Each head's attention, split partial and merge are the wide engine's
  arithmetic on the same keys, so its output equals the wide engine's bit for
  bit, and matches the fp64 oracle's decode step (Eqs. attn_weights /
  head_output) to the bf16 tolerance.
- Stored tails (Algorithm 1's bounded cache, also as a wrapped ring), the
  partials-then-kvd_combine path and sliding-window layers go through it too.

Tolerance (max |gpu - oracle| / max |oracle|): 2e-2 for bf16 inputs."""
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import (TOL, empty_kv, err, f64, gpu_fused, gpu_recompute, gpu_unfused, make_layer, note,
                       oracle_decode)

pytestmark = pytest.mark.gpu

BF = kvd.KVD_BF16
TOL_BF = TOL[BF]
PAIR = kvd.KVD_FUSED_PAIR


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


def _layer(T, seed, B=2, n_q=12, n_kv=2, packed=True, pos0=None):
    return make_layer(C.QWEN_1_5B, B=B, T=T, seed=seed, pos0=pos0 or [3, 700][:B] + [11] * max(0, B - 2),
                      packed=packed, d_model=512, n_q=n_q, n_kv=n_kv, head_dim=128)


@pytest.mark.parametrize("packed", [False, True, "gamma"])
@pytest.mark.parametrize("T", [128, 300])
@pytest.mark.parametrize("n_q,n_kv", [(12, 2), (16, 4), (4, 2), (16, 2)])
def test_pair_kv_bitwise_and_output(packed, T, n_q, n_kv):
    # group sizes 6, 4, 2 and 8; one and two pairs; a full and a ragged last tile
    L = _layer(T, seed=300 + T + n_q + n_kv, n_q=n_q, n_kv=n_kv, packed=packed)
    s = L.shape
    Kp, Vp = gpu_recompute(L)
    kvd.kvd_set_fused_tokens(PAIR)
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T, 1) == -(-T // 128)  # the current token folds
    q, _, out, (dk, dv) = gpu_fused(L, kv_debug=True)
    assert torch.equal(_bits(dk), _bits(Kp)) and torch.equal(_bits(dv), _bits(Vp))
    check("pair fused vs oracle", out, oracle_decode(L))
    kvd.kvd_set_fused_tokens(128)
    _, _, out_w, (dkw, dvw) = gpu_fused(L, q=q, kv_debug=True)
    assert torch.equal(_bits(dkw), _bits(dk)) and torch.equal(_bits(dvw), _bits(dv))
    assert torch.equal(_bits(out_w), _bits(out)), "pair and wide engines differ"


def _tail_tiles(n_rec, T_tail):
    if n_rec > 0 and 0 < T_tail <= 4:
        return 0  # folded into the last recomputed chunk
    return T_tail // 64 if T_tail > 64 and 0 < T_tail % 64 <= 4 else -(-T_tail // 64)


@pytest.mark.parametrize("T_rec,T", [(130, 430), (128, 131), (256, 262), (300, 300), (1, 70), (128, 320),
                                     (300, 302)])
def test_pair_stored_tail(T_rec, T):
    # the oldest T_rec context rows recomputed, the rest and the current token a
    # stored tail: folded into the last chunk when it has <= 4 rows, else 64-row
    # tiles of both heads of a pair, a remainder of <= 4 rows joining the last
    L = _layer(T, seed=320 + T_rec, n_q=16, n_kv=4)
    s = L.shape
    q, K, V, out_u = gpu_unfused(L)
    T_tail = T - T_rec + 1
    kvd.kvd_set_fused_tokens(PAIR)

    def fused(out, ws):
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)

    S = kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    assert S == -(-T_rec // 128) + _tail_tiles(-(-T_rec // 128), T_tail)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    out = torch.empty_like(q)
    fused(out, ws)
    check("pair hybrid vs oracle", out, oracle_decode(L))
    check("pair hybrid vs unfused", out, f64(out_u))
    out2 = torch.empty_like(q)
    fused(out2, ws)  # the counters were left zero
    assert torch.equal(_bits(out), _bits(out2))
    fused(None, ws)  # partials only, merged by kvd_combine
    out3 = torch.empty_like(q)
    kvd.kvd_combine(s, L.B, S, ws, out3)
    assert torch.equal(_bits(out), _bits(out3))
    ctr_bytes = -(-L.B * s.n_kv_heads * 8 // 256) * 256
    assert int(torch.count_nonzero(ws[:ctr_bytes])) == 0
    kvd.kvd_set_fused_tokens(128)
    out_w = torch.empty_like(q)
    fused(out_w, ws)
    assert torch.equal(_bits(out_w), _bits(out)), "pair and wide engines differ"


def test_pair_ring_tail():
    # a bounded cache kept as a ring: the 40 newest context rows and the current
    # token in a ring of 41 slots whose oldest slot is 25 (the view wraps); the
    # older 260 rows recomputed on the pair engine
    T, n_tail, off = 300, 41, 25
    L = _layer(T, seed=97, n_q=16, n_kv=4)
    s = L.shape
    q, K, V, _ = gpu_unfused(L)
    T_rec = T + 1 - n_tail
    ring_k, ring_v = empty_kv(L, n_tail)
    for i in range(n_tail):
        ring_k[:, :, (off + i) % n_tail] = K[:, :, T_rec + i]
        ring_v[:, :, (off + i) % n_tail] = V[:, :, T_rec + i]
    kvd.kvd_set_fused_tokens(PAIR)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, n_tail)
    kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, ring_k, ring_v, n_tail,
                                 off)
    check("pair ring tail vs oracle", out, oracle_decode(L))


def test_pair_by_policy_on_a_full_round():
    # 4 sequences x 4 pairs of KV heads x 16 tiles of 128 = 256 pair tiles: the
    # automatic policy takes the pair engine; its output equals the wide engine's
    L = make_layer(C.QWEN_1_5B, B=4, T=2000, seed=99, d_model=512, n_q=16, n_kv=8, head_dim=128,
                   pos0=[0, 300, 17, 900])
    s = L.shape
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 16
    q, _, out, _ = gpu_fused(L)
    check("auto pair vs oracle (sequences 0, 3)", out[[0, 3]], oracle_decode(L, b_sel=[0, 3]))
    kvd.kvd_set_fused_tokens(PAIR)
    _, _, out_p, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(out_p))
    kvd.kvd_set_fused_tokens(128)
    _, _, out_w, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(out_w))


def test_pair_odd_kv_heads_fall_back():
    # an odd KV head count has no pairs: the forced setting runs the wide engine
    L = _layer(300, seed=41, n_q=9, n_kv=3)
    s = L.shape
    kvd.kvd_set_fused_tokens(PAIR)
    q, _, out, _ = gpu_fused(L)
    check("odd n_kv (wide engine) vs oracle", out, oracle_decode(L))
    kvd.kvd_set_fused_tokens(128)
    _, _, out_w, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(out_w))
    assert kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1) == 3


@pytest.mark.parametrize("window", [130, 201, 500])
def test_pair_window(window):
    T = 200
    L = _layer(T, seed=70 + window, n_q=16, n_kv=4)
    s = L.shape
    n_keep = min(T + 1, window)
    q = torch.empty((L.B, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    tk, tv = empty_kv(L, 1)
    pos = torch.full((L.B,), n_keep - 1, dtype=torch.int32, device="cuda")
    kvd.kvd_project_qkv(s, L.h_new, L.gamma, L.lw_q, L.lw_k, L.lw_v, pos, q, tk, tv, 0)
    kvd.kvd_set_fused_tokens(PAIR)
    out = torch.empty_like(q)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T, 1)
    kvd.kvd_fused_window_attn(s, q, L.h, T, L.gamma, L.lw_k, L.lw_v, window, out, ws, tk, tv, 1)
    ref = O.sliding_window_decode(f64(L.h_new), f64(L.h[:, :L.T]), f64(L.gamma), f64(L.w_q), f64(L.w_k),
                                  f64(L.w_v), window, s.n_q_heads, s.n_kv_heads, s.head_dim, s.rms_eps,
                                  s.rope_theta)
    check(f"pair window {window} vs oracle", out, ref)
