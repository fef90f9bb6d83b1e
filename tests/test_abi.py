"""The C-ABI library on the CPU: it loads, exports every symbol include/kvd.h
declares, and every validation error is returned as the documented status
before any HIP call (no GPU is touched: every call here fails validation)."""
import ctypes

import pytest

kvd = pytest.importorskip("paper_2603_19664_amd.kvd")
lib = kvd.lib

FAKE = 0x10000          # aligned, never dereferenced (validation fails first)
MISALIGNED = 0x10008


def shape(**kw):
    base = dict(d_model=2560, n_q_heads=8, n_kv_heads=4, head_dim=256, rms_eps=1e-6, rope_theta=1e4,
                dtype=kvd.KVD_BF16)
    base.update(kw)
    return kvd.AttnShape(**base)


def view(t_cap=16, t_off=0, k=FAKE, v=FAKE):
    return kvd.KvView(k, v, t_cap, t_off)


def test_loads_and_version():
    assert kvd.abi_version() == 8
    assert kvd.status_str(kvd.KVD_ERR_ALIGN) == "KVD_ERR_ALIGN"


def test_exports_every_header_symbol():
    names = kvd.header_symbols()
    assert {"kvd_recompute_kv", "kvd_decode_attn", "kvd_fused_recompute_attn", "kvd_cached_attn",
            "kvd_project_qkv", "kvd_workspace_bytes"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def recompute(s, h=FAKE, h_ld=16, gamma=FAKE, wk=FAKE, wv=FAKE, pos=FAKE, B=1, T=16, out=None):
    out = view() if out is None else out
    return lib.kvd_recompute_kv(ctypes.byref(s) if s is not None else None, h, h_ld, gamma, wk, wv, pos, B, T,
                                ctypes.byref(out), None)


@pytest.mark.parametrize("kw,status", [
    (dict(d_model=100), kvd.KVD_ERR_SHAPE),
    (dict(d_model=0), kvd.KVD_ERR_SHAPE),
    (dict(head_dim=96), kvd.KVD_ERR_UNSUPPORTED),
    (dict(n_q_heads=6, n_kv_heads=4), kvd.KVD_ERR_SHAPE),
    (dict(n_q_heads=34, n_kv_heads=2), kvd.KVD_ERR_UNSUPPORTED),
    (dict(n_kv_heads=0), kvd.KVD_ERR_SHAPE),
    (dict(rms_eps=-1.0), kvd.KVD_ERR_SHAPE),
    (dict(rms_eps=float("nan")), kvd.KVD_ERR_SHAPE),
    (dict(rope_theta=0.0), kvd.KVD_ERR_SHAPE),
    (dict(dtype=7), kvd.KVD_ERR_UNSUPPORTED),
])
def test_shape_validation(kw, status):
    assert recompute(shape(**kw)) == status
    assert kvd.last_error()


def test_recompute_argument_validation():
    s = shape()
    assert recompute(None) == kvd.KVD_ERR_NULL
    assert recompute(s, h=None) == kvd.KVD_ERR_NULL
    assert recompute(s, h=MISALIGNED) == kvd.KVD_ERR_ALIGN
    assert recompute(s, gamma=None) == kvd.KVD_ERR_NULL
    assert recompute(s, wv=MISALIGNED) == kvd.KVD_ERR_ALIGN
    assert recompute(s, pos=None) == kvd.KVD_ERR_NULL
    assert recompute(s, h_ld=8) == kvd.KVD_ERR_SHAPE
    assert recompute(s, B=-1) == kvd.KVD_ERR_SHAPE
    assert recompute(s, T=-3) == kvd.KVD_ERR_SHAPE
    assert recompute(s, out=view(t_cap=20, t_off=5)) == kvd.KVD_ERR_SHAPE
    assert recompute(s, out=view(k=0)) == kvd.KVD_ERR_NULL
    # empty inputs are a no-op: OK without touching the device or the pointers
    assert recompute(s, B=0) == kvd.KVD_OK
    assert recompute(s, T=0, h=None) == kvd.KVD_OK


def attn(fn, s, q=FAKE, kv=None, B=1, T=16, out=FAKE, ws=FAKE, ws_bytes=1 << 30):
    kv = view() if kv is None else kv
    return fn(ctypes.byref(s), q, ctypes.byref(kv), B, T, out, ws, ws_bytes, None)


def test_attention_validation():
    s = shape()
    for fn in (lib.kvd_decode_attn, lib.kvd_cached_attn):
        assert attn(fn, s, T=0) == kvd.KVD_ERR_SHAPE
        assert attn(fn, s, q=None) == kvd.KVD_ERR_NULL
        assert attn(fn, s, out=MISALIGNED) == kvd.KVD_ERR_ALIGN
        assert attn(fn, s, kv=view(t_cap=15)) == kvd.KVD_ERR_SHAPE
        assert attn(fn, s, ws=None) == kvd.KVD_ERR_WORKSPACE
        assert attn(fn, s, ws_bytes=16) == kvd.KVD_ERR_WORKSPACE
        assert attn(fn, s, ws=FAKE + 16) == kvd.KVD_ERR_ALIGN
    assert attn(lib.kvd_cached_attn, shape(dtype=kvd.KVD_F32)) == kvd.KVD_ERR_UNSUPPORTED


def fused(s, q=FAKE, h=FAKE, h_ld=64, T_rec=64, tail=None, T_tail=1, ws_bytes=1 << 30, dbg=None, B=1):
    tail = view() if tail is None else tail
    return lib.kvd_fused_recompute_attn(ctypes.byref(s), q, h, h_ld, FAKE, FAKE, FAKE, FAKE, B, T_rec,
                                        ctypes.byref(tail), T_tail, FAKE, FAKE, ws_bytes,
                                        ctypes.byref(dbg) if dbg is not None else None, None)


def test_fused_validation():
    s = shape()
    assert fused(s, T_rec=0, T_tail=0) == kvd.KVD_ERR_SHAPE
    assert fused(s, T_rec=-1) == kvd.KVD_ERR_SHAPE
    assert fused(s, h_ld=32) == kvd.KVD_ERR_SHAPE
    assert fused(s, h=None) == kvd.KVD_ERR_NULL
    assert fused(s, tail=view(t_cap=4, t_off=4)) == kvd.KVD_ERR_SHAPE
    assert fused(s, ws_bytes=100) == kvd.KVD_ERR_WORKSPACE
    assert fused(s, dbg=view(t_cap=10)) == kvd.KVD_ERR_SHAPE
    assert fused(s, B=70000) == kvd.KVD_ERR_SHAPE
    # one workgroup per (KV head, sequence, split) must stay below 2^31
    assert fused(s, B=65535, T_rec=1200000, h_ld=1200000) == kvd.KVD_ERR_SHAPE
    assert lib.kvd_fused_recompute_attn(ctypes.byref(s), FAKE, FAKE, 64, FAKE, FAKE, FAKE, FAKE, 1, 64, None, 1,
                                        FAKE, FAKE, 1 << 30, None, None) == kvd.KVD_ERR_NULL


def window_call(s, q=FAKE, h=FAKE, h_ld=64, T_rec=64, tail=None, T_tail=1, window=16, ws_bytes=1 << 30):
    tail = view() if tail is None else tail
    return lib.kvd_fused_window_attn(ctypes.byref(s), q, h, h_ld, FAKE, FAKE, FAKE, 1, T_rec, ctypes.byref(tail),
                                     T_tail, window, FAKE, FAKE, ws_bytes, None)


def test_window_validation():
    s = shape()
    assert window_call(s, window=0) == kvd.KVD_ERR_SHAPE
    assert window_call(s, window=-3) == kvd.KVD_ERR_SHAPE
    assert window_call(s, T_rec=0, T_tail=0) == kvd.KVD_ERR_SHAPE
    assert window_call(s, h_ld=32) == kvd.KVD_ERR_SHAPE
    assert window_call(s, h=None) == kvd.KVD_ERR_NULL
    assert window_call(s, q=None) == kvd.KVD_ERR_NULL
    assert window_call(s, tail=view(t_cap=4, t_off=4)) == kvd.KVD_ERR_SHAPE
    assert window_call(s, ws_bytes=100) == kvd.KVD_ERR_WORKSPACE
    # the kept rows set the split count: 16 kept keys need one split
    assert lib.kvd_num_splits(ctypes.byref(s), kvd.KVD_OP_FUSED, 1, 15, 1) == 1
    assert window_call(s, ws_bytes=_ws_bytes(s, 1, 1) - 1) == kvd.KVD_ERR_WORKSPACE


def test_project_validation():
    s = shape()
    f = lib.kvd_project_qkv
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, FAKE, None, None) == kvd.KVD_ERR_NULL
    assert f(ctypes.byref(s), FAKE, FAKE, None, FAKE, FAKE, FAKE, 1, FAKE, None, None) == kvd.KVD_ERR_NULL
    bad = view(t_cap=3, t_off=3)
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, ctypes.byref(bad), None) == kvd.KVD_ERR_SHAPE


def _stream_splits(pairs, T, target):
    """The bf16 stored-K/V attention's split rule as documented: about `target`
    workgroups over the call, at most one split per 16-key block."""
    nblk = -(-T // 16)
    return min(max(-(-target // pairs), 1), 32, nblk)


def test_split_policy_and_workspace():
    s = shape()
    ns = lambda sh, op, T, Tt, B=1: lib.kvd_num_splits(ctypes.byref(sh), op, B, T, Tt)  # noqa: E731
    # bf16 stored-K/V attention: contiguous key ranges, ~256 workgroups over the call
    for B, T in [(1, 4097), (1, 2049), (8, 2049), (64, 2049), (16, 5121), (1, 1), (3, 17), (256, 100)]:
        want = _stream_splits(B * 4, T, 256)
        assert ns(s, kvd.KVD_OP_DECODE_ATTN, T, 0, B) == want, (B, T)
        assert ns(s, kvd.KVD_OP_CACHED_ATTN, T, 0, B) == want, (B, T)
    assert ns(s, kvd.KVD_OP_DECODE_ATTN, 4097, 0) == 32     # 4 (b, head) pairs: 32 splits of 8-9 blocks
    assert ns(s, kvd.KVD_OP_DECODE_ATTN, 2049, 0, 8) == 8   # 32 pairs: 8 splits each
    assert ns(s, kvd.KVD_OP_DECODE_ATTN, 2049, 0, 64) == 1  # 256 pairs: one split each
    # the split count never falls as the key count grows (one workspace serves a growing context)
    for B in (1, 3, 8):
        counts = [ns(s, kvd.KVD_OP_DECODE_ATTN, T, 0, B) for T in range(1, 6000, 7)]
        assert counts == sorted(counts)
    # the workgroup target moves the split count, and 0 restores the default
    try:
        assert lib.kvd_set_attn_workgroups(1) == 256
        assert ns(s, kvd.KVD_OP_DECODE_ATTN, 4097, 0) == 1
        assert lib.kvd_set_attn_workgroups(1 << 20) == 1
        assert ns(s, kvd.KVD_OP_DECODE_ATTN, 4097, 0) == 32   # at most 32 per (sequence, head)
        assert ns(s, kvd.KVD_OP_DECODE_ATTN, 100, 0) == 7     # and at most one per 16-key block
    finally:
        lib.kvd_set_attn_workgroups(0)
    assert ns(s, kvd.KVD_OP_DECODE_ATTN, 4097, 0) == 32
    # fp32 stored-K/V attention: one split per 64-key tile
    assert ns(shape(dtype=kvd.KVD_F32), kvd.KVD_OP_DECODE_ATTN, 4097, 0) == 65
    assert ns(shape(dtype=kvd.KVD_F32), kvd.KVD_OP_DECODE_ATTN, 64, 0) == 1
    # fused: one split per 64-token recompute tile; a bf16 tail of <= 4 rows joins the
    # last recomputed tile, a longer one (or any fp32 tail) adds its own tiles
    assert ns(s, kvd.KVD_OP_FUSED, 4096, 1) == 64
    assert ns(s, kvd.KVD_OP_FUSED, 4096, 4) == 64
    assert ns(s, kvd.KVD_OP_FUSED, 4096, 5) == 65
    assert ns(s, kvd.KVD_OP_FUSED, 4000, 70) == 65
    assert ns(shape(dtype=kvd.KVD_F32), kvd.KVD_OP_FUSED, 4096, 1) == 65
    assert ns(s, kvd.KVD_OP_FUSED, 0, 1) == 1
    assert lib.kvd_num_splits(ctypes.byref(s), kvd.KVD_OP_DECODE_ATTN, 1, 0, 0) == 0
    n = lib.kvd_workspace_bytes(ctypes.byref(s), kvd.KVD_OP_DECODE_ATTN, 2, 100, 0)
    S = _stream_splits(8, 100, 256)
    assert S == 7
    acc = -(-2 * 8 * S * 256 * 4 // 256) * 256
    ml = -(-2 * 8 * S * 2 * 4 // 256) * 256
    done = -(-2 * 4 * 8 // 256) * 256 + -(-2 * 4 * 4 * 8 // 256) * 256  # split counters, completion words
    assert n == acc + ml + done
    assert lib.kvd_workspace_bytes(ctypes.byref(s), 9, 1, 10, 0) == 0


def _engine(s, B, T_rec, T_tail, tokens):
    """The fused call's engine as documented: 128-token wide tiles (bf16, head_dim 128 /
    256) when forced or when there are at least 256 of them; the split engine (bf16,
    head_dim 128 / 256, T_rec >= 1, T_tail <= 4, <= 256 chunks) with 64-token chunks when
    64-token tiles would number at most 128, or when forced (either chunk size); else
    64-token tiles."""
    big = s.dtype == kvd.KVD_BF16 and s.head_dim in (128, 256)
    wide_ok = big and T_rec > 0

    def split_ok(mt):
        return big and T_rec > 0 and T_tail <= 4 and -(-T_rec // mt) <= 256
    if tokens == 64:
        return "tile64"
    if tokens in (128, kvd.KVD_FUSED_PAIR):  # the pair engine chunks and splits as the wide one
        return "wide" if wide_ok else "tile64"
    if tokens == kvd.KVD_FUSED_SPLIT:
        return "split" if split_ok(128) else "tile64"
    if tokens == kvd.KVD_FUSED_SPLIT64:
        return "split64" if split_ok(64) else "tile64"
    if wide_ok and B * s.n_kv_heads * -(-T_rec // 128) >= 256:
        return "wide"
    if split_ok(64) and B * s.n_kv_heads * -(-T_rec // 64) <= 128:
        return "split64"
    return "tile64"


def _tail_tiles(s, n_rec, T_tail):
    """Stored-tail tiles: none when a bf16 tail of <= 4 rows folds into the last recomputed
    tile; else one per 64 rows, a bf16 remainder of <= 4 rows joining the tile before it."""
    bf = s.dtype == kvd.KVD_BF16
    if bf and n_rec > 0 and 0 < T_tail <= 4:
        return 0
    r = T_tail % 64
    if bf and T_tail > 64 and 0 < r <= 4:
        return T_tail // 64
    return -(-T_tail // 64)


def _fused_splits(s, B, T_rec, T_tail, tokens, engine=None):
    """The fused call's split count: one per recomputed tile plus the stored tail's tiles."""
    engine = engine or _engine(s, B, T_rec, T_tail, tokens)
    if engine == "wide":
        n_rec = -(-T_rec // 128)
        return n_rec + _tail_tiles(s, n_rec, T_tail)
    if engine == "split":
        return -(-T_rec // 128)
    if engine == "split64":
        return -(-T_rec // 64)
    n_rec = -(-T_rec // 64)
    return n_rec + _tail_tiles(s, n_rec, T_tail)


def _ws_bytes(s, B, S, split_chunks=0, mt=128):
    up = lambda x: -(-x // 256) * 256  # noqa: E731
    g = s.n_q_heads // s.n_kv_heads
    xf = -(-(g * (mt + 4) + 2 * g) // 4) * 4
    return (up(B * s.n_kv_heads * 8) + up(B * s.n_kv_heads * 4 * 8) + up(B * s.n_q_heads * S * s.head_dim * 4)
            + up(B * s.n_q_heads * S * 2 * 4) + (up(B * s.n_kv_heads * split_chunks * xf * 4) if split_chunks else 0))


def _fused_ws_bytes(s, B, T, Tt):
    """kvd_workspace_bytes of KVD_OP_FUSED: the largest need over the engines a call can get."""
    n = _ws_bytes(s, B, _fused_splits(s, B, T, Tt, 0, "tile64"))
    big = s.dtype == kvd.KVD_BF16 and s.head_dim in (128, 256) and T > 0
    if big:
        n = max(n, _ws_bytes(s, B, _fused_splits(s, B, T, Tt, 0, "wide")))
    if big and Tt <= 4 and -(-T // 128) <= 256:
        n = max(n, _ws_bytes(s, B, -(-T // 128), -(-T // 128)))
    if big and Tt <= 4 and -(-T // 64) <= 256:
        n = max(n, _ws_bytes(s, B, -(-T // 64), -(-T // 64), mt=64))
    return n


def test_fused_tiling_policy():
    ns = lambda sh, B, T, Tt: lib.kvd_num_splits(ctypes.byref(sh), kvd.KVD_OP_FUSED, B, T, Tt)  # noqa: E731
    gemma, qwen = shape(), shape(d_model=1536, n_q_heads=12, n_kv_heads=2, head_dim=128)
    others = [shape(dtype=kvd.KVD_F32), shape(head_dim=64, d_model=576, n_q_heads=9, n_kv_heads=3)]
    # default: wide tiles with a full round of them, else 64-token tiles (the split
    # engine only when forced)
    assert ns(gemma, 1, 4096, 1) == 64        # 128 wide tiles: 64-token tiles, folded current token
    assert ns(gemma, 2, 4096, 1) == 32        # 256 wide tiles, folded current token
    assert ns(gemma, 8, 2048, 1) == 16
    assert ns(gemma, 1, 3072, 1025) == 48 + 16  # a stored window of 1024 + the current token: 16 tail tiles
    assert ns(gemma, 1, 4096, 5) == 65        # a 5-row tail cannot fold: 64-token tiles + a tail tile
    assert ns(gemma, 1, 2048, 1) == 32        # 128 64-token tiles: split engine, 64-token chunks
    assert ns(gemma, 1, 1023, 1) == 16        # a sliding window at B = 1
    assert ns(qwen, 8, 16384, 1) == 128
    try:
        modes = (0, 64, 128, kvd.KVD_FUSED_SPLIT, kvd.KVD_FUSED_PAIR, kvd.KVD_FUSED_SPLIT64)
        for tokens in modes:
            assert lib.kvd_set_fused_tokens(tokens) in modes
            for sh in [gemma, qwen] + others:
                for B, T, Tt in [(1, 4096, 1), (2, 4096, 1), (8, 2048, 1), (1, 100, 1), (1, 0, 3), (3, 130, 70),
                                 (16, 5120, 0), (1, 64, 4), (1, 64, 5), (1, 32769, 1)]:
                    S = ns(sh, B, T, Tt)
                    assert S == _fused_splits(sh, B, T, Tt, tokens), (tokens, sh.head_dim, B, T, Tt)
                    # the workspace covers every engine
                    n = lib.kvd_workspace_bytes(ctypes.byref(sh), kvd.KVD_OP_FUSED, B, T, Tt)
                    assert n >= _ws_bytes(sh, B, S)
                    assert n == _fused_ws_bytes(sh, B, T, Tt), (tokens, sh.head_dim, B, T, Tt)
        # the workspace size never falls as the context grows, whichever tiling a call gets
        for B in (1, 2, 8):
            sizes = [lib.kvd_workspace_bytes(ctypes.byref(gemma), kvd.KVD_OP_FUSED, B, T, 1) for T in range(1, 5000, 13)]
            assert sizes == sorted(sizes)
        assert lib.kvd_set_fused_tokens(128) == kvd.KVD_FUSED_SPLIT64  # the loop's last setting
        assert lib.kvd_set_fused_tokens(77) == 128  # other values mean 0
        assert lib.kvd_set_fused_tokens(0) == 0
    finally:
        lib.kvd_set_fused_tokens(0)


def test_lds_limit_is_validated():
    # fp32, head_dim 256 and 16 query heads per KV head exceed one workgroup's LDS
    s = shape(dtype=kvd.KVD_F32, n_q_heads=64, n_kv_heads=4, d_model=512)
    assert fused(s) == kvd.KVD_ERR_UNSUPPORTED
    assert attn(lib.kvd_decode_attn, s) == kvd.KVD_ERR_UNSUPPORTED


def test_combine_validation():
    s = shape()
    f = lib.kvd_combine
    assert f(ctypes.byref(s), 1, 0, FAKE, 1 << 30, FAKE, None) == kvd.KVD_ERR_SHAPE
    assert f(ctypes.byref(s), 1, 4, FAKE, 1 << 30, None, None) == kvd.KVD_ERR_NULL
    assert f(ctypes.byref(s), 1, 4, FAKE, 64, FAKE, None) == kvd.KVD_ERR_WORKSPACE
    assert f(ctypes.byref(s), 1, 4, FAKE + 64, 1 << 30, FAKE, None) == kvd.KVD_ERR_ALIGN


def test_lds_limit_of_projection_is_validated():
    # the current-token projection holds gamma, its weight ring and at least one
    # residual row in LDS (fewer tokens per workgroup as d_model grows)
    f = lib.kvd_project_qkv
    s = shape(d_model=40960)
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, FAKE, None, None) == kvd.KVD_ERR_UNSUPPORTED
    assert "LDS" in kvd.last_error()
    s = shape(d_model=8192)  # fits: validation goes on to the NULL q_out (nothing is launched)
    assert f(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, None, None, None) == kvd.KVD_ERR_NULL


def test_weight_layout_validation():
    assert recompute(shape(w_layout=5)) == kvd.KVD_ERR_UNSUPPORTED
    assert recompute(shape(w_layout=kvd.KVD_W_PACKED, dtype=kvd.KVD_F32)) == kvd.KVD_ERR_UNSUPPORTED
    f = lib.kvd_pack_weights
    s = shape()
    assert f(ctypes.byref(s), FAKE, 48, FAKE + (1 << 24), None) == kvd.KVD_ERR_SHAPE       # rows % 32
    assert f(ctypes.byref(s), FAKE, 64, FAKE + 4096, None) == kvd.KVD_ERR_SHAPE            # overlap
    assert f(ctypes.byref(s), None, 64, FAKE, None) == kvd.KVD_ERR_NULL
    assert f(ctypes.byref(shape(dtype=kvd.KVD_F32)), FAKE, 64, FAKE + (1 << 24), None) == kvd.KVD_ERR_UNSUPPORTED


def block_call(s, h_in=FAKE, h_out=FAKE + (1 << 24), pos=FAKE, B=1, T=64, d_ff=1024, ws_bytes=1 << 30, nullw=None):
    ptrs = [FAKE] * 9
    if nullw is not None:
        ptrs[nullw] = None
    w = kvd.BlockWeights(*ptrs, d_ff)
    return lib.kvd_block_forward(ctypes.byref(s), ctypes.byref(w), h_in, h_out, pos, B, T, FAKE, ws_bytes, None)


def test_block_forward_validation():
    s = shape(d_model=1024, n_q_heads=8, n_kv_heads=4, head_dim=128)
    assert block_call(shape(d_model=1024, n_q_heads=8, n_kv_heads=4, head_dim=128, dtype=kvd.KVD_F32)) == \
        kvd.KVD_ERR_UNSUPPORTED
    assert block_call(shape(d_model=1024, n_q_heads=8, n_kv_heads=4, head_dim=64)) == kvd.KVD_ERR_UNSUPPORTED
    assert block_call(shape(d_model=768, n_q_heads=8, n_kv_heads=4, head_dim=128)) == kvd.KVD_ERR_UNSUPPORTED
    assert block_call(s, d_ff=100) == kvd.KVD_ERR_SHAPE
    assert block_call(s, T=-1) == kvd.KVD_ERR_SHAPE
    assert block_call(s, h_in=None) == kvd.KVD_ERR_NULL
    assert block_call(s, pos=None) == kvd.KVD_ERR_NULL
    for i in range(9):
        assert block_call(s, nullw=i) == kvd.KVD_ERR_NULL
    assert block_call(s, h_out=FAKE) == kvd.KVD_ERR_SHAPE          # aliasing
    assert block_call(s, ws_bytes=100) == kvd.KVD_ERR_WORKSPACE
    assert lib.kvd_block_forward(ctypes.byref(s), None, FAKE, FAKE, FAKE, 1, 1, FAKE, 1 << 30, None) == kvd.KVD_ERR_NULL
    n = lib.kvd_block_workspace_bytes(ctypes.byref(s), 1024, 2, 100)
    qd, kvd_ = 8 * 128, 4 * 128
    parts = [2 * 200 * qd, 2 * 200 * kvd_, 2 * 200 * kvd_, 2 * 200 * qd, 2 * 200 * 1024, 2 * 200 * 1024, 2 * 1024]
    assert n == sum(-(-p // 256) * 256 for p in parts)
    assert lib.kvd_block_workspace_bytes(ctypes.byref(s), 100, 2, 100) == 0


def _prefill_split(B, T, n_q, target=256):
    # the causal attention's key-range split (host policy): parts of at most P key blocks
    nqb = -(-T // 128)
    nkb = [min(128 * qb + 127, T - 1) // 64 + 1 for qb in range(nqb)]
    P = min(max(8, -(-sum(nkb) * B * n_q // target)), nkb[-1])
    return P, -(-nkb[-1] // P), nqb


@pytest.mark.parametrize("B,T", [(1, 4096), (1, 1100), (2, 777), (8, 4096), (1, 100)])
def test_block_workspace_holds_the_attention_split(B, T):
    s = shape(d_model=1024, n_q_heads=8, n_kv_heads=4, head_dim=128)
    qd, kvd_, dff = 8 * 128, 4 * 128, 1024
    bt = B * T
    parts = [2 * bt * qd, 2 * bt * kvd_, 2 * bt * kvd_, 2 * bt * qd, 2 * bt * 1024, 2 * bt * dff, 2 * 1024]
    P, NP, nqb = _prefill_split(B, T, 8)
    if NP > 1:  # partial states (4 waves x (32 x 128 O + 128 max/sum) floats) and one counter per query block
        parts += [4 * B * 8 * nqb * NP * 4 * (4 * 16 * 64 + 128), 8 * B * 8 * nqb]
    assert lib.kvd_block_workspace_bytes(ctypes.byref(s), dff, B, T) == sum(-(-p // 256) * 256 for p in parts)
    if (B, T) == (1, 4096):
        assert (P, NP) == (33, 2)
    if (B, T) == (8, 4096):
        assert NP == 1  # enough blocks to fill the chip: nothing split


def test_pack_matrix_validation():
    f = lib.kvd_pack_matrix
    assert f(FAKE, 33, 64, FAKE + (1 << 24), None) == kvd.KVD_ERR_SHAPE
    assert f(FAKE, 64, 24, FAKE + (1 << 24), None) == kvd.KVD_ERR_SHAPE
    assert f(None, 64, 64, FAKE, None) == kvd.KVD_ERR_NULL
    assert f(FAKE, 64, 64, FAKE + 64, None) == kvd.KVD_ERR_SHAPE     # overlap


# ------------------------------------------------------------------ binding extent checks (no GPU)

def _layer_tensors(B=2, T=8, d=512, nq=8, nkv=4, hd=64, dt=None):
    import torch
    dt = dt or torch.bfloat16
    return dict(h=torch.zeros(B, T, d, dtype=dt), gamma=torch.zeros(d, dtype=dt),
                w_q=torch.zeros(nq * hd, d, dtype=dt), w_k=torch.zeros(nkv * hd, d, dtype=dt),
                w_v=torch.zeros(nkv * hd, d, dtype=dt), pos=torch.zeros(B, dtype=torch.int32),
                q=torch.zeros(B, nq, hd, dtype=dt), k=torch.zeros(B, nkv, T + 1, hd, dtype=dt),
                v=torch.zeros(B, nkv, T + 1, hd, dtype=dt), h_new=torch.zeros(B, d, dtype=dt))


SH = kvd.Shape(512, 8, 4, 64, 1e-6, 1e4, kvd.KVD_BF16)


def _raises(match, fn, *a, **kw):
    with pytest.raises(ValueError, match=match):
        fn(*a, **kw)


def test_binding_rejects_mismatched_extents_before_any_launch():
    import torch
    x = _layer_tensors()
    bad_k = torch.zeros(2, 3, 9, 64, dtype=torch.bfloat16)   # 3 KV heads, the shape says 4
    # recompute_kv
    _raises("h has shape", kvd.kvd_recompute_kv, SH, torch.zeros(2, 8, 256, dtype=torch.bfloat16), x["gamma"],
            x["w_k"], x["w_v"], x["pos"], 8, x["k"], x["v"])
    _raises("gamma has shape", kvd.kvd_recompute_kv, SH, x["h"], torch.zeros(256, dtype=torch.bfloat16), x["w_k"],
            x["w_v"], x["pos"], 8, x["k"], x["v"])
    _raises("w_k has shape", kvd.kvd_recompute_kv, SH, x["h"], x["gamma"], x["w_q"], x["w_v"], x["pos"], 8, x["k"],
            x["v"])
    _raises("pos0 has shape", kvd.kvd_recompute_kv, SH, x["h"], x["gamma"], x["w_k"], x["w_v"],
            torch.zeros(3, dtype=torch.int32), 8, x["k"], x["v"])
    _raises("out_k has shape", kvd.kvd_recompute_kv, SH, x["h"], x["gamma"], x["w_k"], x["w_v"], x["pos"], 8, bad_k,
            bad_k)
    _raises("exceed t_cap", kvd.kvd_recompute_kv, SH, x["h"], x["gamma"], x["w_k"], x["w_v"], x["pos"], 8, x["k"],
            x["v"], 2)
    # project
    _raises("q_out has shape", kvd.kvd_project_qkv, SH, x["h_new"], x["gamma"], x["w_q"], x["w_k"], x["w_v"], x["pos"],
            torch.zeros(2, 4, 64, dtype=torch.bfloat16))
    _raises("w_q has shape", kvd.kvd_project_q, SH, x["h_new"], x["gamma"], x["w_k"], x["pos"], x["q"])
    # attention
    _raises("out has shape", kvd.kvd_decode_attn, SH, x["q"], x["k"], x["v"], 9, torch.zeros(1, 8, 64), x["q"])
    _raises("kv_k has shape", kvd.kvd_cached_attn, SH, x["q"], bad_k, bad_k, 9, x["q"], x["q"])
    _raises("exceed t_cap", kvd.kvd_decode_attn, SH, x["q"], x["k"], x["v"], 10, x["q"], x["q"])
    _raises("out has shape", kvd.kvd_combine, SH, 2, 3, x["q"], torch.zeros(2, 8, 32))
    # fused
    _raises("h has shape", kvd.kvd_fused_recompute_attn, SH, x["q"], torch.zeros(3, 8, 512, dtype=torch.bfloat16), 8,
            x["gamma"], x["w_k"], x["w_v"], x["pos"], x["q"], x["q"])
    _raises("tail_k has shape", kvd.kvd_fused_recompute_attn, SH, x["q"], x["h"], 8, x["gamma"], x["w_k"], x["w_v"],
            x["pos"], x["q"], x["q"], bad_k, bad_k, 1)
    _raises("tail_k / tail_v are required", kvd.kvd_fused_recompute_attn, SH, x["q"], x["h"], 8, x["gamma"], x["w_k"],
            x["w_v"], x["pos"], x["q"], x["q"], None, None, 1)
    _raises("kv_debug_k has shape", kvd.kvd_fused_recompute_attn, SH, x["q"], x["h"], 8, x["gamma"], x["w_k"],
            x["w_v"], x["pos"], x["q"], x["q"], x["k"], x["v"], 1, 0, bad_k, bad_k)
    _raises("h has shape", kvd.kvd_fused_window_attn, SH, x["q"], torch.zeros(2, 8, 64, dtype=torch.bfloat16), 8,
            x["gamma"], x["w_k"], x["w_v"], 4, x["q"], x["q"])
    # block forward weights against the shape
    d_ff = 256
    z = lambda *s: torch.zeros(*s, dtype=torch.bfloat16)  # noqa: E731
    _raises("w_o has shape", kvd.block_weights, x["gamma"], x["w_q"], x["w_k"], x["w_v"], z(512, 256), x["gamma"],
            z(d_ff, 512), z(d_ff, 512), z(512, d_ff), shape=SH)
    _raises("h_out has shape", kvd.kvd_block_forward, SH, None, x["h"], z(2, 7, 512), x["pos"], x["q"])
    with pytest.raises(ValueError, match="d_model=512"):
        kvd.kvd_pack_weights(SH, z(64, 256))


def test_binding_rejects_host_tensors_of_the_right_extents():
    # extents pass; the device check then refuses host memory (still before any launch)
    x = _layer_tensors()
    _raises("on the GPU", kvd.kvd_recompute_kv, SH, x["h"], x["gamma"], x["w_k"], x["w_v"], x["pos"], 8, x["k"],
            x["v"])
    _raises("on the GPU", kvd.kvd_decode_attn, SH, x["q"], x["k"], x["v"], 9, x["q"], x["q"])


def test_noalloc_rejects_work_beyond_its_scratch():
    # 64 sequences of 16384 recomputed keys need ~134 MB of split-K partials, more
    # than the 32 MiB static scratch: refused before any HIP call
    s = shape()
    need = lib.kvd_workspace_bytes(ctypes.byref(s), kvd.KVD_OP_FUSED, 64, 16384, 1)
    assert need > 32 << 20
    tail = view(t_cap=1)
    st = lib.kvd_fused_recompute_attn_noalloc(ctypes.byref(s), FAKE, FAKE, 16384, FAKE, FAKE, FAKE, FAKE, 64, 16384,
                                              ctypes.byref(tail), 1, FAKE, None)
    assert st == kvd.KVD_ERR_WORKSPACE and "static scratch" in kvd.last_error()
    # the partial-only form has no place in it: out is required
    st = lib.kvd_fused_recompute_attn_noalloc(ctypes.byref(s), FAKE, FAKE, 100, FAKE, FAKE, FAKE, FAKE, 1, 100,
                                              ctypes.byref(tail), 1, None, None)
    assert st == kvd.KVD_ERR_NULL
