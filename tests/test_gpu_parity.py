"""GPU parity: the HIP library (through its C ABI) against the fp64 oracle, on
seeded inputs shaped like the paper's models, plus the bit-identity properties
of the reconstruction identity (Prop. reconstruction) on the GPU.

Tolerances (max |gpu - oracle| / max |oracle| per tensor): 1e-5 for fp32
inputs, 2e-2 for bf16 inputs."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import (TOL, err, f64, gpu_fused, gpu_project, gpu_recompute, gpu_unfused, make_layer, note,
                       oracle_decode, oracle_kv, oracle_qkv)

pytestmark = pytest.mark.gpu

BF, F32 = kvd.KVD_BF16, kvd.KVD_F32


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()


def check(name, x, ref, tol):
    e = err(f64(x) if isinstance(x, torch.Tensor) else x, ref)
    note(f"    {name}: err {e:.3e} (tol {tol:g})")
    assert e < tol, f"{name}: err {e:.3e} >= {tol:g}"


# ------------------------------------------------------------------ SmolLM2-135M layer, fp32 (C1)

def test_smollm_fp32_full_step():
    L = make_layer(C.SMOLLM_FP32, B=1, T=256)
    K, V = gpu_recompute(L)
    Kr, Vr = oracle_kv(L)
    check("K", K, Kr, 1e-5)
    check("V", V, Vr, 1e-5)
    qr, ktr, vtr = oracle_qkv(L)
    q, K1, V1, out = gpu_unfused(L)
    check("q", q, qr, 1e-5)
    check("K_t", K1[:, :, 256], ktr, 1e-5)
    check("V_t", V1[:, :, 256], vtr, 1e-5)
    ref = oracle_decode(L)
    check("out (recompute_kv + decode_attn)", out, ref, 1e-5)
    _, _, outf, _ = gpu_fused(L)
    check("out (fused)", outf, ref, 1e-5)


# ------------------------------------------------------------------ Gemma 3-4B layer, bf16 (C2 layer)

def test_gemma_layer_bf16_full():
    L = make_layer(C.GEMMA3_4B, B=1, T=4096, layer=3)
    K, V = gpu_recompute(L)
    Kr, Vr = oracle_kv(L)
    check("K", K, Kr, 2e-2)
    check("V", V, Vr, 2e-2)
    ref = oracle_decode(L)
    q, _, _, out = gpu_unfused(L)
    check("q", q, oracle_qkv(L)[0], 2e-2)
    check("out (unfused)", out, ref, 2e-2)
    _, _, outf, _ = gpu_fused(L)
    check("out (fused)", outf, ref, 2e-2)


# ------------------------------------------------------------------ shapes, tails and groups

SHAPES = [  # (d, n_q, n_kv, hd)
    (256, 4, 2, 64),
    (512, 6, 2, 128),
    (512, 12, 2, 128),
    (512, 6, 2, 256),
    (576, 9, 3, 64),
]


@pytest.mark.parametrize("dtype", [BF, F32])
@pytest.mark.parametrize("shp", SHAPES)
@pytest.mark.parametrize("T", [1, 31, 64, 65, 200])
def test_tails_groups_dtypes(dtype, shp, T):
    d, nq, nkv, hd = shp
    L = make_layer(C.SMOLLM_FP32, B=2, T=T, seed=T, d_model=d, n_q=nq, n_kv=nkv, head_dim=hd,
                   dtype="bf16" if dtype == BF else "f32", pos0=[0, 37])
    tol = TOL[dtype]
    K, V = gpu_recompute(L)
    Kr, Vr = oracle_kv(L)
    check("K", K, Kr, tol)
    check("V", V, Vr, tol)
    ref = oracle_decode(L)
    _, _, _, out = gpu_unfused(L)
    check("out unfused", out, ref, tol)
    _, _, outf, _ = gpu_fused(L)
    check("out fused", outf, ref, tol)


@pytest.mark.parametrize("T", [16, 32, 33, 127, 128, 255, 256, 257])
def test_sequence_lengths_bf16(T):
    # the sequence lengths the paper checks reconstruction at, plus tile edges
    L = make_layer(C.GEMMA3_4B, B=1, T=T, seed=100 + T, d_model=512)
    K, V = gpu_recompute(L)
    Kr, Vr = oracle_kv(L)
    check("K", K, Kr, 2e-2)
    check("V", V, Vr, 2e-2)
    _, _, outf, _ = gpu_fused(L)
    check("out fused", outf, oracle_decode(L), 2e-2)


def test_sharpened_scores_fp32():
    # W_q std 0.2 makes scores ~10x larger (a peaked softmax), so a wrong RoPE
    # position or head mapping cannot hide behind near-uniform weights.
    L = make_layer(C.SMOLLM_FP32, B=2, T=300, seed=7, w_q_std=0.2, d_model=512, n_q=8, n_kv=4, head_dim=256,
                   pos0=[5, 1000])
    ref = oracle_decode(L)
    _, _, outf, _ = gpu_fused(L)
    check("out fused (sharp)", outf, ref, 1e-5)
    _, _, _, out = gpu_unfused(L)
    check("out unfused (sharp)", out, ref, 1e-5)


def test_stagewise_attention_bf16():
    # oracle attention evaluated on the GPU's own bf16 q/K/V isolates the attention kernels
    L = make_layer(C.GEMMA3_4B, B=2, T=1000, seed=3, w_q_std=0.2, d_model=512)
    q, K, V, out = gpu_unfused(L)
    ref = O.decode_attention(f64(q), f64(K), f64(V))
    check("decode_attn vs oracle on gpu K/V", out, ref, 5e-3)
    _, _, outf, _ = gpu_fused(L, q=q)
    check("fused vs oracle on gpu K/V", outf, ref, 5e-3)


def test_random_position_offsets_qwen_shape():
    # Qwen-1.5B layer shape, theta 1e6, positions offset per sequence (C4 recipe)
    L = make_layer(C.QWEN_1_5B, B=4, T=700, seed=11)
    assert int(L.pos0.max()) > 0
    Kr, Vr = oracle_kv(L)
    K, V = gpu_recompute(L)
    check("K", K, Kr, 2e-2)
    check("V", V, Vr, 2e-2)
    _, _, outf, _ = gpu_fused(L)
    check("out fused", outf, oracle_decode(L), 2e-2)


# ------------------------------------------------------------------ edge cases

def test_tail_only_and_no_tail():
    L = make_layer(C.GEMMA3_4B, B=2, T=0, seed=5, d_model=512)
    _, _, outf, _ = gpu_fused(L)
    ref = oracle_decode(L)  # attention over the current token alone: its V
    check("T_rec=0 (tail only)", outf, ref, 2e-2)
    L2 = make_layer(C.GEMMA3_4B, B=2, T=130, seed=6, d_model=512)
    _, _, outn, _ = gpu_fused(L2, with_current=False)
    check("T_tail=0", outn, oracle_decode(L2, with_current=False), 2e-2)


def test_zero_residuals_give_zero_kv():
    L = make_layer(C.GEMMA3_4B, B=1, T=70, seed=8, d_model=512)
    L.h.zero_()
    K, V = gpu_recompute(L)
    assert torch.count_nonzero(K) == 0 and torch.count_nonzero(V) == 0
    _, _, outf, _ = gpu_fused(L)
    assert torch.isfinite(outf.float()).all()
    check("out fused, h = 0", outf, oracle_decode(L), 2e-2)


def test_layer_scale_homogeneity():
    # RMSNorm is degree-0 homogeneous (Sec. 3.1): with eps = 0, scaling a layer's
    # residuals by a power of two is exact in every step, so K and V are unchanged bitwise.
    L = make_layer(C.GEMMA3_4B, B=1, T=96, seed=9, d_model=512, rms_eps=0.0)
    K, V = gpu_recompute(L)
    L.h.mul_(4.0)  # exact in bf16 (power of two)
    K4, V4 = gpu_recompute(L)
    assert torch.equal(K, K4) and torch.equal(V, V4)


# ------------------------------------------------------------------ bit-identity (Prop. reconstruction)

def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


@pytest.mark.parametrize("dtype", [BF, F32])
def test_prefill_equals_recompute_bitwise(dtype):
    wl = dataclasses.replace(C.GEMMA3_4B, d_model=512, dtype="bf16" if dtype == BF else "f32")
    L = make_layer(wl, B=3, T=300, seed=21, pos0=[0, 17, 4000])
    Kp, Vp = gpu_recompute(L)                     # prefill: every token at once
    # recompute of sub-ranges with odd lengths, at other offsets and capacities (in bf16,
    # calls of at most 1024 streaming workgroups at head_dim 256, here 64 per 16 rows, run
    # on the streaming kernel: (0, 1), (1, 66), (66, 67), (299, 300), (100, 120); the
    # others and the prefill on the tile engine)
    for a, b in [(0, 1), (1, 66), (66, 67), (67, 299), (299, 300), (5, 250), (100, 120)]:
        Lr = dataclasses.replace(L, h=L.h[:, a:b].contiguous(), T=b - a, pos0=(L.pos0 + a).to(torch.int32))
        K, V = gpu_recompute(Lr, t_cap=b - a + 9, t_off=7)
        assert torch.equal(_bits(K[:, :, 7:7 + b - a]), _bits(Kp[:, :, a:b])), (a, b)
        assert torch.equal(_bits(V[:, :, 7:7 + b - a]), _bits(Vp[:, :, a:b])), (a, b)
    # a short recompute reading its rows out of a longer checkpoint buffer (h_ld > T)
    K, V = gpu_recompute(dataclasses.replace(L, T=20))
    assert torch.equal(_bits(K), _bits(Kp[:, :, :20])) and torch.equal(_bits(V), _bits(Vp[:, :, :20]))
    # one sequence alone vs inside the batch
    Lb = dataclasses.replace(L, B=1, h=L.h[2:3].contiguous(), pos0=L.pos0[2:3].contiguous())
    K, V = gpu_recompute(Lb)
    assert torch.equal(_bits(K[0]), _bits(Kp[2])) and torch.equal(_bits(V[0]), _bits(Vp[2]))
    # run to run
    K2, V2 = gpu_recompute(L)
    assert torch.equal(_bits(K2), _bits(Kp)) and torch.equal(_bits(V2), _bits(Vp))


def test_long_recompute_on_the_streaming_kernel_bitwise():
    # Qwen2.5-1.5B layer shape (2 KV heads of 128: 16 streaming workgroups per 16 rows):
    # a 500-token recompute runs on the streaming kernel (512 workgroups), the 2 x 600
    # prefill on the tile engine; the K/V agree bit for bit
    L = make_layer(C.QWEN_1_5B, B=2, T=600, seed=33)
    Kp, Vp = gpu_recompute(L)
    Lr = dataclasses.replace(L, B=1, h=L.h[1:2, 50:550].contiguous(), T=500,
                             pos0=(L.pos0[1:2] + 50).to(torch.int32))
    K, V = gpu_recompute(Lr, t_cap=503, t_off=3)
    assert torch.equal(_bits(K[0, :, 3:]), _bits(Kp[1, :, 50:550]))
    assert torch.equal(_bits(V[0, :, 3:]), _bits(Vp[1, :, 50:550]))
    Kr, Vr = oracle_kv(Lr)
    check("K (streaming, 500 rows) vs oracle", K[:, :, 3:], Kr, 2e-2)


@pytest.mark.parametrize("dtype", [BF, F32])
def test_fused_and_decode_time_kv_bitwise(dtype):
    wl = dataclasses.replace(C.GEMMA3_4B, d_model=512, dtype="bf16" if dtype == BF else "f32")
    L = make_layer(wl, B=2, T=200, seed=22, pos0=[3, 90])
    Kp, Vp = gpu_recompute(L)
    # the fused kernel's LDS K/V (dumped through kv_debug) are the prefill K/V
    _, (tk, tv), _, (dk, dv) = gpu_fused(L, kv_debug=True)
    assert torch.equal(_bits(dk), _bits(Kp)) and torch.equal(_bits(dv), _bits(Vp))
    # the current token's K_t/V_t from project_qkv equal a later recompute of its residual
    Lnew = dataclasses.replace(L, h=L.h_new[:, None].contiguous(), T=1, pos0=L.pos_new)
    K1, V1 = gpu_recompute(Lnew)
    assert torch.equal(_bits(K1), _bits(tk)) and torch.equal(_bits(V1), _bits(tv))


def test_fused_equals_unfused_bitwise_on_shared_chunking():
    # fp32: recomputing rows 0..191 and reading rows 192..256 (the last context
    # tile plus the current token) as a stored tail gives the fused kernel the
    # same 64-key chunks as decode_attn over all 257 keys: identical arithmetic,
    # so the outputs agree bit for bit.  (The bf16 stored-K/V attention streams
    # whole key ranges per workgroup instead of 64-key tiles; there the two
    # paths agree to the bf16 tolerance, checked below and in every end-to-end
    # test.)
    L = make_layer(C.SMOLLM_FP32, B=2, T=256, seed=23, d_model=512, n_q=8, n_kv=4, head_dim=64, pos0=[3, 250])
    q, K, V, out = gpu_unfused(L)
    assert kvd.kvd_num_splits(L.shape, kvd.KVD_OP_DECODE_ATTN, L.B, 257) == 5
    ws = kvd.workspace(L.shape, kvd.KVD_OP_FUSED, L.B, 192, 65)
    assert kvd.kvd_num_splits(L.shape, kvd.KVD_OP_FUSED, L.B, 192, 65) == 5
    outf = torch.empty_like(out)
    kvd.kvd_fused_recompute_attn(L.shape, q, L.h, 192, L.gamma, L.lw_k, L.lw_v, L.pos0, outf, ws, K, V, 65, 192)
    assert torch.equal(_bits(out), _bits(outf))
    # budget 0: the current token is the fifth split on both paths
    _, _, outc, _ = gpu_fused(L, q=q)
    assert torch.equal(_bits(out), _bits(outc))
    check("fp32 fused vs oracle", outc, oracle_decode(L), 1e-5)
    # bf16: fused (64-key recompute tiles) and unfused (streamed stored keys) to tolerance
    Lb = make_layer(C.GEMMA3_4B, B=2, T=256, seed=23, d_model=512)
    qb, _, _, outb = gpu_unfused(Lb)
    _, _, outbf, _ = gpu_fused(Lb, q=qb)
    check("bf16 fused vs unfused", outbf, f64(outb), 2e-2)
    check("bf16 fused vs oracle", outbf, oracle_decode(Lb), 2e-2)


def test_cached_attn_matches_decode_attn():
    L = make_layer(C.GEMMA3_4B, B=2, T=500, seed=24, d_model=512)
    q, K, V, out = gpu_unfused(L)
    ws = kvd.workspace(L.shape, kvd.KVD_OP_CACHED_ATTN, L.B, L.T + 1)
    outc = torch.empty_like(out)
    kvd.kvd_cached_attn(L.shape, q, K, V, L.T + 1, outc, ws)
    assert torch.equal(_bits(outc), _bits(out))
    check("cached vs oracle", outc, oracle_decode(L), 2e-2)


def test_partials_then_combine_equals_one_call():
    # out=None leaves the split-K partials in the workspace; kvd_combine merges them
    # exactly as the one-call form does.
    L = make_layer(C.GEMMA3_4B, B=2, T=333, seed=25, d_model=512)
    q, (tk, tv), out1, _ = gpu_fused(L)
    s = L.shape
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, L.T, 1)
    kvd.kvd_fused_recompute_attn(s, q, L.h, L.T, L.gamma, L.lw_k, L.lw_v, L.pos0, None, ws, tk, tv, 1)
    out2 = torch.empty_like(out1)
    kvd.kvd_combine(s, L.B, kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, L.T, 1), ws, out2)
    assert torch.equal(_bits(out1), _bits(out2))
    q, K, V, outd = gpu_unfused(L)
    wsd = kvd.workspace(s, kvd.KVD_OP_DECODE_ATTN, L.B, L.T + 1)
    kvd.kvd_decode_attn(s, q, K, V, L.T + 1, None, wsd)
    out3 = torch.empty_like(outd)
    kvd.kvd_combine(s, L.B, kvd.kvd_num_splits(s, kvd.KVD_OP_DECODE_ATTN, L.B, L.T + 1), wsd, out3)
    assert torch.equal(_bits(outd), _bits(out3))


@pytest.mark.parametrize("dtype", [BF, F32])
@pytest.mark.parametrize("T_rec,T", [(130, 430), (0, 200), (64, 384), (200, 260), (126, 129), (128, 131), (61, 64),
                                     (64, 66)])
def test_hybrid_budget_stored_window(dtype, T_rec, T):
    # Algorithm 1 with a cache budget: the T - T_rec most recent context tokens
    # keep stored K/V (the library's own, bit-identical to what prefill stores)
    # and form the tail with the current token; the older T_rec are recomputed
    # in the kernel.  (130, 430) has more tail tiles than recompute tiles;
    # (0, 200) is tail-only.  Tails of
    # <= 4 rows join the last recomputed tile in bf16: after a full tile
    # (128, 131), or moved down over a partial one, overlapping (126, 129) or not
    # (61, 64), (64, 66).
    kw = dict(d_model=512) if dtype == BF else dict(d_model=512, n_q=8, n_kv=4, head_dim=64)
    L = make_layer(C.GEMMA3_4B if dtype == BF else C.SMOLLM_FP32, B=2, T=T, seed=40 + T_rec, pos0=[3, 250], **kw)
    s, tol = L.shape, TOL[dtype]
    q, K, V, out_u = gpu_unfused(L)   # K/V rows 0..T-1 recomputed, row T the current token
    T_tail = T - T_rec + 1

    def fused(out, ws):
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)

    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    out = torch.empty_like(q)
    fused(out, ws)
    check("hybrid fused vs oracle", out, oracle_decode(L), tol)
    check("hybrid fused vs unfused", out, f64(out_u), tol)
    if dtype == F32 and T_rec % 64 == 0 and \
            kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail) == -(-(T + 1) // 64):
        assert torch.equal(_bits(out), _bits(out_u))  # identical 64-key chunking: identical arithmetic
    out2 = torch.empty_like(q)
    fused(out2, ws)  # the workspace's counters were left zero
    assert torch.equal(_bits(out), _bits(out2))
    fused(None, ws)  # partials only
    out3 = torch.empty_like(q)
    kvd.kvd_combine(s, L.B, kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail), ws, out3)
    assert torch.equal(_bits(out), _bits(out3))
    ctr_bytes = -(-L.B * s.n_kv_heads * 8 // 256) * 256  # the split counters open the workspace
    assert int(torch.count_nonzero(ws[:ctr_bytes])) == 0


def test_workspace_shared_across_key_counts_and_ops():
    # a decode loop keeps one workspace (sized for its largest call) while its
    # context grows or restarts: the split counters sit at a place that depends
    # on B only, so every call finds them zero whatever the previous call's split
    # count was.  Each output equals the one computed with a fresh workspace.
    L = make_layer(C.GEMMA3_4B, B=2, T=330, seed=77, d_model=512)
    s = L.shape
    q, K, V, _ = gpu_unfused(L)   # K/V rows 0..329 recomputed, row 330 the current token
    def fused(T_rec, T_tail, ws):
        out = torch.empty_like(q)
        kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)
        return out

    def decode(T, ws):
        out = torch.empty_like(q)
        kvd.kvd_decode_attn(s, q, K, V, T, out, ws, 331 - T)
        return out

    calls = [(fused, (330, 1)), (fused, (65, 1)), (decode, (331,)), (fused, (1, 1)), (fused, (260, 71)),
             (decode, (5,)), (fused, (200, 131)), (fused, (330, 1))]
    op_of = lambda fn: kvd.KVD_OP_DECODE_ATTN if fn is decode else kvd.KVD_OP_FUSED
    big = max(kvd.kvd_workspace_bytes(s, op_of(fn), L.B, *args) for fn, args in calls)
    shared = torch.zeros(big, dtype=torch.uint8, device="cuda")
    for fn, args in calls:
        fresh = kvd.workspace(s, op_of(fn), L.B, *args)
        ref = fn(*args, fresh)
        got = fn(*args, shared)
        note(f"    {fn.__name__}{args}")
        assert torch.equal(_bits(got), _bits(ref)), (fn.__name__, args)
    ctr_bytes = -(-L.B * s.n_kv_heads * 8 // 256) * 256
    assert int(torch.count_nonzero(shared[:ctr_bytes])) == 0


@pytest.mark.parametrize("hd", [64, 128, 256])
def test_packed_weights_bitwise_equal_rowmajor(hd):
    # the packed MFMA layout holds the same values and feeds the same arithmetic
    kw = dict(B=2, T=150, seed=26, d_model=512, n_q=4, n_kv=2, head_dim=hd, pos0=[3, 700])
    Lr = make_layer(C.GEMMA3_4B, packed=False, **kw)
    Lp = make_layer(C.GEMMA3_4B, packed=True, **kw)
    assert Lp.shape.w_layout == kvd.KVD_W_PACKED and not torch.equal(Lp.lw_k, Lp.w_k)
    for a, b in zip(gpu_recompute(Lr), gpu_recompute(Lp)):
        assert torch.equal(_bits(a), _bits(b))
    qr, (tkr, tvr), outr, (dkr, dvr) = gpu_fused(Lr, kv_debug=True)
    qp, (tkp, tvp), outp, (dkp, dvp) = gpu_fused(Lp, kv_debug=True)
    for a, b in [(qr, qp), (tkr, tkp), (tvr, tvp), (outr, outp), (dkr, dkp), (dvr, dvp)]:
        assert torch.equal(_bits(a), _bits(b))
    check("out fused (row-major weights)", outr, oracle_decode(Lr), 2e-2)
