"""GPU parity of the stored-K/V attention (kvd_decode_attn / kvd_cached_attn) and
of the recompute-vs-cached batch sweep at its full layer shape.

The bf16 stored-K/V attention streams each split's keys in 16-key blocks
(MFMA scores, online softmax, vector-ALU P V) and merges its waves and splits
in the log2 domain.  It is checked against the fp64 oracle's attention
(Eqs. attn_weights / head_output) evaluated on the same bf16 q, K and V, over
every head_dim, every query-group size the kernel is compiled for (including
group sizes it rounds up), ragged key counts around the 16-key block, rows
offset inside a larger cache, and split counts from one split per (sequence,
KV head) to the policy's most (32, or one per block).  Tolerance: 5e-3 of max |out| (the output's bf16
rounding is 2^-9 relative; scores and probabilities stay fp32).

The batch sweep test runs the Gemma-3-4B layer (d 2560, 8 q / 4 KV heads,
head_dim 256) at 2048 context tokens plus the current one for every batch the
benchmark sweeps, in the benchmark's launch configuration: fused and cached
outputs against the oracle on two sampled sequences, fused against cached on
every sequence (2e-2, bf16)."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import inputs
from paper_2603_19664_amd import kvd

from gpu_cases import err, f64, gpu_fused, gpu_project, make_layer, note, oracle_decode

pytestmark = pytest.mark.gpu

BF = kvd.KVD_BF16
TOL_ATTN = 5e-3
TOL = 2e-2


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()
    kvd.kvd_set_attn_workgroups(0)


def check(name, x, ref, tol):
    e = err(f64(x) if isinstance(x, torch.Tensor) else x, ref)
    note(f"    {name}: err {e:.3e} (tol {tol:g})")
    assert e < tol, f"{name}: err {e:.3e} >= {tol:g}"


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _qkv(B, n_q, n_kv, hd, t_cap, seed, q_std=2.0):
    """Seeded bf16 q [B, n_q, hd] and a K/V cache [B, n_kv, t_cap, hd]; q_std 2 gives
    scores of standard deviation ~2 (a peaked softmax that exposes key/head mix-ups)."""
    q = inputs.normal((B, n_q, hd), q_std, "cuda", seed, 90, 0).to(torch.bfloat16)
    K = inputs.normal((B, n_kv, t_cap, hd), 1.0, "cuda", seed, 90, 1).to(torch.bfloat16)
    V = inputs.normal((B, n_kv, t_cap, hd), 1.0, "cuda", seed, 90, 2).to(torch.bfloat16)
    return q, K, V


def _shape(n_q, n_kv, hd):
    return kvd.Shape(512, n_q, n_kv, hd, 1e-6, 1e4, BF)


def _attend(s, q, K, V, T, t_off, cached=False):
    ws = kvd.workspace(s, kvd.KVD_OP_CACHED_ATTN if cached else kvd.KVD_OP_DECODE_ATTN, q.shape[0], T)
    out = torch.empty_like(q)
    (kvd.kvd_cached_attn if cached else kvd.kvd_decode_attn)(s, q, K, V, T, out, ws, t_off)
    return out, ws


@pytest.mark.parametrize("hd", [64, 128, 256])
@pytest.mark.parametrize("g", [1, 2, 3, 5, 6, 8, 16])
def test_stream_attention_groups_and_head_dims(hd, g):
    n_kv = 2
    B, T, t_off, t_cap = 3, 1000, 9, 1020
    s = _shape(g * n_kv, n_kv, hd)
    q, K, V = _qkv(B, g * n_kv, n_kv, hd, t_cap, seed=hd * 100 + g)
    ref = O.decode_attention(f64(q), f64(K[:, :, t_off:t_off + T]), f64(V[:, :, t_off:t_off + T]))
    out, ws = _attend(s, q, K, V, T, t_off)
    check(f"decode_attn hd={hd} g={g}", out, ref, TOL_ATTN)
    outc, _ = _attend(s, q, K, V, T, t_off, cached=True)
    assert torch.equal(_bits(out), _bits(outc))
    ctr_bytes = -(-B * n_kv * 8 // 256) * 256
    assert int(torch.count_nonzero(ws[:ctr_bytes])) == 0


@pytest.mark.parametrize("T", [1, 2, 15, 16, 17, 63, 64, 65, 100, 257, 4097])
def test_stream_attention_key_counts(T):
    B, n_q, n_kv, hd = 2, 8, 4, 256
    s = _shape(n_q, n_kv, hd)
    q, K, V = _qkv(B, n_q, n_kv, hd, T + 3, seed=T)
    ref = O.decode_attention(f64(q), f64(K[:, :, 3:3 + T]), f64(V[:, :, 3:3 + T]))
    out, _ = _attend(s, q, K, V, T, 3)
    check(f"T={T} (splits {kvd.kvd_num_splits(s, kvd.KVD_OP_DECODE_ATTN, B, T)})", out, ref, TOL_ATTN)


@pytest.mark.parametrize("target", [1, 3, 8, 64, 512, 4096, 1 << 20])
def test_stream_attention_split_counts(target):
    # the split policy's workgroup target moves the key ranges of the splits; every
    # setting gives the same attention, in-kernel merges equal kvd_combine bitwise,
    # and the workspace's split counters are left zero
    B, n_q, n_kv, hd, T = 2, 12, 2, 128, 777
    s = _shape(n_q, n_kv, hd)
    q, K, V = _qkv(B, n_q, n_kv, hd, T, seed=31)
    ref = O.decode_attention(f64(q), f64(K), f64(V))
    kvd.kvd_set_attn_workgroups(target)
    S = kvd.kvd_num_splits(s, kvd.KVD_OP_DECODE_ATTN, B, T)
    assert 1 <= S <= -(-T // 16)
    out, ws = _attend(s, q, K, V, T, 0)
    check(f"target {target}: S={S}", out, ref, TOL_ATTN)
    out2, _ = _attend(s, q, K, V, T, 0)
    assert torch.equal(_bits(out), _bits(out2))  # run to run
    wsp = kvd.workspace(s, kvd.KVD_OP_DECODE_ATTN, B, T)
    kvd.kvd_decode_attn(s, q, K, V, T, None, wsp)  # partials only
    out3 = torch.empty_like(out)
    kvd.kvd_combine(s, B, S, wsp, out3)
    assert torch.equal(_bits(out), _bits(out3))
    ctr_bytes = -(-B * n_kv * 8 // 256) * 256
    assert int(torch.count_nonzero(ws[:ctr_bytes])) == 0


def test_stream_attention_extreme_scores():
    # one key far above the rest in every head (its weight ~1) and a sequence whose
    # keys all score alike (weights 1/T): the online max and rescaling across blocks,
    # waves and splits must keep both
    B, n_q, n_kv, hd, T = 2, 8, 4, 256, 900
    s = _shape(n_q, n_kv, hd)
    q, K, V = _qkv(B, n_q, n_kv, hd, T, seed=5, q_std=1.0)
    K[0, :, 611] = (q[0].float().view(n_kv, 2, hd).sum(1) * 8.0).to(torch.bfloat16)  # dominant key of b = 0
    K[1] = K[1, :, :1].expand_as(K[1])  # equal keys in b = 1
    ref = O.decode_attention(f64(q), f64(K), f64(V))
    for target in (1, 512, 1 << 20):
        kvd.kvd_set_attn_workgroups(target)
        out, _ = _attend(s, q, K, V, T, 0)
        check(f"extreme scores, target {target}", out, ref, TOL_ATTN)


@pytest.mark.parametrize("B", [1, 2, 4, 8, 16, 32, 64])
def test_batch_sweep_full_shape_gemma_ctx2048(B):
    # the recompute-vs-cached crossover workload at every swept batch, as timed:
    # packed weights, kvd_project_qkv for q and the current token's K/V, the fused
    # kernel with a one-row tail, and kvd_cached_attn over a prefilled 2049-row cache
    wl = C.GEMMA3_SWEEP
    T = wl.ctx
    L = make_layer(wl, B=B, T=T, layer=0)
    s = L.shape
    q, _, out_f, _ = gpu_fused(L)
    Kc = torch.empty((B, s.n_kv_heads, T + 1, s.head_dim), dtype=torch.bfloat16, device="cuda")
    Vc = torch.empty_like(Kc)
    kvd.kvd_recompute_kv(s, L.h, L.gamma, L.lw_k, L.lw_v, L.pos0, T, Kc, Vc, 0)
    q2 = gpu_project(L, (Kc, Vc), t_off=T)
    assert torch.equal(_bits(q), _bits(q2))
    out_c, _ = _attend(s, q, Kc, Vc, T + 1, 0, cached=True)
    note(f"    B={B}: fused splits {kvd.kvd_num_splits(s, kvd.KVD_OP_FUSED, B, T, 1)}, "
         f"cached splits {kvd.kvd_num_splits(s, kvd.KVD_OP_CACHED_ATTN, B, T + 1)}")
    for b in sorted({0, B - 1}):
        ref = oracle_decode(L, b_sel=[b])
        check(f"fused out[{b}] vs oracle", out_f[b:b + 1], ref, TOL)
        check(f"cached out[{b}] vs oracle", out_c[b:b + 1], ref, TOL)
    for b in range(B):
        e = err(f64(out_f[b:b + 1]), f64(out_c[b:b + 1]))
        assert e < TOL, (b, e)
    note(f"    fused vs cached, all {B} sequences: max err "
         f"{max(err(f64(out_f[b:b + 1]), f64(out_c[b:b + 1])) for b in range(B)):.3e}")
    assert torch.isfinite(out_f.float()).all() and torch.isfinite(out_c.float()).all()
