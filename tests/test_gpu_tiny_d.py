"""GPU parity at the smallest residual widths (d_model = 64 .. 320: one to five
K-steps of 64), where the tile engines' prefetch rings (weights and residual
rows loaded up to four K-steps ahead) run only their clamped first and last
iterations.  Every fused engine's recomputed K/V (dumped through kv_debug) must
equal the prefill K/V of kvd_recompute_kv bit for bit (Prop. reconstruction:
one MFMA chain over d per element), and the decode-step output must match the
fp64 oracle (Eqs. attn_weights / head_output) within the bf16 tolerance, 2e-2.
The current token's K_t / V_t from kvd_project_qkv must equal a recompute of
the same residual row."""
import pytest
import torch

from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import TOL, empty_kv, err, f64, gpu_fused, gpu_project, gpu_recompute, make_layer, note, oracle_decode

pytestmark = pytest.mark.gpu

TOL_BF = TOL[kvd.KVD_BF16]
ENGINES = {"tile64": 64, "wide": 128, "pair": kvd.KVD_FUSED_PAIR, "split64": kvd.KVD_FUSED_SPLIT64,
           "split128": kvd.KVD_FUSED_SPLIT}


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()
    kvd.kvd_set_fused_tokens(0)


def _bits(t):
    return t.view(torch.int16)


@pytest.mark.parametrize("d", [64, 128, 192, 320])
@pytest.mark.parametrize("hd", [128, 256])
def test_tiny_d_every_engine(d, hd):
    n_q, n_kv = (12, 2) if hd == 128 else (8, 4)
    wl = C.QWEN_1_5B if hd == 128 else C.GEMMA3_4B
    L = make_layer(wl, B=2, T=300, seed=500 + d + hd, pos0=[5, 900], d_model=d, n_q=n_q, n_kv=n_kv, head_dim=hd)
    K, V = gpu_recompute(L)
    ref = oracle_decode(L)
    q = None
    for name, mode in ENGINES.items():
        kvd.kvd_set_fused_tokens(mode)
        q_, _, out, (dk, dv) = gpu_fused(L, q=q, kv_debug=True)
        q = q_ if q is None else q
        assert torch.equal(_bits(dk), _bits(K)) and torch.equal(_bits(dv), _bits(V)), f"{name}: K/V differ"
        e = err(f64(out), ref)
        note(f"    d={d} hd={hd} {name}: K/V bit-identical to the prefill; err vs oracle {e:.3e}")
        assert e < TOL_BF, (name, e)


@pytest.mark.parametrize("d", [64, 192])
def test_tiny_d_current_token_matches_recompute(d):
    # K_t / V_t of the current token equal the recompute of the same residual row
    # at the same position (the row appended after the context)
    L = make_layer(C.GEMMA3_4B, B=2, T=40, seed=600 + d, pos0=[0, 77], d_model=d, n_q=8, n_kv=4, head_dim=256)
    s = L.shape
    tk, tv = empty_kv(L, 1)
    gpu_project(L, (tk, tv), 0)
    h = torch.cat([L.h[:, :L.T], L.h_new[:, None, :]], dim=1).contiguous()
    K, V = empty_kv(L, L.T + 1)
    kvd.kvd_recompute_kv(s, h, L.gamma, L.lw_k, L.lw_v, L.pos0, L.T + 1, K, V, 0)
    assert torch.equal(_bits(tk[:, :, 0]), _bits(K[:, :, L.T])) and torch.equal(_bits(tv[:, :, 0]), _bits(V[:, :, L.T]))
