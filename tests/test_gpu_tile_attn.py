"""GPU parity of the fused kernels' bf16 tile attention (16x16x32 MFMAs: S^T = K q^T
from the tile's K rows, O^T = V^T P^T with V^T taken from the row-major V rows by LDS
transpose reads) over the group sizes and head dims the boundary accepts, on every
fused engine: 64-token tiles, 128-token wide tiles, and the split engine with 64- and
128-token chunks (its K role scores, its V role multiplies).

Each case recomputes T = 200 context rows (a ragged last tile) and attends them with
the current token folded into the last tile, or with a stored tail of 70 rows (64-row
tail tiles plus a remainder of 6, attended by the same tile code from stored K/V).
Tolerance (max |gpu - oracle| / max |oracle|): 2e-2 for bf16 (Eqs. attn_weights /
head_output; the probabilities enter the P V product rounded to bf16)."""
import pytest
import torch

from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import TOL, err, f64, gpu_fused, gpu_unfused, make_layer, note, oracle_decode

pytestmark = pytest.mark.gpu

BF = kvd.KVD_BF16
MODES = {"tile64": 64, "wide": 128, "split64": kvd.KVD_FUSED_SPLIT64, "split128": kvd.KVD_FUSED_SPLIT}


@pytest.fixture(autouse=True)
def _announce(request):
    note(f"[gpu] {request.node.nodeid}")
    yield
    torch.cuda.synchronize()
    kvd.kvd_set_fused_tokens(0)


def _layer(hd, g, seed, T=200):
    wl = C.GEMMA3_4B if hd == 256 else C.QWEN_1_5B
    return make_layer(wl, B=2, T=T, seed=seed, pos0=[5, 900], d_model=512, n_q=2 * g, n_kv=2, head_dim=hd)


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("g", [1, 3, 16])
@pytest.mark.parametrize("hd", [64, 128, 256])
def test_tile_attention_groups(hd, g, mode):
    L = _layer(hd, g, seed=300 + 7 * g + hd)
    kvd.kvd_set_fused_tokens(MODES[mode])
    _, _, out, _ = gpu_fused(L)
    e = err(f64(out), oracle_decode(L))
    note(f"    hd={hd} g={g} {mode}: err {e:.3e}")
    assert torch.isfinite(out.float()).all()
    assert e < TOL[BF], e


@pytest.mark.parametrize("g", [1, 6, 16])
@pytest.mark.parametrize("hd", [128, 256])
def test_tile_attention_stored_tail_tiles(hd, g):
    # the oldest 131 rows recomputed, the other 69 context rows and the current
    # token read as a 70-row stored tail: one 64-row tail tile plus a remainder
    # of 6 rows in a second (each attended by the tile code from stored K/V)
    T, T_rec = 200, 131
    L = _layer(hd, g, seed=400 + g + hd, T=T)
    s = L.shape
    q, K, V, out_u = gpu_unfused(L)
    T_tail = T - T_rec + 1
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, T_rec, T_tail)
    out = torch.empty_like(q)
    kvd.kvd_fused_recompute_attn(s, q, L.h, T_rec, L.gamma, L.lw_k, L.lw_v, L.pos0, out, ws, K, V, T_tail, T_rec)
    e = err(f64(out), oracle_decode(L))
    note(f"    hd={hd} g={g} stored tail: err {e:.3e} (vs unfused {err(f64(out), f64(out_u)):.3e})")
    assert e < TOL[BF], e
    assert err(f64(out), f64(out_u)) < TOL[BF]
