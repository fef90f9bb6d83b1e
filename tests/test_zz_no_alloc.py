"""The allocation-free fused call (kvd_fused_recompute_attn_noalloc) against the
workspace form (kvd_fused_recompute_attn) through the C ABI: two calls in a row on
the shared static scratch, the second with a smaller input, each output
bit-identical to the workspace call's (the same kernels run on the same values)
and within the bf16 tolerance (2e-2) of the fp64 oracle; then an fp32 call
(1e-5), one at the Gemma-3-4B headline size and a head_dim 128 call on the pair
engine (two KV heads per tile)."""
import pytest
import torch

from paper_2603_19664_amd import configs as C
from paper_2603_19664_amd import kvd

from gpu_cases import TOL, empty_kv, err, f64, gpu_project, make_layer, note, oracle_decode

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t.view(torch.int32)


def _both(L):
    s = L.shape
    tk, tv = empty_kv(L, 1)
    q = gpu_project(L, (tk, tv), 0)
    ws = kvd.workspace(s, kvd.KVD_OP_FUSED, L.B, L.T, 1)
    out_ws = torch.empty_like(q)
    kvd.kvd_fused_recompute_attn(s, q, L.h, L.T, L.gamma, L.lw_k, L.lw_v, L.pos0, out_ws, ws, tk, tv, 1)
    out_na = torch.full_like(q, float("nan"))
    kvd.kvd_fused_recompute_attn_noalloc(s, q, L.h, L.T, L.gamma, L.lw_k, L.lw_v, L.pos0, out_na, tk, tv, 1)
    torch.cuda.synchronize()
    return out_ws, out_na


@pytest.mark.parametrize("case", ["bf16_two_calls_second_smaller", "fp32", "gemma_headline_size", "pair_engine"])
def test_noalloc_matches_workspace_call(case):
    note(f"[gpu] noalloc {case}")
    if case == "bf16_two_calls_second_smaller":
        layers = [make_layer(C.GEMMA3_4B, B=3, T=700, seed=61, d_model=512, pos0=[0, 9, 500]),
                  make_layer(C.GEMMA3_4B, B=1, T=130, seed=62, d_model=512)]
    elif case == "fp32":
        layers = [make_layer(C.SMOLLM_FP32, B=2, T=256, seed=63, pos0=[0, 31]),
                  make_layer(C.SMOLLM_FP32, B=1, T=40, seed=64)]
    elif case == "pair_engine":
        # head_dim 128: 4 sequences x 4 pairs of KV heads x 16 tiles = 256 pair tiles (the
        # pair engine), then a call too small for it
        qw = dict(d_model=512, n_q=16, n_kv=8, head_dim=128)
        layers = [make_layer(C.QWEN_1_5B, B=4, T=2000, seed=65, pos0=[0, 300, 17, 900], **qw),
                  make_layer(C.QWEN_1_5B, B=1, T=300, seed=66, **qw)]
    else:
        layers = [make_layer(C.GEMMA3_4B, B=1, T=4096, layer=7), make_layer(C.GEMMA3_4B, B=1, T=1000, layer=8)]
    for i, L in enumerate(layers):
        out_ws, out_na = _both(L)
        assert torch.equal(_bits(out_ws), _bits(out_na)), (case, i)
        e = err(f64(out_na), oracle_decode(L))
        note(f"    call {i}: B={L.B} T={L.T}: bitwise equal to the workspace call; err vs oracle {e:.3e}")
        assert e < TOL[L.shape.dtype]
