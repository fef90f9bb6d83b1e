"""Closed-form accounting against the numbers the paper prints (Section 3.4 worked
example; Table tab:models).  Runs on the CPU."""
import json
import os

import pytest

from paper_2603_19664_amd import accounting as acc


@pytest.fixture(scope="module")
def golden(golden_dir):
    with open(os.path.join(golden_dir, "paper_memory.json")) as f:
        return json.load(f)


def test_worked_example(golden):
    w = golden["worked_example"]
    assert acc.kv_bytes_per_token(w["L"], w["n_kv"], w["head_dim"], w["b"]) == w["kv_bytes"]
    assert acc.residual_bytes_per_token(w["d_hidden"], w["b"]) == w["res_bytes"]
    assert round(acc.compression_ratio(w["L"], w["n_kv"], w["head_dim"], w["d_hidden"]), 1) == w["rho"]
    assert round(w["kv_bytes"] / 1024) == w["kv_kb_approx"]


def test_model_table(golden):
    for m in golden["models"]:
        kv = acc.kv_bytes_per_token(m["L"], m["n_kv"], m["head_dim"], 2) / 1024
        res = acc.residual_bytes_per_token(m["d"], 2) / 1024
        rho = acc.compression_ratio(m["L"], m["n_kv"], m["head_dim"], m["d"])
        assert round(kv, 1) == m["kv_kb"], m["model"]
        assert round(res, 1) == m["res_kb"], m["model"]
        assert round(rho, 1) == m["rho"], m["model"]
        assert round(100 * (1 - 1 / rho)) == m["saving_pct"], m["model"]


def test_rho_range(golden):
    rhos = {m["model"]: acc.compression_ratio(m["L"], m["n_kv"], m["head_dim"], m["d"]) for m in golden["models"]}
    r = golden["rho_range"]
    assert round(min(rhos.values()), 1) == r["min"] and min(rhos, key=rhos.get) == r["min_model"]
    assert round(max(rhos.values()), 1) == r["max"] and max(rhos, key=rhos.get) == r["max_model"]


def test_recompute_vs_read_intensity():
    # Eq. recomp_flops / Eq. read_bytes = d_hidden flop per byte at b = 2 (Section 3.4).
    for d, n_kv, hd in [(2560, 4, 256), (1536, 2, 128), (576, 3, 64)]:
        assert acc.recompute_flops(7, n_kv, d, hd) / acc.read_bytes(7, n_kv, hd, 2) == d


def test_total_memory_limits():
    L, n_kv, hd, d, b = 34, 4, 256, 2560, 2
    T = 1000
    # budget = T: the plain KV cache; budget = 0: residuals only (Eq. total_mem).
    assert acc.total_memory(T, T, L, n_kv, hd, d, b) == T * acc.kv_bytes_per_token(L, n_kv, hd, b)
    assert acc.total_memory(T, 0, L, n_kv, hd, d, b) == T * acc.residual_bytes_per_token(d, b)
    # growth rate in T at fixed budget is d*b per token
    assert acc.total_memory(T + 1, 64, L, n_kv, hd, d, b) - acc.total_memory(T, 64, L, n_kv, hd, d, b) == d * b
