"""Algorithm 1's bounded cache on the host (Sec. 3.4; Eq. total_mem): the ring
bookkeeping of paper_2603_19664_amd.budget.RingState, checked step by step against
a plain list model of the cache, and an fp64 run of Algorithm 1 with the oracle's
own recompute showing that every budget attends the keys and values of an
unbounded cache (the paper's exactness claim, Prop. reconstruction), equal to
fp64 rounding."""
import numpy as np
import pytest

import oracle as O
from paper_2603_19664_amd import accounting
from paper_2603_19664_amd.budget import RingState


@pytest.mark.parametrize("budget", [0, 1, 2, 3, 7, 64])
def test_ring_state_matches_a_list_model_of_the_cache(budget):
    st = RingState(budget)
    cache = []                # token ids in the cache, oldest first (Algorithm 1's K[l])
    evicted = []              # token ids whose residual is a checkpoint
    ring = [None] * st.slots  # what each ring slot holds
    for t in range(400):
        assert st.T == t == st.T_rec + st.n_cached
        assert st.T_rec == max(0, t - budget) == len(evicted)
        assert st.keys_in_order() == evicted + cache + [t] == list(range(t + 1))
        free = st.free_slot()
        assert free not in {st.slot_of(c) for c in cache}
        assert st.slot_of(t) == free
        ring[free] = t                      # K_t / V_t written by the projection
        for c in cache:                     # the cached tokens are where the ring says
            assert ring[st.slot_of(c)] == c
        assert st.tail_rows() == len(cache) + 1 <= st.slots
        # tail rows read from slot head, wrapping: the cache oldest first, then the current token
        assert [ring[(st.head + i) % st.slots] for i in range(st.tail_rows())] == cache + [t]
        st.advance()
        cache.append(t)
        if len(cache) > budget:             # EVICT_OLDEST + STORE_RESIDUAL
            evicted.append(cache.pop(0))


def test_memory_against_eq_total_mem():
    # per layer and sequence, Gemma-3-4B layer shape: the evicted residuals are exactly
    # Eq. total_mem's (T - B) d b term; the cache holds B entries plus the current
    # token's slot, and the cached tokens' residuals are kept for their eviction
    d, n_kv, hd, b, budget = 2560, 4, 256, 2, 64
    st = RingState(budget)
    for _ in range(300):
        st.advance()
    m = st.memory_bytes(d, n_kv, hd, b)
    T = 300
    assert m["eq_total_mem"] == 2 * budget * n_kv * hd * b + (T - budget) * d * b
    assert m["eq_total_mem"] == accounting.total_memory(T, budget, 1, n_kv, hd, d, b)
    assert m["held"]["evicted_residuals"] == (T - budget) * d * b
    assert m["held"]["total"] - m["eq_total_mem"] == budget * d * b + 2 * n_kv * hd * b


@pytest.mark.parametrize("budget", [0, 2, 5])
def test_algorithm1_in_fp64_attends_the_full_cache(budget):
    # Algorithm 1 run with the oracle's arithmetic: each step concatenates the keys
    # recomputed from the evicted tokens' checkpoints, the ring's cached keys (oldest
    # first) and the current token's; its attention equals attention over an
    # unbounded cache of every token's K/V
    rng = np.random.default_rng(3)
    B, d, n_q, n_kv, hd, N = 2, 64, 4, 2, 16, 24
    h = rng.standard_normal((B, N, d))
    gamma = 1 + 0.1 * rng.standard_normal(d)
    w_q, w_k, w_v = (0.1 * rng.standard_normal((n * hd, d)) for n in (n_q, n_kv, n_kv))
    pos0 = np.array([0, 7])
    pos = pos0[:, None] + np.arange(N)[None, :]
    K_full, V_full = O.recompute_kv(h, gamma, w_k, w_v, pos, n_kv, hd, 1e-6, 1e4)
    st = RingState(budget)
    ring_k = np.zeros((B, n_kv, st.slots, hd))
    ring_v = np.zeros_like(ring_k)
    for t in range(N):
        q, k_t, v_t = O.project_qkv(h[:, t], gamma, w_q, w_k, w_v, pos[:, t], n_q, n_kv, hd, 1e-6, 1e4)
        ring_k[:, :, st.free_slot()] = k_t
        ring_v[:, :, st.free_slot()] = v_t
        K_old, V_old = O.recompute_kv(h[:, :st.T_rec], gamma, w_k, w_v, pos[:, :st.T_rec], n_kv, hd, 1e-6, 1e4)
        order = [(st.head + i) % st.slots for i in range(st.tail_rows())]
        K_all = np.concatenate([K_old, ring_k[:, :, order]], axis=2)
        V_all = np.concatenate([V_old, ring_v[:, :, order]], axis=2)
        # equal up to fp64 rounding (the BLAS product's summation order depends on the row count)
        np.testing.assert_allclose(K_all, K_full[:, :, :t + 1], rtol=0, atol=1e-13)
        np.testing.assert_allclose(V_all, V_full[:, :, :t + 1], rtol=0, atol=1e-13)
        out = O.decode_attention(q, K_all, V_all)
        np.testing.assert_allclose(out, O.decode_attention(q, K_full[:, :, :t + 1], V_full[:, :, :t + 1]),
                                   rtol=0, atol=1e-13)
        st.advance()
