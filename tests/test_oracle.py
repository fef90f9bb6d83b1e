"""Pins of the fp64 oracle against facts the paper and mathematics fix, independent
of the oracle's own formulas: closed forms, invariants, special cases and brute
force on tiny inputs.  CPU only."""
import math

import numpy as np
import pytest

import oracle as O

rng = np.random.default_rng(1234)


# ---------------------------------------------------------------- RMSNorm (Sec. 3.1)

def test_rmsnorm_constant_vector_closed_form():
    # h = c * 1: mean(h^2) = c^2, so hbar = gamma * c / sqrt(c^2 + eps).
    d = 12
    gamma = rng.normal(1.0, 0.3, d)
    for c, eps in [(2.0, 0.5), (-3.0, 0.0), (0.25, 1e-6)]:
        hbar = O.rms_normalize(np.full(d, c), gamma, eps)
        np.testing.assert_allclose(hbar, gamma * c / math.sqrt(c * c + eps), rtol=1e-15)


def test_rmsnorm_unit_rms_without_eps():
    # With eps = 0 and gamma = 1 the normalised vector has RMS exactly 1 (Eq. rms_def).
    h = rng.normal(0, 5, (7, 33))
    hbar = O.rms_normalize(h, np.ones(33), 0.0)
    np.testing.assert_allclose(np.sqrt(np.mean(hbar ** 2, axis=-1)), 1.0, rtol=1e-14)


def test_rmsnorm_degree_zero_homogeneity():
    # Sec. 3.1: RMSNorm(a x) = RMSNorm(x) for a > 0 (exact at eps = 0) ...
    h = rng.normal(0, 1, (5, 64))
    g = rng.normal(1, 0.1, 64)
    for a in [0.5, 1.7, 4.0]:
        np.testing.assert_allclose(O.rms_normalize(a * h, g, 0.0), O.rms_normalize(h, g, 0.0), rtol=1e-14)
    # ... and otherwise within the eps-induced first-order bound |1 - 1/a^2| eps / (2 ms).
    eps = 1e-6
    ms = np.mean(h ** 2, axis=-1, keepdims=True)
    for a in [0.5, 4.0]:
        r = O.rms_normalize(a * h, g, eps) / O.rms_normalize(h, g, eps)
        assert np.max(np.abs(r - 1)) <= np.max(abs(1 - 1 / a ** 2) * eps / (2 * ms)) * 1.01


def test_rmsnorm_negative_scale_flips_sign():
    h = rng.normal(0, 1, 16)
    g = rng.normal(1, 0.1, 16)
    np.testing.assert_allclose(O.rms_normalize(-2 * h, g, 0.0), -O.rms_normalize(h, g, 0.0), rtol=1e-14)


# ---------------------------------------------------------------- RoPE (Sec. 3.2)

def test_rope_quarter_turn_and_pairing():
    # phi_0 = p * theta^0 = p.  With p = pi/2 the first pair turns by +90 degrees:
    # (1, 0) -> (0, 1) and (0, 1) -> (-1, 0) (Eqs. rope_cos / rope_sin: consecutive pairs,
    # rotation by +phi).  The other pair (frequency theta^(-2/4) = 1/2 at theta = 4)
    # turns by pi/4.
    hd, theta = 4, 4.0
    p = math.pi / 2
    e0 = O.apply_rope(np.array([1.0, 0, 0, 0]), p, theta)
    np.testing.assert_allclose(e0, [0, 1, 0, 0], atol=1e-15)
    e1 = O.apply_rope(np.array([0, 1.0, 0, 0]), p, theta)
    np.testing.assert_allclose(e1, [-1, 0, 0, 0], atol=1e-15)
    e2 = O.apply_rope(np.array([0, 0, 1.0, 0]), p, theta)
    s = math.sqrt(0.5)
    np.testing.assert_allclose(e2, [0, 0, s, s], atol=1e-15)


def test_rope_consecutive_pairs_not_half_split():
    # A basis vector only mixes with its neighbour in the same consecutive pair.
    hd = 16
    for i in range(hd):
        x = np.zeros(hd)
        x[i] = 1.0
        y = O.apply_rope(x, 37, 10000.0)
        nz = set(np.nonzero(np.abs(y) > 1e-12)[0])
        assert nz <= {i - i % 2, i - i % 2 + 1}


def test_rope_identity_at_zero_and_norm_preserving():
    x = rng.normal(0, 1, (9, 64))
    np.testing.assert_array_equal(O.apply_rope(x, 0, 1e4), x)
    for p in [1, 255, 4096, 17407]:
        y = O.apply_rope(x, p, 1e4)
        np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-14)


def test_rope_dense_matrix_orthogonal_and_matches():
    # R_p^T R_p = I (Sec. 3.2) and the dense block matrix equals the pairwise rotation.
    for hd, p, th in [(8, 3, 1e4), (64, 256, 1e4), (128, 9999, 1e6)]:
        R = O.rope_matrix(p, hd, th)
        np.testing.assert_allclose(R.T @ R, np.eye(hd), atol=1e-14)
        x = rng.normal(0, 1, hd)
        np.testing.assert_allclose(R @ x, O.apply_rope(x, p, th), atol=1e-13)


def test_rope_relative_position():
    # <R_p x, R_p' y> depends only on p - p' (the property RoPE is built for).
    x, y = rng.normal(0, 1, 64), rng.normal(0, 1, 64)
    base = O.apply_rope(x, 10, 1e4) @ O.apply_rope(y, 3, 1e4)
    for s in [1, 100, 5000]:
        np.testing.assert_allclose(O.apply_rope(x, 10 + s, 1e4) @ O.apply_rope(y, 3 + s, 1e4), base, rtol=1e-9)


def test_rope_frequencies_span_one_to_inverse_theta():
    # The adopted 0-based reading: phi_0 = p and phi_{hd/2-1} = p * theta^(-(hd-2)/hd).
    phi = O.rope_angles(np.array(5.0), 8, 10000.0)
    np.testing.assert_allclose(phi, 5.0 * np.array([1, 10000 ** -0.25, 10000 ** -0.5, 10000 ** -0.75]), rtol=1e-15)


def test_sliding_window_error_closed_form():
    # Eq. sw_error: || K_recon - K_window || = || (R_j - R_{j-w}) k ||, nonzero for w != 0;
    # V carries no rotation.  Here k is one head's un-rotated key.
    k = rng.normal(0, 1, 64)
    j, w = 700, 512
    lhs = np.linalg.norm(O.apply_rope(k, j, 1e4) - O.apply_rope(k, j - w, 1e4))
    rhs = np.linalg.norm((O.rope_matrix(j, 64, 1e4) - O.rope_matrix(j - w, 64, 1e4)) @ k)
    np.testing.assert_allclose(lhs, rhs, rtol=1e-12)
    assert lhs > 1e-3


def _sw_layer(B=2, T=13, d=32, n_q=4, n_kv=2, hd=8, seed=7):
    r = np.random.default_rng(seed)
    h_ctx = r.normal(0, 1, (B, T, d))
    h_new = r.normal(0, 1, (B, d))
    gamma = r.normal(1, 0.1, d)
    wq, wk, wv = (r.normal(0, 0.3, (n * hd, d)) for n in (n_q, n_kv, n_kv))
    return h_ctx, h_new, gamma, wq, wk, wv, n_q, n_kv, hd


def test_sliding_window_start():
    assert O.window_start(10, 4) == 6 and O.window_start(10, 10) == 0 and O.window_start(3, 1024) == 0
    assert O.window_start(5, 1) == 4
    with pytest.raises(ValueError):
        O.window_start(5, 0)


def test_sliding_window_wide_window_is_global_attention():
    # A window holding every key (w = 0) is plain global attention at positions 0..T.
    h_ctx, h_new, gamma, wq, wk, wv, n_q, n_kv, hd = _sw_layer()
    B, T, _ = h_ctx.shape
    rows = np.concatenate([h_ctx, h_new[:, None]], axis=1)
    K, V = O.recompute_kv(rows, gamma, wk, wv, np.tile(np.arange(T + 1.0), (B, 1)), n_kv, hd, 1e-6, 1e4)
    q = O.project_qkv(h_new, gamma, wq, wk, wv, np.full(B, float(T)), n_q, n_kv, hd, 1e-6, 1e4)[0]
    ref = O.decode_attention(q, K, V)
    for window in (T + 1, T + 50):
        out = O.sliding_window_decode(h_new, h_ctx, gamma, wq, wk, wv, window, n_q, n_kv, hd, 1e-6, 1e4)
        np.testing.assert_allclose(out, ref, rtol=1e-13, atol=1e-15)


def test_sliding_window_rotation_offset_cancels_in_scores():
    # Window-relative rotation of keys (R_{j-w}) and query (R_{T-w}) gives the same
    # scores as absolute rotation over the same keys (R_j, R_T): <R_a x, R_b y> depends
    # on b - a only.  A query and keys rotated with different offsets would not.
    h_ctx, h_new, gamma, wq, wk, wv, n_q, n_kv, hd = _sw_layer(T=21)
    B, T, _ = h_ctx.shape
    for window in (1, 5, 9, 21):
        w = O.window_start(T + 1, window)
        rows = np.concatenate([h_ctx[:, w:], h_new[:, None]], axis=1)
        K, V = O.recompute_kv(rows, gamma, wk, wv, np.tile(np.arange(w, T + 1.0), (B, 1)), n_kv, hd, 1e-6, 1e4)
        q = O.project_qkv(h_new, gamma, wq, wk, wv, np.full(B, float(T)), n_q, n_kv, hd, 1e-6, 1e4)[0]
        out = O.sliding_window_decode(h_new, h_ctx, gamma, wq, wk, wv, window, n_q, n_kv, hd, 1e-6, 1e4)
        np.testing.assert_allclose(out, O.decode_attention(q, K, V), rtol=1e-9, atol=1e-12)


def test_sliding_window_of_one_returns_current_value():
    # window = 1 keeps only the current token: softmax over one key is 1, so every
    # query head returns its KV head's V_t = RMSNorm(h_new) W_v (brute-force loops).
    h_ctx, h_new, gamma, wq, wk, wv, n_q, n_kv, hd = _sw_layer()
    B, T, d = h_ctx.shape
    out = O.sliding_window_decode(h_new, h_ctx, gamma, wq, wk, wv, 1, n_q, n_kv, hd, 1e-6, 1e4)
    g = n_q // n_kv
    for b in range(B):
        r = 1.0 / math.sqrt(sum(x * x for x in h_new[b]) / d + 1e-6)
        for h in range(n_q):
            j = h // g
            for c in range(hd):
                v = sum(wv[j * hd + c, i] * h_new[b, i] * r * gamma[i] for i in range(d))
                assert abs(out[b, h, c] - v) <= 1e-12 * max(1.0, abs(v))


def test_sliding_window_masks_older_keys():
    # Keys older than the window do not take part: changing their residuals leaves
    # the output bit-identical, changing the oldest kept key does not.
    h_ctx, h_new, gamma, wq, wk, wv, n_q, n_kv, hd = _sw_layer(T=17)
    window = 6
    w = O.window_start(18, window)
    base = O.sliding_window_decode(h_new, h_ctx, gamma, wq, wk, wv, window, n_q, n_kv, hd, 1e-6, 1e4)
    h2 = h_ctx.copy()
    h2[:, :w] = rng.normal(0, 3, h2[:, :w].shape)
    assert np.array_equal(O.sliding_window_decode(h_new, h2, gamma, wq, wk, wv, window, n_q, n_kv, hd, 1e-6, 1e4),
                          base)
    h3 = h_ctx.copy()
    h3[:, w] += 1.0
    assert np.max(np.abs(O.sliding_window_decode(h_new, h3, gamma, wq, wk, wv, window, n_q, n_kv, hd, 1e-6, 1e4)
                         - base)) > 1e-6


# ---------------------------------------------------------------- projection (Eqs. k_proj / v_proj)

def test_projection_brute_force_loops():
    B, T, d, nh, hd = 2, 3, 10, 3, 4
    h = rng.normal(0, 1, (B, T, d))
    W = rng.normal(0, 1, (nh * hd, d))
    got = O.project_heads(h, W, nh, hd)
    for b in range(B):
        for t in range(T):
            for head in range(nh):
                for c in range(hd):
                    ref = 0.0
                    for i in range(d):
                        ref += h[b, t, i] * W[head * hd + c, i]
                    assert abs(got[b, t, head, c] - ref) < 1e-12


def test_recompute_unit_vector_rows():
    # W rows equal to basis vectors select coordinates of RMSNorm(h); K is those
    # coordinates rotated at each token's position, V the coordinates themselves.
    B, T, d, n_kv, hd = 2, 5, 16, 2, 4
    perm = rng.permutation(d)[: n_kv * hd]
    W = np.zeros((n_kv * hd, d))
    W[np.arange(n_kv * hd), perm] = 1.0
    h = rng.normal(0, 1, (B, T, d))
    gamma = rng.normal(1, 0.2, d)
    pos = np.arange(T)[None, :] + np.array([[0], [7]])
    K, V = O.recompute_kv(h, gamma, W, W, pos, n_kv, hd, 1e-6, 1e4)
    for b in range(B):
        for t in range(T):
            ms = np.mean(h[b, t] ** 2)
            sel = (h[b, t] * gamma / math.sqrt(ms + 1e-6))[perm].reshape(n_kv, hd)
            np.testing.assert_allclose(V[b, :, t], sel, rtol=1e-14)
            for j in range(n_kv):
                np.testing.assert_allclose(K[b, j, t], O.rope_matrix(pos[b, t], hd, 1e4) @ sel[j], atol=1e-14)


def test_value_free_of_position_key_not():
    # Eq. v_recon carries no rotation: V is the same at any position, K is not.
    B, T, d, n_kv, hd = 1, 3, 32, 2, 8
    h = rng.normal(0, 1, (B, T, d))
    g = np.ones(d)
    W = rng.normal(0, 0.1, (n_kv * hd, d))
    K0, V0 = O.recompute_kv(h, g, W, W, np.zeros((B, T)), n_kv, hd, 1e-6, 1e4)
    K1, V1 = O.recompute_kv(h, g, W, W, np.full((B, T), 123), n_kv, hd, 1e-6, 1e4)
    np.testing.assert_array_equal(V0, V1)
    assert np.max(np.abs(K0 - K1)) > 1e-3
    # at position 0 the key equals the value when W_k = W_v (R_0 = I)
    np.testing.assert_allclose(K0, V0, atol=1e-15)


# ---------------------------------------------------------------- attention (Eqs. attn_weights / head_output)

def test_attention_two_keys_closed_form():
    # scores 0 and ln 3 give weights 1/4 and 3/4; the 1/sqrt(d_head) scale is part of the score.
    hd = 16
    q = np.zeros((1, 1, hd))
    q[0, 0, 0] = math.sqrt(hd)
    K = np.zeros((1, 1, 2, hd))
    K[0, 0, 1, 0] = math.log(3.0)
    V = rng.normal(0, 1, (1, 1, 2, hd))
    out = O.decode_attention(q, K, V)
    np.testing.assert_allclose(out[0, 0], 0.25 * V[0, 0, 0] + 0.75 * V[0, 0, 1], rtol=1e-14)


def test_attention_special_cases():
    B, n_q, n_kv, T, hd = 2, 4, 2, 9, 8
    V = rng.normal(0, 1, (B, n_kv, T, hd))
    K = rng.normal(0, 1, (B, n_kv, T, hd))
    # q = 0: uniform weights, the mean of V
    out = O.decode_attention(np.zeros((B, n_q, hd)), K, V)
    for h in range(n_q):
        np.testing.assert_allclose(out[:, h], V[:, h // 2].mean(axis=1), rtol=1e-13)
    # T = 1: the single value
    q = rng.normal(0, 1, (B, n_q, hd))
    out1 = O.decode_attention(q, K[:, :, :1], V[:, :, :1])
    for h in range(n_q):
        np.testing.assert_allclose(out1[:, h], V[:, h // 2, 0], rtol=1e-14)
    # one dominant key (score ~ 1e4 above the rest): its value
    K2 = K.copy()
    K2[:, :, 5] = q[:, ::2] * 1e4 / np.linalg.norm(q[:, ::2], axis=-1, keepdims=True) ** 2 * math.sqrt(hd) / 1.0
    out2 = O.decode_attention(q[:, ::2].repeat(2, axis=1), K2, V)
    np.testing.assert_allclose(out2[:, 0], V[:, 0, 5], rtol=1e-10)
    # huge common score offsets do not overflow (max subtraction)
    out3 = O.decode_attention(q * 1e3, K, V)
    assert np.all(np.isfinite(out3))


def test_attention_gqa_head_mapping():
    # query heads 0..g-1 read KV head 0, g..2g-1 read KV head 1 (contiguous groups).
    B, n_q, n_kv, T, hd = 1, 6, 2, 5, 4
    V = np.zeros((B, n_kv, T, hd))
    V[:, 0] = 1.0
    V[:, 1] = 2.0
    out = O.decode_attention(rng.normal(0, 1, (B, n_q, hd)), rng.normal(0, 1, (B, n_kv, T, hd)), V)
    np.testing.assert_allclose(out[0, :3], 1.0, rtol=1e-14)
    np.testing.assert_allclose(out[0, 3:], 2.0, rtol=1e-14)


def test_attention_equals_online_chunked_softmax():
    # A streaming (online-softmax) evaluation over arbitrary chunks gives the same result,
    # the identity split-K decode attention rests on.
    B, n_q, n_kv, T, hd = 2, 6, 3, 101, 16
    q = rng.normal(0, 2, (B, n_q, hd))
    K = rng.normal(0, 2, (B, n_kv, T, hd))
    V = rng.normal(0, 1, (B, n_kv, T, hd))
    ref = O.decode_attention(q, K, V)
    g = n_q // n_kv
    for chunk in [1, 7, 32, 100]:
        for b in range(B):
            for h in range(n_q):
                m, l, acc = -np.inf, 0.0, np.zeros(hd)
                for c0 in range(0, T, chunk):
                    s = K[b, h // g, c0:c0 + chunk] @ q[b, h] / math.sqrt(hd)
                    mc = s.max()
                    pc = np.exp(s - mc)
                    m_new = max(m, mc)
                    l = l * math.exp(m - m_new) + pc.sum() * math.exp(mc - m_new)
                    acc = acc * math.exp(m - m_new) + (pc @ V[b, h // g, c0:c0 + chunk]) * math.exp(mc - m_new)
                    m = m_new
                np.testing.assert_allclose(acc / l, ref[b, h], rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- decode step (Algorithm 1, budget 0)

def test_decode_step_concat_and_current_token():
    # The current token's own K_t, V_t (projected at its position) equal what
    # recomputation from its residual gives, and a decode step equals attention over
    # [recomputed context || current token] (Algorithm 1's CONCAT + ATTENTION).
    B, T, d, n_q, n_kv, hd = 2, 11, 32, 4, 2, 8
    h = rng.normal(0, 1, (B, T + 1, d))
    gamma = rng.normal(1, 0.1, d)
    wq, wk, wv = (rng.normal(0, 0.2, (n * hd, d)) for n in (n_q, n_kv, n_kv))
    pos = np.arange(T + 1)[None, :] + np.array([[0], [40]])
    q, kt, vt = O.project_qkv(h[:, T], gamma, wq, wk, wv, pos[:, T], n_q, n_kv, hd, 1e-6, 1e4)
    Kall, Vall = O.recompute_kv(h, gamma, wk, wv, pos, n_kv, hd, 1e-6, 1e4)
    np.testing.assert_allclose(kt, Kall[:, :, T], rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(vt, Vall[:, :, T], rtol=1e-13, atol=1e-15)
    out = O.kv_direct_decode(q, h[:, :T], gamma, wk, wv, pos[:, :T], kt[:, :, None], vt[:, :, None],
                             n_kv, hd, 1e-6, 1e4)
    np.testing.assert_allclose(out, O.decode_attention(q, Kall, Vall), rtol=1e-12, atol=1e-14)
    # the query at the last position scores against RoPE'd keys: shifting every position by
    # the same offset leaves the output unchanged (relative positions only)
    q2, kt2, vt2 = O.project_qkv(h[:, T], gamma, wq, wk, wv, pos[:, T] + 1000, n_q, n_kv, hd, 1e-6, 1e4)
    out2 = O.kv_direct_decode(q2, h[:, :T], gamma, wk, wv, pos[:, :T] + 1000, kt2[:, :, None],
                              vt2[:, :, None], n_kv, hd, 1e-6, 1e4)
    np.testing.assert_allclose(out2, out, rtol=1e-9, atol=1e-12)


# ---------------------------------------------------------------- single-checkpoint scheme (Sec. 3.1 block)

def test_silu_closed_forms():
    x = rng.normal(0, 3, 50)
    np.testing.assert_allclose(O.silu(x) - O.silu(-x), x, rtol=1e-14, atol=1e-14)  # x s(x) + x s(-x) = x
    assert O.silu(0.0) == 0.0
    np.testing.assert_allclose(O.silu(1.0), 1.0 / (1.0 + math.exp(-1.0)), rtol=1e-15)
    np.testing.assert_allclose(O.silu(40.0), 40.0, rtol=1e-15)


def _block_params(d, n_q, n_kv, hd, dff, r):
    return (r.normal(1, 0.1, d), r.normal(0, 0.3, (n_q * hd, d)), r.normal(0, 0.3, (n_kv * hd, d)),
            r.normal(0, 0.3, (n_kv * hd, d)), r.normal(0, 0.3, (d, n_q * hd)), r.normal(1, 0.1, d),
            r.normal(0, 0.3, (dff, d)), r.normal(0, 0.3, (dff, d)), r.normal(0, 0.3, (d, dff)))


def test_swiglu_mlp_brute_force():
    r = np.random.default_rng(3)
    d, dff = 5, 7
    x = r.normal(0, 1, (2, d))
    wg, wu, wd = r.normal(0, 1, (dff, d)), r.normal(0, 1, (dff, d)), r.normal(0, 1, (d, dff))
    out = O.swiglu_mlp(x, wg, wu, wd)
    for b in range(2):
        for o in range(d):
            acc = 0.0
            for f in range(dff):
                gt = sum(wg[f, i] * x[b, i] for i in range(d))
                ut = sum(wu[f, i] * x[b, i] for i in range(d))
                acc += wd[o, f] * gt / (1.0 + math.exp(-gt)) * ut
            assert abs(out[b, o] - acc) <= 1e-12 * max(1.0, abs(acc))


def test_causal_attention_first_position_causality_and_last_position():
    r = np.random.default_rng(4)
    B, n_q, n_kv, T, hd = 2, 4, 2, 9, 8
    q = r.normal(0, 1, (B, n_q, T, hd))
    K, V = r.normal(0, 1, (B, n_kv, T, hd)), r.normal(0, 1, (B, n_kv, T, hd))
    out = O.causal_attention(q, K, V)
    # position 0 has one key: its output is V_0 of its KV head
    for h in range(n_q):
        np.testing.assert_allclose(out[:, 0, h * hd:(h + 1) * hd], V[:, h // 2, 0], rtol=1e-14)
    # keys after p do not reach p
    K2, V2 = K.copy(), V.copy()
    K2[:, :, 5:] += 3.0
    V2[:, :, 5:] -= 2.0
    assert np.array_equal(O.causal_attention(q, K2, V2)[:, :5], out[:, :5])
    # the last position sees every key: the decode attention of its query
    last = O.decode_attention(q[:, :, T - 1], K, V)
    np.testing.assert_allclose(out[:, T - 1].reshape(B, n_q, hd), last, rtol=1e-12, atol=1e-14)


def test_block_with_zero_output_projections_is_identity():
    # Eqs. attn_sublayer / mlp_sublayer add to the residual: with W_o = 0 and W_down = 0
    # both sub-layers add exactly zero.
    r = np.random.default_rng(5)
    B, T, d, n_q, n_kv, hd, dff = 2, 6, 16, 4, 2, 4, 24
    p = list(_block_params(d, n_q, n_kv, hd, dff, r))
    p[4] = np.zeros_like(p[4])
    p[8] = np.zeros_like(p[8])
    h = r.normal(0, 1, (B, T, d))
    pos = np.tile(np.arange(T), (B, 1))
    assert np.array_equal(O.block_forward(h, pos, *p, n_q, n_kv, hd, 1e-6, 1e4), h)


def test_block_brute_force_tiny():
    # The whole block written out with scalar loops (math.cos / math.sin RoPE on
    # consecutive pairs, explicit causal softmax, SiLU-gated MLP).
    r = np.random.default_rng(6)
    T, d, n_q, n_kv, hd, dff, eps, theta = 4, 6, 2, 1, 4, 5, 1e-6, 100.0
    ga, wq, wk, wv, wo, gm, wg, wu, wd = _block_params(d, n_q, n_kv, hd, dff, r)
    h = r.normal(0, 1, (1, T, d))
    pos = np.array([[3, 4, 5, 6]])
    got = O.block_forward(h, pos, ga, wq, wk, wv, wo, gm, wg, wu, wd, n_q, n_kv, hd, eps, theta)[0]

    def norm(x, g):
        ms = sum(v * v for v in x) / len(x)
        return [x[i] / math.sqrt(ms + eps) * g[i] for i in range(len(x))]

    def rope(v, p):
        o = list(v)
        for i in range(len(v) // 2):
            a = p * theta ** (-2.0 * i / len(v))
            o[2 * i] = v[2 * i] * math.cos(a) - v[2 * i + 1] * math.sin(a)
            o[2 * i + 1] = v[2 * i] * math.sin(a) + v[2 * i + 1] * math.cos(a)
        return o

    def mat(W, x, r0, n):
        return [sum(W[r0 + o, i] * x[i] for i in range(len(x))) for o in range(n)]

    x = [list(h[0, t]) for t in range(T)]
    xb = [norm(x[t], ga) for t in range(T)]
    Q = [[rope(mat(wq, xb[t], hh * hd, hd), pos[0, t]) for hh in range(n_q)] for t in range(T)]
    Kt = [rope(mat(wk, xb[t], 0, hd), pos[0, t]) for t in range(T)]
    Vt = [mat(wv, xb[t], 0, hd) for t in range(T)]
    for t in range(T):
        heads = []
        for hh in range(n_q):
            s = [sum(Q[t][hh][c] * Kt[j][c] for c in range(hd)) / math.sqrt(hd) for j in range(t + 1)]
            m = max(s)
            e = [math.exp(v - m) for v in s]
            z = sum(e)
            heads += [sum(e[j] / z * Vt[j][c] for j in range(t + 1)) for c in range(hd)]
        hhat = [x[t][o] + sum(wo[o, i] * heads[i] for i in range(n_q * hd)) for o in range(d)]
        hn = norm(hhat, gm)
        gu = [(mat(wg, hn, f, 1)[0], mat(wu, hn, f, 1)[0]) for f in range(dff)]
        act = [gv / (1.0 + math.exp(-gv)) * uv for gv, uv in gu]
        ref = [hhat[o] + sum(wd[o, f] * act[f] for f in range(dff)) for o in range(d)]
        np.testing.assert_allclose(got[t], ref, rtol=1e-12, atol=1e-12)


def test_recompute_residual_composes_blocks():
    r = np.random.default_rng(7)
    B, T, d, n_q, n_kv, hd, dff = 1, 5, 8, 2, 1, 4, 12
    layers = [_block_params(d, n_q, n_kv, hd, dff, r) for _ in range(3)]
    h0 = r.normal(0, 1, (B, T, d))
    pos = np.tile(np.arange(T), (B, 1))
    assert np.array_equal(O.recompute_residual(h0, pos, layers, 0, n_q, n_kv, hd, 1e-6, 1e4), h0)
    h2 = O.block_forward(O.block_forward(h0, pos, *layers[0], n_q, n_kv, hd, 1e-6, 1e4), pos, *layers[1],
                         n_q, n_kv, hd, 1e-6, 1e4)
    assert np.array_equal(O.recompute_residual(h0, pos, layers, 2, n_q, n_kv, hd, 1e-6, 1e4), h2)
