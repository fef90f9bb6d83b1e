"""fp64 reference for KV-Direct's recompute-K/V + GQA decode attention.

TEST INFRASTRUCTURE ONLY (see the package docstring): nothing on the product
path may import this module.

Every function computes the plain definition from the paper, in float64, with
numpy; a matmul is the only library primitive used as a step.  Inputs are the
exact values the GPU sees (bf16 values upcast exactly), so differences against
the GPU measure only the GPU's arithmetic.

Conventions (readings of the paper, each listed in the design doc):

* RMSNorm (Sec. 3.1, Eqs. rmsnorm / rms_def): x / sqrt(mean(x^2) + eps) * gamma.
  The paper writes no epsilon; it is placed inside the square root.
* Weights are stored [out][in]: W_k holds the n_kv heads' d_head x d_model
  blocks stacked, i.e. the transpose of the paper's row-vector W_k^{(h)}
  (Eqs. k_proj / v_proj), so the projection is hbar @ W.T.
* RoPE (Sec. 3.2, Eqs. rope_cos / rope_sin) rotates consecutive pairs
  (2i, 2i+1) (0-based) by phi_i = p * theta^(-2i/d_head), i = 0 .. d_head/2-1,
  by +phi.  The paper's 1-based index literally gives theta^(-2i/d_head) for
  i = 1 .. d_head/2; the 0-based frequency follows RoFormer, which the paper
  cites.  This frequency index is a stated convention (parity unpinned: no
  printed value fixes it).
* Positions are 0-based absolute token indices.
* GQA: query head h reads KV head floor(h / g), g = n_q / n_kv.
* Attention (Eqs. attn_weights / head_output): softmax_j(q.K_j / sqrt(d_head))
  with explicit max subtraction, then the weighted sum of V_j.
* A decode step (Algorithm 1 at cache budget 0) attends over the recomputed
  context keys followed by the current token's own K/V, optionally with a block
  of stored (cached) K/V between them.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "rms_normalize",
    "rope_angles",
    "rope_matrix",
    "apply_rope",
    "project_heads",
    "recompute_kv",
    "project_qkv",
    "decode_attention",
    "kv_direct_decode",
    "window_start",
    "sliding_window_decode",
    "silu",
    "swiglu_mlp",
    "causal_attention",
    "block_forward",
    "recompute_residual",
]


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def rms_normalize(h, gamma, eps):
    """RMSNorm(h) over the last axis (Sec. 3.1, Eqs. rmsnorm and rms_def).

    hbar = h / ||h||_RMS * gamma with ||h||_RMS = sqrt(mean_i h_i^2 + eps).
    """
    h = _f64(h)
    gamma = _f64(gamma)
    ms = np.mean(h * h, axis=-1, keepdims=True)
    return h / np.sqrt(ms + float(eps)) * gamma


def rope_angles(pos, head_dim, theta):
    """phi[..., i] = p * theta^(-2i/d_head), i = 0 .. d_head/2 - 1 (Sec. 3.2)."""
    pos = _f64(pos)
    i = np.arange(head_dim // 2, dtype=np.float64)
    omega = np.power(float(theta), -2.0 * i / head_dim)
    return pos[..., None] * omega


def rope_matrix(p, head_dim, theta):
    """Dense R_p (Sec. 3.2, matrix form of Eqs. rope_cos / rope_sin).

    Block-diagonal with one 2x2 rotation [[cos, -sin], [sin, cos]] per
    consecutive pair.  Used by tests to cross-check apply_rope.
    """
    phi = rope_angles(np.asarray(p), head_dim, theta)
    R = np.zeros((head_dim, head_dim), dtype=np.float64)
    for i in range(head_dim // 2):
        c, s = math.cos(phi[i]), math.sin(phi[i])
        R[2 * i, 2 * i] = c
        R[2 * i, 2 * i + 1] = -s
        R[2 * i + 1, 2 * i] = s
        R[2 * i + 1, 2 * i + 1] = c
    return R


def apply_rope(x, pos, theta):
    """RoPE(x, p) on the last axis of x (length d_head), pairs (2i, 2i+1).

    x has shape [..., d_head] and pos broadcasts against x.shape[:-1].
    out_{2i}   = x_{2i} cos phi_i - x_{2i+1} sin phi_i
    out_{2i+1} = x_{2i} sin phi_i + x_{2i+1} cos phi_i
    """
    x = _f64(x)
    hd = x.shape[-1]
    phi = rope_angles(np.broadcast_to(_f64(pos), x.shape[:-1]), hd, theta)
    c, s = np.cos(phi), np.sin(phi)
    a, b = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = a * c - b * s
    out[..., 1::2] = a * s + b * c
    return out


def project_heads(hbar, W, n_heads, head_dim):
    """Per-head projection hbar W^{(h)} (Eqs. q_proj / k_proj / v_proj, before RoPE).

    hbar [..., d]; W [n_heads*head_dim, d] ([out][in]).  Returns
    [..., n_heads, head_dim].
    """
    W = _f64(W)
    assert W.shape[0] == n_heads * head_dim
    y = _f64(hbar) @ W.T
    return y.reshape(y.shape[:-1] + (n_heads, head_dim))


def recompute_kv(h, gamma, w_k, w_v, pos, n_kv, head_dim, eps, theta):
    """K/V reconstruction from residual checkpoints (Sec. 3.2, Eqs. k_recon / v_recon).

    h [B, T, d]; pos [B, T] absolute positions.
    K_p = R_p (RMSNorm(h_p) W_k), V_p = RMSNorm(h_p) W_v.
    Returns K, V of shape [B, n_kv, T, head_dim] (float64).
    """
    hbar = rms_normalize(h, gamma, eps)
    k = project_heads(hbar, w_k, n_kv, head_dim)              # [B, T, n_kv, hd]
    v = project_heads(hbar, w_v, n_kv, head_dim)
    k = apply_rope(k, _f64(pos)[..., None], theta)
    return k.transpose(0, 2, 1, 3).copy(), v.transpose(0, 2, 1, 3).copy()


def project_qkv(h_new, gamma, w_q, w_k, w_v, pos, n_q, n_kv, head_dim, eps, theta):
    """Current-token projections of a decode step (Algorithm 1; Eqs. q_proj..v_proj).

    h_new [B, d]; pos [B].  Q and K are rotated at the token's own position.
    Returns q [B, n_q, hd], k [B, n_kv, hd], v [B, n_kv, hd].
    """
    hbar = rms_normalize(h_new, gamma, eps)
    p = _f64(pos)[:, None]
    q = apply_rope(project_heads(hbar, w_q, n_q, head_dim), p, theta)
    k = apply_rope(project_heads(hbar, w_k, n_kv, head_dim), p, theta)
    v = project_heads(hbar, w_v, n_kv, head_dim)
    return q, k, v


def decode_attention(q, K, V):
    """One query per sequence and head over T keys (Eqs. attn_weights / head_output).

    q [B, n_q, hd]; K, V [B, n_kv, T, hd].  Query head h reads KV head
    floor(h / g).  alpha_j = softmax_j(q.K_j / sqrt(hd)) with the maximum
    subtracted before exponentiation; out = sum_j alpha_j V_j.
    """
    q, K, V = _f64(q), _f64(K), _f64(V)
    B, n_q, hd = q.shape
    n_kv = K.shape[1]
    g = n_q // n_kv
    out = np.empty((B, n_q, hd), dtype=np.float64)
    for b in range(B):
        for h in range(n_q):
            j = h // g
            s = K[b, j] @ q[b, h] / math.sqrt(hd)
            e = np.exp(s - np.max(s))
            alpha = e / np.sum(e)
            out[b, h] = alpha @ V[b, j]
    return out


def kv_direct_decode(q, h_ctx, gamma, w_k, w_v, pos_ctx, k_tail, v_tail,
                     n_kv, head_dim, eps, theta):
    """One KV-Direct decode step for one layer at cache budget 0 (Algorithm 1).

    RECOMPUTE_KV over the checkpointed context residuals h_ctx [B, T, d] at
    positions pos_ctx [B, T]; CONCAT with the stored tail K/V
    ([B, n_kv, T_tail, hd]: cached slots and/or the current token's own K_t,
    V_t); ATTENTION for the query q [B, n_q, hd].
    """
    K, V = recompute_kv(h_ctx, gamma, w_k, w_v, pos_ctx, n_kv, head_dim, eps, theta)
    if k_tail is not None:
        K = np.concatenate([K, _f64(k_tail)], axis=2)
        V = np.concatenate([V, _f64(v_tail)], axis=2)
    return decode_attention(q, K, V)


def window_start(n_keys, window):
    """Index w of the oldest key a sliding window of `window` keys keeps out of
    n_keys keys (the newest are kept): w = max(0, n_keys - window)."""
    if window < 1:
        raise ValueError("window must be >= 1")
    return max(0, n_keys - window)


def sliding_window_decode(h_new, h_ctx, gamma, w_q, w_k, w_v, window, n_q, n_kv, head_dim, eps, theta):
    """One decode step of a sliding-window layer (Sec. 3.2, the sliding-window
    boundary paragraph and Eq. sw_error; Sec. 5, the sliding-window limitation:
    window-relative rotation plus a local attention mask).

    The keys are the T checkpointed context rows h_ctx [B, T, d] followed by the
    current token h_new [B, d] (key T).  Only the newest `window` of these T + 1
    keys are attended (the local attention mask): keys j >= w = window_start(T + 1,
    window).  Each kept key is rotated by R_{j-w}, its index inside the window,
    instead of R_j, and the query by R_{T-w} (its own index in the window); V
    carries no rotation.  K and V are recomputed from the residuals of the kept
    rows exactly as in recompute_kv.
    """
    h_ctx, h_new = _f64(h_ctx), _f64(h_new)
    B, T, _ = h_ctx.shape
    w = window_start(T + 1, window)
    rows = np.concatenate([h_ctx[:, w:T], h_new[:, None, :]], axis=1)   # keys w .. T
    local = np.broadcast_to(np.arange(T + 1 - w, dtype=np.float64), (B, T + 1 - w))
    K, V = recompute_kv(rows, gamma, w_k, w_v, local, n_kv, head_dim, eps, theta)
    q, _, _ = project_qkv(h_new, gamma, w_q, w_k, w_v, np.full(B, float(T - w)), n_q, n_kv, head_dim, eps, theta)
    return decode_attention(q, K, V)


# ---------------------------------------------------------------- single-checkpoint scheme

def silu(x):
    """SiLU(x) = x * sigmoid(x) = x / (1 + e^-x)."""
    x = _f64(x)
    return x / (1.0 + np.exp(-x))


def swiglu_mlp(x, w_gate, w_up, w_down):
    """The MLP of Eq. mlp_sublayer.  The paper leaves its form open; the reading is
    the gated SiLU MLP of the LLaMA and Qwen families the paper evaluates:
    MLP(x) = (SiLU(x W_gate) * (x W_up)) W_down, weights stored [out][in]."""
    x = _f64(x)
    return (silu(x @ _f64(w_gate).T) * (x @ _f64(w_up).T)) @ _f64(w_down).T


def causal_attention(q, K, V):
    """Attention of every position over itself and the positions before it
    (Eqs. attn_weights / head_output with the decoder's causal order: position p
    attends keys j <= p).  q [B, n_q, T, hd]; K, V [B, n_kv, T, hd]; query head h
    reads KV head floor(h / g).  Returns [B, T, n_q * hd] (heads concatenated, the
    input of W_o in Eq. attn_sublayer)."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    B, n_q, T, hd = q.shape
    g = n_q // K.shape[1]
    out = np.empty((B, T, n_q * hd), dtype=np.float64)
    for b in range(B):
        for h in range(n_q):
            Kh, Vh = K[b, h // g], V[b, h // g]
            for p in range(T):
                s = Kh[:p + 1] @ q[b, h, p] / math.sqrt(hd)
                e = np.exp(s - np.max(s))
                out[b, p, h * hd:(h + 1) * hd] = (e / np.sum(e)) @ Vh[:p + 1]
    return out


def block_forward(h, pos, gamma_attn, w_q, w_k, w_v, w_o, gamma_mlp, w_gate, w_up, w_down,
                  n_q, n_kv, head_dim, eps, theta):
    """One pre-norm transformer block over all T positions of each sequence
    (Sec. 3.1, Eqs. q_proj .. mlp_sublayer): h [B, T, d] at positions pos [B, T]
    -> h^(l+1) [B, T, d].

    hbar = RMSNorm(h; gamma_attn); q, K, V per Eqs. q_proj / k_proj / v_proj (RoPE
    on q and K); heads by causal attention; hhat = h + [heads] W_o (Eq.
    attn_sublayer); h' = hhat + MLP(RMSNorm(hhat; gamma_mlp)) (Eq. mlp_sublayer).
    W_o is stored [d][n_q * head_dim]."""
    h = _f64(h)
    hbar = rms_normalize(h, gamma_attn, eps)
    q = apply_rope(project_heads(hbar, w_q, n_q, head_dim), _f64(pos)[..., None], theta)
    K, V = recompute_kv(h, gamma_attn, w_k, w_v, pos, n_kv, head_dim, eps, theta)
    heads = causal_attention(q.transpose(0, 2, 1, 3), K, V)
    hhat = h + heads @ _f64(w_o).T
    return hhat + swiglu_mlp(rms_normalize(hhat, gamma_mlp, eps), w_gate, w_up, w_down)


def recompute_residual(h0, pos, layers, n_layers, n_q, n_kv, head_dim, eps, theta):
    """The single-checkpoint scheme (Eq. res_mem: one residual vector per token
    serves every layer): h^(l) for l = n_layers, from the checkpoint h^(0) by
    running blocks 0 .. n_layers - 1 over all positions.  layers[i] holds block i's
    (gamma_attn, w_q, w_k, w_v, w_o, gamma_mlp, w_gate, w_up, w_down)."""
    h = _f64(h0)
    for i in range(n_layers):
        h = block_forward(h, pos, *layers[i], n_q, n_kv, head_dim, eps, theta)
    return h
