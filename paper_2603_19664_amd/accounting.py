"""Closed-form memory and work accounting (Section 3.4 of the paper).

Per-token memory (Eqs. kv_mem, res_mem, compression_ratio), recompute cost
(Eq. recomp_flops), cache-read traffic (Eq. read_bytes) and the bounded
total (Eq. total_mem), plus the algorithmic flop/byte counts of each kernel
that the roofline figures divide by.
"""
from __future__ import annotations


def kv_bytes_per_token(L: int, n_kv: int, head_dim: int, b: int) -> int:
    """Eq. kv_mem: 2 L n_kv d_head b bytes of KV cache per token."""
    return 2 * L * n_kv * head_dim * b


def residual_bytes_per_token(d_hidden: int, b: int) -> int:
    """Eq. res_mem: one residual vector of d_hidden elements per token."""
    return d_hidden * b


def compression_ratio(L: int, n_kv: int, head_dim: int, d_hidden: int) -> float:
    """Eq. compression_ratio: rho = 2 L n_kv d_head / d_hidden."""
    return 2.0 * L * n_kv * head_dim / d_hidden


def recompute_flops(N: int, n_kv: int, d_hidden: int, head_dim: int) -> int:
    """Eq. recomp_flops: 4 N n_kv d_hidden d_head (K and V projections)."""
    return 4 * N * n_kv * d_hidden * head_dim


def read_bytes(N: int, n_kv: int, head_dim: int, b: int) -> int:
    """Eq. read_bytes: 2 N n_kv d_head b bytes to read N cached K/V entries."""
    return 2 * N * n_kv * head_dim * b


def total_memory(T: int, budget: int, L: int, n_kv: int, head_dim: int, d_hidden: int, b: int) -> int:
    """Eq. total_mem: budget cached entries per layer plus (T - budget) shared residuals."""
    return 2 * budget * L * n_kv * head_dim * b + (T - budget) * d_hidden * b


# --- per-launch algorithmic work of the library's kernels -------------------

def attention_flops(B: int, T: int, n_q: int, head_dim: int) -> int:
    """q.K and alpha.V for one decode query per head over T keys: 4 B T n_q d_head."""
    return 4 * B * T * n_q * head_dim


def fused_flops(B: int, T_rec: int, T_tail: int, n_q: int, n_kv: int, d: int, head_dim: int) -> int:
    """Fused recompute + attention: Eq. recomp_flops over the recomputed keys plus attention."""
    return recompute_flops(B * T_rec, n_kv, d, head_dim) + attention_flops(B, T_rec + T_tail, n_q, head_dim)


def fused_bytes(B: int, T_rec: int, T_tail: int, n_q: int, n_kv: int, d: int, head_dim: int,
                b: int, n_splits: int) -> int:
    """Compulsory HBM bytes of one fused launch: residuals, gamma, W_k/W_v, q, tail K/V, fp32 partials."""
    return (B * T_rec * d * b + d * b + 2 * n_kv * head_dim * d * b + B * n_q * head_dim * b
            + read_bytes(B * T_tail, n_kv, head_dim, b) + B * n_q * n_splits * (head_dim + 2) * 4)


def cached_bytes(B: int, T: int, n_q: int, n_kv: int, head_dim: int, b: int, n_splits: int) -> int:
    """Compulsory HBM bytes of one cached-attention partial launch: K/V (Eq. read_bytes), q, partials."""
    return read_bytes(B * T, n_kv, head_dim, b) + B * n_q * head_dim * b + B * n_q * n_splits * (head_dim + 2) * 4
