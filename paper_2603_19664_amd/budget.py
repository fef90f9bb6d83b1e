"""Algorithm 1's bounded cache (Sec. 3.4): the host bookkeeping of a decode loop
with cache budget B > 0 around libkvd's C-ABI calls.

Per layer, for a batch of sequences decoded in lockstep:

  ckpt   [batch][t_max][d]            residual checkpoints.  Row t is token t's
                                      residual h^(l) (position pos0[b] + t).  Rows
                                      0 .. T_rec-1 are the evicted tokens, which
                                      every step recomputes (RECOMPUTE_KV); rows
                                      T_rec .. T-1 belong to tokens still in the
                                      cache and wait there for their eviction.
  ring   K, V [batch][n_kv][B+1][hd]  the KV cache K[l] of B slots plus one slot
                                      for the token being decoded, used as a ring:
                                      the cached tokens sit in slots head,
                                      head + 1, ... (mod B + 1), oldest first.

One decode step (BoundedCache.step) issues, in Algorithm 1's order:
  1. kvd_store_residual: the current token's residual into ckpt row T (its
     h^(l) exists only now; STORE_RESIDUAL moves it into the recomputed range
     when it is evicted later);
  2. kvd_project_qkv: Q, K_t, V_t (Eqs. q_proj, k_proj, v_proj), K_t / V_t into
     the ring's free slot;
  3. kvd_fused_recompute_attn: RECOMPUTE_KV of ckpt rows 0 .. T_rec-1, CONCAT
     with the ring read from its oldest slot (the cache, then K_t / V_t), and
     ATTENTION, in one kernel;
  4. EVICT_OLDEST (host only): the current token has joined the cache; past
     the budget the oldest cached token leaves the ring (head advances) and its
     residual, already in ckpt row T_rec, joins the recomputed rows.

Memory per layer and sequence: (T - B) evicted residuals plus B cached K/V
entries (Eq. total_mem per layer), plus what Algorithm 1 holds beside them and
the equation leaves out: the current token's K_t / V_t (the ring's extra slot)
and the residuals of the B cached tokens, kept for their eviction.
"""
from __future__ import annotations

import dataclasses

from . import accounting


@dataclasses.dataclass
class RingState:
    """Indexes of Algorithm 1's cache for one layer (no device state).

    budget: cache slots B.  T: tokens decoded so far.  T_rec: evicted tokens
    (recomputed from checkpoints).  head: ring slot of the oldest cached token.
    n_cached: tokens in the cache (<= budget).  Invariant: T = T_rec + n_cached.
    """
    budget: int
    T: int = 0
    T_rec: int = 0
    head: int = 0
    n_cached: int = 0

    def __post_init__(self):
        if self.budget < 0:
            raise ValueError("budget must be >= 0")

    @property
    def slots(self) -> int:
        return self.budget + 1

    def free_slot(self) -> int:
        """Ring slot that receives the current token's K_t / V_t."""
        return (self.head + self.n_cached) % self.slots

    def tail_rows(self) -> int:
        """Rows the step attends from the ring: the cache, then the current token."""
        return self.n_cached + 1

    def slot_of(self, t: int) -> int:
        """Ring slot of cached token t (T_rec <= t < T_rec + n_cached), or of the current token t = T."""
        if not self.T_rec <= t <= self.T:
            raise ValueError(f"token {t} is not in the cache")
        return (self.head + (t - self.T_rec)) % self.slots

    def keys_in_order(self) -> list:
        """Tokens the step attends, in CONCAT order: recomputed, cached (oldest first), current."""
        return list(range(self.T_rec)) + [self.T_rec + i for i in range(self.n_cached)] + [self.T]

    def advance(self):
        """After the step's attention: the current token joins the cache; past the budget
        EVICT_OLDEST drops the oldest cached token, whose residual joins the recomputed rows."""
        self.T += 1
        self.n_cached += 1
        if self.n_cached > self.budget:
            self.head = (self.head + 1) % self.slots
            self.n_cached -= 1
            self.T_rec += 1

    def memory_bytes(self, d: int, n_kv: int, hd: int, b: int) -> dict:
        """Per layer and sequence: Eq. total_mem at the current T and budget, and what this
        cache holds (evicted residuals, retained residuals of cached tokens, ring slots)."""
        eq = accounting.total_memory(self.T, min(self.budget, self.T), 1, n_kv, hd, d, b)
        held = {"evicted_residuals": self.T_rec * d * b, "retained_residuals": self.n_cached * d * b,
                "ring_kv": self.slots * 2 * n_kv * hd * b}
        held["total"] = sum(held.values())
        return {"eq_total_mem": eq, "held": held}


class BoundedCache:
    """One layer's Algorithm 1 state on the GPU for `batch` sequences, `budget` cache slots and
    room for t_max tokens; step() runs one decode step through the C ABI (see module doc)."""

    def __init__(self, shape, batch: int, budget: int, t_max: int, pos0, device="cuda"):
        import torch

        from . import kvd
        self.kvd, self.torch = kvd, torch
        self.shape, self.B = shape, batch
        self.state = RingState(budget)
        dt = shape.torch_dtype
        self.t_max = t_max
        self.ckpt = torch.zeros((batch, t_max, shape.d_model), dtype=dt, device=device)
        self.ring_k = torch.zeros((batch, shape.n_kv_heads, budget + 1, shape.head_dim), dtype=dt, device=device)
        self.ring_v = torch.zeros_like(self.ring_k)
        self.pos0 = pos0
        self.q = torch.empty((batch, shape.n_q_heads, shape.head_dim), dtype=dt, device=device)
        # one workspace for every step: sized for the largest call (all t_max tokens recomputed or cached)
        ws_bytes = max(kvd.kvd_workspace_bytes(shape, kvd.KVD_OP_FUSED, batch, t_rec, budget + 1)
                       for t_rec in (0, max(t_max - 1, 0), max(t_max - budget - 1, 0)))
        ws_bytes = max(ws_bytes, kvd.kvd_workspace_bytes(shape, kvd.KVD_OP_FUSED, batch, t_max, 1))
        self.ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device=device)

    def step(self, h_new, gamma, w_q, w_k, w_v, out):
        """Decode one token per sequence: h_new [batch, d] is its residual h^(l); out [batch, n_q, hd]."""
        kvd, st = self.kvd, self.state
        if st.T >= self.t_max:
            raise ValueError(f"the checkpoint store holds {self.t_max} tokens")
        pos = (self.pos0 + st.T).to(self.torch.int32)
        kvd.kvd_store_residual(self.shape, h_new, self.ckpt, st.T)                              # STORE_RESIDUAL
        kvd.kvd_project_qkv(self.shape, h_new, gamma, w_q, w_k, w_v, pos, self.q, self.ring_k, self.ring_v,
                            st.free_slot())                                                      # Q, K_t, V_t
        kvd.kvd_fused_recompute_attn(self.shape, self.q, self.ckpt, st.T_rec, gamma, w_k, w_v, self.pos0, out,
                                     self.ws, self.ring_k, self.ring_v, st.tail_rows(), st.head)  # RECOMPUTE+ATTN
        st.advance()                                                                             # EVICT_OLDEST
        return self.q
