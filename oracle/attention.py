"""Oracle for decode attention over a paged KV pool (test infrastructure only).

FlowKV (arXiv 2504.03775) changes the KV pool's layout to the block-major
(B, L, 2, H) of Eq. 5 and adapts the PagedAttention kernel to it (section
3.3).  The decode step it serves is the paper's Eq. 2: each new token's query
attends to the request's K and V of every earlier token, layer by layer.
The paper does not restate attention itself; this is the standard scaled
dot-product attention with grouped KV heads (Llama-3's layout: ``Hq`` query
heads share ``Hkv`` KV heads, query head ``h`` reading KV head
``h // (Hq / Hkv)``), written out plainly in float64:

    s_t   = scale * sum_d q[h, d] * K[t, g, d]          for t < T
    p_t   = exp(s_t - max_t s_t) / sum_t exp(s_t - max_t s_t)
    o[h]  = sum_t p_t * V[t, g, :]

K[t] and V[t] of token ``t`` are read from the pool through the request's
block list: block ``table[t // bs]``, slot ``t % bs``, with the slot address
of ``oracle.kvcopy.slot_address`` (both Eq. 5 layouts).

Parity: pinned in ``tests/test_oracle_attention.py`` -- one token returns its
V exactly, equal scores average V, a query that singles out one key returns
that key's V, with a constant V per KV head every query head returns its
group's constant, agreement with a separate dense softmax-attention computed
from numpy's einsum on a contiguous copy, and invariance under relabelling
the pool's blocks.

``decode_attention_scales`` returns, next to each output element, the sizes
its rounding errors scale with in any float32 evaluation of the same sums
(test infrastructure for setting tolerances; see its docstring).
"""

from __future__ import annotations

from typing import Sequence

import numpy as np

from .kvcopy import HostPool, slot_address


def _bf16_bytes_to_f64(raw: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (little-endian uint16) to float64, exactly."""
    u16 = raw.view(np.uint16).astype(np.uint32)
    return (u16 << 16).view(np.float32).astype(np.float64)


def gather_kv(pool: HostPool, table: Sequence[int], T: int, layer: int, kv_heads: int,
              head_dim: int, elem: str = "bf16") -> np.ndarray:
    """K (kv=0) and V (kv=1) of tokens 0..T-1 of one layer as float64 arrays
    shaped (2, T, kv_heads, head_dim), read slot by slot from the pool."""
    if elem != "bf16":
        raise ValueError("the oracle reads bfloat16 pools")
    bs = pool.block_size
    if T > len(table) * bs:
        raise ValueError("sequence longer than its block list")
    if pool.slot_bytes != kv_heads * head_dim * 2:
        raise ValueError("slot size does not match kv_heads * head_dim bf16 values")
    out = np.zeros((2, T, kv_heads, head_dim), dtype=np.float64)
    for t in range(T):
        for kv in (0, 1):
            bi, off = slot_address(pool, int(table[t // bs]), layer, kv, t % bs)
            raw = pool.buffers[bi][off:off + pool.slot_bytes]
            out[kv, t] = _bf16_bytes_to_f64(raw).reshape(kv_heads, head_dim)
    return out


def _weights(K: np.ndarray, qh: np.ndarray, scale: float):
    """Scores s_t = scale * q . K_t and softmax weights p_t over tokens."""
    s = scale * (K @ qh)
    p = np.exp(s - s.max())
    return s, p / p.sum()


def decode_attention_scales(pool: HostPool, q: np.ndarray, tables, seq_lens, layer: int,
                            kv_heads: int, head_dim: int, scale: float):
    """decode_attention plus, per output element (r, h, d), the quantities its
    rounding errors scale with (float64):

      out  the attention output o[r, h, d] (as decode_attention);
      w1   sum_t p_t |V_t,d|: bounds every partial sum of p_t V_t,d, so an
           error of relative size e in each addition of those sums moves
           o by at most about e * w1 per addition;
      w2   sqrt(sum_t p_t^2 (V_t,d - o_d)^2): independent relative errors
           delta_t in the weights move o by sum_t p_t delta_t (V_t,d - o_d),
           whose spread is |delta| * w2;
      s1   per (r, h): scale * max_t sum_d |q_d K_t,d|, the largest sum of
           absolute products in a score, which bounds a score's rounding
           error relative to the number of its roundings."""
    q = np.asarray(q, dtype=np.float64)
    n, Hq, D = q.shape
    if D != head_dim or Hq % kv_heads:
        raise ValueError("query shape does not match the pool's heads")
    group = Hq // kv_heads
    out = np.zeros((n, Hq, D))
    w1 = np.zeros((n, Hq, D))
    w2 = np.zeros((n, Hq, D))
    s1 = np.zeros((n, Hq))
    for r in range(n):
        T = int(seq_lens[r])
        if T < 1:
            raise ValueError("a request needs at least one token")
        kvr = gather_kv(pool, tables[r], T, layer, kv_heads, head_dim)
        K, V = kvr[0], kvr[1]
        for h in range(Hq):
            g = h // group
            _, p = _weights(K[:, g, :], q[r, h], scale)
            o = p @ V[:, g, :]
            out[r, h] = o
            w1[r, h] = p @ np.abs(V[:, g, :])
            w2[r, h] = np.sqrt((p ** 2) @ (V[:, g, :] - o) ** 2)
            s1[r, h] = scale * np.max(np.abs(K[:, g, :]) @ np.abs(q[r, h]))
    return out, w1, w2, s1


def decode_attention(pool: HostPool, q: np.ndarray, tables, seq_lens, layer: int,
                     kv_heads: int, head_dim: int, scale: float) -> np.ndarray:
    """Decode attention of ``n`` requests, float64.

    q: (n, Hq, head_dim) float array (the query values, already rounded to
    whatever precision the caller feeds the kernel); tables[r]: request r's
    block list; seq_lens[r]: its token count T_r >= 1.  Returns (n, Hq,
    head_dim) float64."""
    q = np.asarray(q, dtype=np.float64)
    n, Hq, D = q.shape
    if D != head_dim or Hq % kv_heads:
        raise ValueError("query shape does not match the pool's heads")
    group = Hq // kv_heads
    out = np.zeros((n, Hq, D), dtype=np.float64)
    for r in range(n):
        T = int(seq_lens[r])
        if T < 1:
            raise ValueError("a request needs at least one token")
        kvr = gather_kv(pool, tables[r], T, layer, kv_heads, head_dim)
        K, V = kvr[0], kvr[1]
        for h in range(Hq):
            g = h // group
            _, p = _weights(K[:, g, :], q[r, h], scale)
            out[r, h] = p @ V[:, g, :]
    return out
