"""Oracle for the KV-cache transfer result (test infrastructure only).

Follows section 3.3 of FlowKV (arXiv 2504.03775): the KV cache of a request
lives in fixed-size physical blocks named by a per-request block-ID list
(PagedAttention's logical->physical mapping); the transfer moves the K and V
of every layer of the request from the sender's blocks to the receiver's
blocks, which the receiver names with its own block-ID list (Figure 3
caption).  Eq. 5 gives the two pool layouts:

* layer-major ``(L, 2, B, H)`` -- one tensor per layer holding K (index 0) and
  V (index 1) for all ``B`` blocks; each layer is its own buffer here, as
  per-layer paged tensors are allocated;
* block-major ``(B, L, 2, H)`` -- every layer's K and V of one block adjacent.

``H`` (the "remaining KV vector" of one block) is read as
``block_size * kv_heads * head_dim`` elements stored token-major, so one token
slot of one (block, layer, K-or-V) is ``slot_bytes = kv_heads * head_dim *
elem_bytes`` contiguous bytes.  The result is byte-exact and dtype-blind.

The result has a plain definition, written out here: for every logical token
slot ``t`` in ``[0, n * block_size)``, every layer ``l`` and ``kv`` in {K, V},

    dst[slot(D[t // bs], l, kv, t % bs)] = src[slot(S[t // bs], l, kv, t % bs)]

and every other destination byte keeps its old value.  Whole blocks move (the
paper transfers blocks), so the stale tail slots of a request's last, partly
filled block move too.

Parity: pinned by the tests in ``tests/test_oracle_copy.py`` -- unique tags
read back through numpy's own shaped-array indexing, layout equivalence via
numpy transposes, the single-memcpy special case, and the pure-Python loop
against the vectorised form.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Sequence

import numpy as np

LAYER_MAJOR = 0  # Eq. 5 left-hand side, (L, 2, B, H), one buffer per layer
BLOCK_MAJOR = 1  # Eq. 5 right-hand side, (B, L, 2, H), one buffer


@dataclass
class HostPool:
    """A paged KV pool held as raw bytes in host memory.

    ``buffers`` holds ``num_layers`` uint8 arrays of ``2 * num_blocks *
    block_size * slot_bytes`` bytes each (layer-major) or one uint8 array of
    ``num_blocks * num_layers * 2 * block_size * slot_bytes`` bytes
    (block-major).
    """

    layout: int
    num_layers: int
    num_blocks: int
    block_size: int
    slot_bytes: int
    buffers: List[np.ndarray] = field(default_factory=list)

    @classmethod
    def zeros(cls, layout, num_layers, num_blocks, block_size, slot_bytes):
        if layout == LAYER_MAJOR:
            per = 2 * num_blocks * block_size * slot_bytes
            bufs = [np.zeros(per, dtype=np.uint8) for _ in range(num_layers)]
        elif layout == BLOCK_MAJOR:
            tot = num_blocks * num_layers * 2 * block_size * slot_bytes
            bufs = [np.zeros(tot, dtype=np.uint8)]
        else:
            raise ValueError(f"unknown layout {layout}")
        return cls(layout, num_layers, num_blocks, block_size, slot_bytes, bufs)

    def copy(self) -> "HostPool":
        return HostPool(self.layout, self.num_layers, self.num_blocks,
                        self.block_size, self.slot_bytes,
                        [b.copy() for b in self.buffers])


def slot_address(pool: HostPool, b: int, l: int, kv: int, s: int):
    """Return ``(buffer index, byte offset)`` of token slot ``s`` of block ``b``,
    layer ``l``, K (``kv=0``) or V (``kv=1``), per Eq. 5's two layouts."""
    L, B, bs, sb = pool.num_layers, pool.num_blocks, pool.block_size, pool.slot_bytes
    if pool.layout == LAYER_MAJOR:
        # layer l's tensor is (2, B, bs, slot): K/V, then block, then slot
        return l, ((kv * B + b) * bs + s) * sb
    # one tensor (B, L, 2, bs, slot): block, then layer, then K/V, then slot
    return 0, (((b * L + l) * 2 + kv) * bs + s) * sb


def _check(src: HostPool, dst: HostPool, S: Sequence[int], D: Sequence[int]):
    if len(S) != len(D):
        raise ValueError("sender and receiver block lists differ in length")
    for a, b in ((src, dst),):
        if (a.num_layers, a.block_size, a.slot_bytes) != (b.num_layers, b.block_size, b.slot_bytes):
            raise ValueError("pools disagree on layers, block size or slot bytes")
    S = np.asarray(S, dtype=np.int64)
    D = np.asarray(D, dtype=np.int64)
    if S.size and (S.min() < 0 or S.max() >= src.num_blocks):
        raise ValueError("sender block ID out of range")
    if D.size and (D.min() < 0 or D.max() >= dst.num_blocks):
        raise ValueError("receiver block ID out of range")
    if len(np.unique(D)) != len(D):
        # two logical blocks written to one physical block: the result would
        # depend on write order, so the definition does not cover it
        raise ValueError("receiver block list repeats a block ID")
    return S, D


def _layer_range(pool: HostPool, layers):
    if layers is None:
        return range(pool.num_layers)
    layers = range(layers.start, layers.stop) if isinstance(layers, range) else layers
    for l in layers:
        if l < 0 or l >= pool.num_layers:
            raise ValueError(f"layer {l} outside the pool's {pool.num_layers} layers")
    return layers


def transfer_ref(src: HostPool, dst: HostPool, S: Sequence[int], D: Sequence[int],
                 layers=None) -> None:
    """The definition as a literal loop over (token slot, layer, K/V).

    ``layers`` restricts the copy to those layers (the layer-at-a-time
    transmission the paper's section 4.4 compares against); all by default.
    Pure Python: for small pools only (a few thousand slot copies)."""
    S, D = _check(src, dst, S, D)
    bs, sb = src.block_size, src.slot_bytes
    for t in range(len(S) * bs):
        for l in _layer_range(src, layers):
            for kv in (0, 1):
                si, so = slot_address(src, int(S[t // bs]), l, kv, t % bs)
                di, do = slot_address(dst, int(D[t // bs]), l, kv, t % bs)
                dst.buffers[di][do:do + sb] = src.buffers[si][so:so + sb]


def _slot_rows(pool: HostPool, blocks: np.ndarray, l: int, kv: int, slots: np.ndarray):
    """Vectorised ``slot_address`` divided by ``slot_bytes`` (row index of the
    slot when the buffer is viewed as ``(-1, slot_bytes)``)."""
    L, B, bs = pool.num_layers, pool.num_blocks, pool.block_size
    if pool.layout == LAYER_MAJOR:
        return l, (kv * B + blocks) * bs + slots
    return 0, ((blocks * L + l) * 2 + kv) * bs + slots


def transfer_fast(src: HostPool, dst: HostPool, S: Sequence[int], D: Sequence[int],
                  layers=None) -> None:
    """The same definition, vectorised over the token axis for each (layer,
    K/V) with numpy fancy indexing (one gather and one scatter per pair);
    ``layers`` as for ``transfer_ref``."""
    S, D = _check(src, dst, S, D)
    bs, sb = src.block_size, src.slot_bytes
    t = np.arange(len(S) * bs, dtype=np.int64)
    sblk, dblk, slot = S[t // bs], D[t // bs], t % bs
    for l in _layer_range(src, layers):
        for kv in (0, 1):
            si, srows = _slot_rows(src, sblk, l, kv, slot)
            di, drows = _slot_rows(dst, dblk, l, kv, slot)
            s2 = src.buffers[si].reshape(-1, sb)
            d2 = dst.buffers[di].reshape(-1, sb)
            d2[drows] = s2[srows]


def transfer_batch_fast(src: HostPool, dst: HostPool, tables) -> None:
    """Union of single-request transfers over ``tables = [(S_r, D_r), ...]``.

    Receiver IDs must be disjoint across requests (each physical block is
    written once); sender IDs may repeat across requests (shared prefix
    blocks are read twice)."""
    seen = set()
    for _, D in tables:
        for d in D:
            if int(d) in seen:
                raise ValueError("receiver block written by two requests")
            seen.add(int(d))
    for S, D in tables:
        transfer_fast(src, dst, S, D)
