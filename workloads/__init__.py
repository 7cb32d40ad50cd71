"""Seeded synthetic inputs for the KV-cache transfer workloads.

Shared by the tests and the benchmark on both sides of every parity check
(the HIP path and the CPU oracle).  It holds no step of the method: no
allocation policy, no alignment, no copy.  It produces only the raw inputs
those steps consume -- pool geometries, seeded random block lists,
pre-occupied block sets, request lengths, alloc/free operation streams and
the K/V data -- plus ``replay``, which feeds an operation stream to whatever
allocator object it is given.

The shapes follow the paper's workloads (FlowKV, arXiv 2504.03775): the
Llama-3.1-8B and -70B KV geometries of section 4.1 and the 13k-token request
of Figure 1.  The paper's real-world requests come from LongBench, which is
not used here: synthetic lengths and N(0, 1) K/V data of the same shapes stand
in for it.  Random numbers come from numpy's PCG64 (tables, lengths, ops) and
torch's device generator (K/V data), each from a fixed seed.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Sequence, Tuple

import numpy as np

# seed roles (base 0)
SEED_DATA = 0
SEED_DATA_DST = 1
SEED_SRC_TABLE = 2
SEED_DST_TABLE = 3
SEED_OCCUPANCY = 4
SEED_LENGTHS = 5
SEED_OPS = 6
SEED_SAMPLE = 7


@dataclass(frozen=True)
class Geometry:
    """KV geometry of one model (or one tensor-parallel share of it)."""

    name: str
    num_layers: int
    kv_heads: int
    head_dim: int
    block_size: int
    dtype: str  # "float16" or "bfloat16"

    @property
    def elem_bytes(self) -> int:
        return 2

    @property
    def slot_bytes(self) -> int:  # one token of one (layer, K-or-V)
        return self.kv_heads * self.head_dim * self.elem_bytes

    @property
    def chunk_bytes(self) -> int:  # one (block, layer, K-or-V)
        return self.block_size * self.slot_bytes

    @property
    def block_bytes(self) -> int:  # one block, all layers, K and V
        return 2 * self.num_layers * self.chunk_bytes

    @property
    def token_bytes(self) -> int:
        return 2 * self.num_layers * self.slot_bytes


TINY = Geometry("tiny", 2, 2, 64, 16, "float16")
LLAMA3_8B = Geometry("llama3-8b", 32, 8, 128, 16, "bfloat16")
LLAMA3_70B_TP8 = Geometry("llama3-70b-tp8-share", 80, 1, 128, 16, "bfloat16")


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def blocks_for(tokens: int, block_size: int) -> int:
    return -(-tokens // block_size)


def random_table(pool_blocks: int, n: int, seed: int) -> np.ndarray:
    """n distinct block IDs: the head of a seeded permutation of the pool."""
    return rng(seed).permutation(pool_blocks)[:n].astype(np.int32)


def occupied_blocks(pool_blocks: int, fraction: float, seed: int) -> np.ndarray:
    """round(fraction * pool) distinct block IDs chosen uniformly, ascending."""
    k = int(round(fraction * pool_blocks))
    return np.sort(rng(seed).choice(pool_blocks, size=k, replace=False)).astype(np.int32)


def uniform_lengths(n: int, lo: int, hi: int, seed: int) -> np.ndarray:
    """n request lengths in tokens, uniform on the integers [lo, hi]."""
    return rng(seed).integers(lo, hi + 1, size=n).astype(np.int64)


def lognormal_length(g: np.random.Generator, median: float, sigma: float, cap: int) -> int:
    return int(min(cap, max(1, round(float(g.lognormal(math.log(median), sigma))))))


def churn_ops(n_ops: int = 10_000, live: int = 128, median: float = 4_000.0,
              sigma: float = 0.8, cap: int = 32_000, seed_lengths: int = SEED_LENGTHS,
              seed_ops: int = SEED_OPS) -> List[Tuple[str, int, int]]:
    """Alloc/free stream: `live` allocations, then (free a uniformly chosen
    live request, allocate a new one) pairs until n_ops operations, ending with
    exactly `live` requests alive.  Items are ('alloc', rid, tokens) or
    ('free', rid, 0)."""
    if (n_ops - live) % 2:
        raise ValueError("n_ops - live must be even")
    gl, go = rng(seed_lengths), rng(seed_ops)
    ops: List[Tuple[str, int, int]] = []
    alive: List[int] = []
    rid = 0
    for _ in range(live):
        ops.append(("alloc", rid, lognormal_length(gl, median, sigma, cap)))
        alive.append(rid)
        rid += 1
    for _ in range((n_ops - live) // 2):
        victim = alive.pop(int(go.integers(len(alive))))
        ops.append(("free", victim, 0))
        ops.append(("alloc", rid, lognormal_length(gl, median, sigma, cap)))
        alive.append(rid)
        rid += 1
    return ops


def replay(ops, allocator, block_size: int) -> Dict[int, np.ndarray]:
    """Run an op stream against any object with alloc(n) and free(ids);
    returns the live requests' block lists keyed by request id (in order of
    allocation)."""
    live: Dict[int, np.ndarray] = {}
    for kind, rid, tokens in ops:
        if kind == "alloc":
            live[rid] = np.asarray(allocator.alloc(blocks_for(tokens, block_size)), dtype=np.int32)
        else:
            allocator.free(live.pop(rid))
    return live


def compact_ids(tables: Sequence[np.ndarray]) -> Tuple[List[np.ndarray], int]:
    """Relabel block IDs into a dense space with every adjacency kept: sort the
    distinct IDs used; each gets prev + 1 if it was adjacent to the previous
    used ID, else prev + 2.  Two IDs are consecutive after relabelling iff
    they were before, so every block list keeps its runs.  Returns the
    relabelled tables and the size of the new ID space."""
    used = np.unique(np.concatenate([np.asarray(t, dtype=np.int64) for t in tables])
                     if len(tables) else np.zeros(0, dtype=np.int64))
    if used.size == 0:
        return [np.asarray(t, dtype=np.int32) for t in tables], 1
    step = np.where(np.diff(used) == 1, 1, 2)
    new = np.concatenate(([0], np.cumsum(step)))
    lut = dict(zip(used.tolist(), new.tolist()))
    out = [np.asarray([lut[int(b)] for b in t], dtype=np.int32) for t in tables]
    return out, int(new[-1]) + 1


def sample_indices(n: int, k: int, seed: int) -> np.ndarray:
    """min(n, k) distinct indices of [0, n), ascending, seeded."""
    if k >= n:
        return np.arange(n, dtype=np.int64)
    return np.sort(rng(seed).choice(n, size=k, replace=False)).astype(np.int64)


# ---- device data (torch only as a source of seeded device memory) ----------

def torch_dtype(geom: Geometry):
    import torch
    return {"float16": torch.float16, "bfloat16": torch.bfloat16}[geom.dtype]


def fill_normal_(tensors, seed: int, chunk_elems: int = 1 << 28) -> None:
    """Fill device tensors with N(0, 1) values (fp32 draws cast to the tensor
    dtype), chunk by chunk from a generator seeded with `seed`."""
    import torch

    for t in tensors:
        flat = t.view(-1)
        g = torch.Generator(device=t.device)
        g.manual_seed(seed)
        for lo in range(0, flat.numel(), chunk_elems):
            hi = min(flat.numel(), lo + chunk_elems)
            flat[lo:hi].copy_(torch.randn(hi - lo, generator=g, device=t.device,
                                          dtype=torch.float32))
        seed += 1


def make_device_pool(geom: Geometry, layout: int, num_blocks: int, device, seed=None):
    """Allocate a pool's tensors (layout 0: L tensors (2, B, bs, Hkv, Dh);
    layout 1: one tensor (B, L, 2, bs, Hkv, Dh)); N(0, 1) data if seeded."""
    import torch

    dt = torch_dtype(geom)
    shape_slot = (geom.block_size, geom.kv_heads, geom.head_dim)
    if layout == 1:
        ts = [torch.empty((num_blocks, geom.num_layers, 2) + shape_slot, dtype=dt, device=device)]
    else:
        ts = [torch.empty((2, num_blocks) + shape_slot, dtype=dt, device=device)
              for _ in range(geom.num_layers)]
    if seed is not None:
        fill_normal_(ts, seed)
    return ts


def pool_bytes(geom: Geometry, num_blocks: int) -> int:
    return num_blocks * geom.block_bytes
