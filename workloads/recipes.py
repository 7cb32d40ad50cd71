"""The five transfer workloads, built from seeded inputs.

Each recipe takes ``make_alloc(num_blocks, policy, seed)`` -- the product
allocator or the oracle's, whichever the caller is testing -- and returns the
per-request sender/receiver block lists plus the pool sizes the device needs.
The allocation itself happens inside the object ``make_alloc`` returns; this
module only decides which inputs (pool sizes, occupancy, lengths, op streams,
seeds) go in.

Workloads:
  tiny      2 layers, 2 KV heads, head_dim 64, fp16, block 16; one 256-token
            request in a 64-block pool, both lists seeded permutations.
  8b        Llama-3-8B KV shape (32 layers, 8 KV heads, head_dim 128, bf16,
            block 16); one 13,000-token request; 65,536-block pools; the
            sender's list from the segment allocator on a fresh pool, the
            receiver's from a free list over a pool with 30% of blocks
            occupied at random.
  batch     8B shape, 32 requests of U[2,000, 20,000] tokens, 200,000-ID
            allocators on both sides (segment policy or shuffled free list);
            IDs relabelled gap-preservingly so the device pools fit.
  70b       Llama-3-70B share under 8-way tensor parallelism (80 layers, 1 KV
            head, head_dim 128, bf16, block 16); 16 requests of 32,000 tokens;
            each pool 30% of 288 GB.
  churn     8B shape; 10,000 seeded alloc/free operations with lognormal
            lengths (median 4,000, sigma 0.8, cap 32,000) leave 128 live
            requests; the receiver pool starts 10% occupied.  Worst cases:
            both sides shuffled free lists, or stride-2 lists where every
            block is its own run.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, List, Tuple

import numpy as np

from . import (LLAMA3_70B_TP8, LLAMA3_8B, SEED_DST_TABLE, SEED_LENGTHS, SEED_OCCUPANCY,
               SEED_SRC_TABLE, TINY, Geometry, blocks_for, churn_ops, compact_ids,
               occupied_blocks, random_table, replay, uniform_lengths)

POLICY_SEGMENT, POLICY_FIFO_SORTED, POLICY_FIFO_SHUFFLED = 0, 1, 2
POLICIES = {"segment": POLICY_SEGMENT, "fifo_sorted": POLICY_FIFO_SORTED,
            "fifo_shuffled": POLICY_FIFO_SHUFFLED}

HBM_BYTES_MI355X = 288e9  # decimal, as the product is specified

MakeAlloc = Callable[[int, int, int], object]


@dataclass
class Workload:
    name: str
    geom: Geometry
    src_pool_blocks: int
    dst_pool_blocks: int
    tables: List[Tuple[np.ndarray, np.ndarray]] = field(default_factory=list)
    tokens: List[int] = field(default_factory=list)
    note: str = ""

    @property
    def n_blocks(self) -> int:
        return int(sum(len(s) for s, _ in self.tables))

    @property
    def payload_bytes(self) -> int:
        return self.n_blocks * self.geom.block_bytes

    def offsets(self) -> np.ndarray:
        return np.concatenate(([0], np.cumsum([len(s) for s, _ in self.tables]))).astype(np.int64)

    def flat(self) -> Tuple[np.ndarray, np.ndarray]:
        if not self.tables:
            return np.zeros(0, np.int32), np.zeros(0, np.int32)
        return (np.concatenate([s for s, _ in self.tables]).astype(np.int32),
                np.concatenate([d for _, d in self.tables]).astype(np.int32))


def tiny() -> Workload:
    g = TINY
    n = blocks_for(256, g.block_size)
    S = random_table(64, n, SEED_SRC_TABLE)
    D = random_table(64, n, SEED_DST_TABLE)
    return Workload("tiny", g, 64, 64, [(S, D)], [256], "seeded permutations, 16 blocks")


def llama8b_13k(make_alloc: MakeAlloc, dst_policy: str = "fifo_sorted",
                pool_blocks: int = 65_536, tokens: int = 13_000,
                dst_pool_blocks: int = 0, occupied: float = 0.30) -> Workload:
    """dst_pool_blocks (0: the same as pool_blocks) shrinks the receiver's
    pool where a device cannot hold two full ones; `occupied` is the
    fraction of its blocks held at random before the request arrives."""
    g = LLAMA3_8B
    n = blocks_for(tokens, g.block_size)
    dst_blocks = dst_pool_blocks or pool_blocks
    src = make_alloc(pool_blocks, POLICY_SEGMENT, SEED_SRC_TABLE)
    S = np.asarray(src.alloc(n), dtype=np.int32)
    dst = make_alloc(dst_blocks, POLICIES[dst_policy], SEED_DST_TABLE)
    dst.mark_used(occupied_blocks(dst_blocks, occupied, SEED_OCCUPANCY))
    D = np.asarray(dst.alloc(n), dtype=np.int32)
    return Workload(f"llama3-8b-13k/{dst_policy}", g, pool_blocks, dst_blocks, [(S, D)],
                    [tokens], f"receiver pool of {dst_blocks} blocks {occupied:.0%} occupied, "
                              f"receiver policy {dst_policy}")


def batch32(make_alloc: MakeAlloc, policy: str = "segment", id_space: int = 200_000,
            n_req: int = 32) -> Workload:
    g = LLAMA3_8B
    lengths = uniform_lengths(n_req, 2_000, 20_000, SEED_LENGTHS)
    src = make_alloc(id_space, POLICIES[policy], SEED_SRC_TABLE)
    dst = make_alloc(id_space, POLICIES[policy], SEED_DST_TABLE)
    Ss, Ds = [], []
    for T in lengths:
        n = blocks_for(int(T), g.block_size)
        Ss.append(np.asarray(src.alloc(n), dtype=np.int32))
        Ds.append(np.asarray(dst.alloc(n), dtype=np.int32))
    Ss, src_blocks = compact_ids(Ss)
    Ds, dst_blocks = compact_ids(Ds)
    return Workload(f"batch32/{policy}", g, src_blocks, dst_blocks, list(zip(Ss, Ds)),
                    [int(t) for t in lengths],
                    f"{id_space}-ID allocators, {policy}; IDs relabelled gap-preservingly")


def llama70b_tp8(make_alloc: MakeAlloc, policy: str = "segment", n_req: int = 16,
                 tokens: int = 32_000) -> Workload:
    g = LLAMA3_70B_TP8
    pool_blocks = int(0.6 * HBM_BYTES_MI355X / 2 // g.block_bytes)
    src = make_alloc(pool_blocks, POLICIES[policy], SEED_SRC_TABLE)
    dst = make_alloc(pool_blocks, POLICIES[policy], SEED_DST_TABLE)
    n = blocks_for(tokens, g.block_size)
    tables = [(np.asarray(src.alloc(n), dtype=np.int32), np.asarray(dst.alloc(n), dtype=np.int32))
              for _ in range(n_req)]
    return Workload(f"llama3-70b-tp8/{policy}", g, pool_blocks, pool_blocks, tables,
                    [tokens] * n_req, f"pools 30% of 288 GB each, {policy}")


def churn(make_alloc: MakeAlloc, variant: str = "segment", pool_blocks: int = 65_536) -> Workload:
    """variant: 'segment' (both sides segment allocator, receiver 10% occupied),
    'shuffled' (both sides shuffled free lists), 'stride2' (S[i]=2i, D[i]=2i+1
    over the first pool_blocks/2 blocks of the segment run's requests)."""
    g = LLAMA3_8B
    ops = churn_ops()
    if variant == "stride2":
        n = pool_blocks // 2
        S = (2 * np.arange(n)).astype(np.int32)
        D = (2 * np.arange(n) + 1).astype(np.int32)
        return Workload("churn/stride2", g, pool_blocks, pool_blocks, [(S, D)],
                        [n * g.block_size], "every block its own run")
    policy = POLICY_SEGMENT if variant == "segment" else POLICY_FIFO_SHUFFLED
    src = make_alloc(pool_blocks, policy, SEED_SRC_TABLE)
    dst = make_alloc(pool_blocks, policy, SEED_DST_TABLE)
    dst.mark_used(occupied_blocks(pool_blocks, 0.10, SEED_OCCUPANCY))
    live_s = replay(ops, src, g.block_size)
    live_d = replay(ops, dst, g.block_size)
    assert list(live_s) == list(live_d)
    tokens = {rid: t for kind, rid, t in ops if kind == "alloc"}
    tables = [(live_s[r], live_d[r]) for r in live_s]
    return Workload(f"churn/{variant}", g, pool_blocks, pool_blocks, tables,
                    [tokens[r] for r in live_s], f"10,000 ops, 128 live, {variant}")
