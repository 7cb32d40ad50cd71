"""Shared plumbing for the GPU parity tests: pools on the device, downloads
into the oracle's host pools, and the comparison used at full size.

Expected values always come from ``oracle`` run on host copies of device
memory that the transfer kernel has not touched yet (the seeded source pool
and the receiver's pre-image)."""

from __future__ import annotations

import gc

import numpy as np
import torch

import oracle
from paper_2504_03775_amd import flowkv as fk
from workloads import make_device_pool, pool_bytes, sample_indices

LM, BM = fk.LAYOUT_LAYER_MAJOR, fk.LAYOUT_BLOCK_MAJOR


def device_pool(geom, layout, num_blocks, seed):
    ts = make_device_pool(geom, layout, num_blocks, "cuda", seed)
    return fk.KVPool(layout, ts)


def download_blocks(pool: fk.KVPool, ids) -> oracle.HostPool:
    """Blocks `ids` of a device pool as a compact oracle pool of len(ids) blocks
    (block i of the result = block ids[i] of the device pool), same layout."""
    idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device=pool.device)
    slot = pool.kv_heads * pool.head_dim * pool.elem_bytes
    hp = oracle.HostPool.zeros(pool.layout, pool.num_layers, len(ids), pool.block_size, slot)
    if len(ids) == 0:
        return hp
    # in pieces of at most ~256 MiB so full-size pools leave room for them
    step = max(1, (256 << 20) // pool.block_bytes)
    if pool.layout == BM:
        out = hp.buffers[0].reshape(len(ids), -1)
        for lo in range(0, len(ids), step):
            sub = pool.tensors[0].index_select(0, idx[lo:lo + step]).contiguous()
            out[lo:lo + step] = sub.view(torch.uint8).reshape(sub.shape[0], -1).cpu().numpy()
    else:
        for l, t in enumerate(pool.tensors):
            out = hp.buffers[l].reshape(2, len(ids), -1)
            for lo in range(0, len(ids), step):
                sub = t.index_select(1, idx[lo:lo + step]).contiguous()
                out[:, lo:lo + step] = sub.view(torch.uint8).reshape(2, sub.shape[1], -1).cpu().numpy()
    return hp


def download_all(pool: fk.KVPool) -> oracle.HostPool:
    return download_blocks(pool, np.arange(pool.num_blocks))


def host_equal(a: oracle.HostPool, b: oracle.HostPool) -> bool:
    return all(np.array_equal(x, y) for x, y in zip(a.buffers, b.buffers))


def first_mismatch(a: oracle.HostPool, b: oracle.HostPool):
    for i, (x, y) in enumerate(zip(a.buffers, b.buffers)):
        d = np.flatnonzero(x != y)
        if d.size:
            return i, int(d[0]), int(d.size)
    return None


def run_transfer(src, dst, segs, stream=None, inline=False, layerwise=False, **cfg):
    """The plan moved as bench.py moves it: one launch with the plan in device
    memory, or (inline) carried in the kernel's arguments, as bench.py sends
    every plan that fits there (``fk.inline_capacity``); or (layerwise) one
    launch per layer from device memory, as its Table 3 sweep times the
    layer-wise form."""
    total = fk.plan_total_blocks(segs)
    if inline:
        fk.flowkv_transfer_inline(src, dst, segs, total, stream=stream, **cfg)
        torch.cuda.synchronize()
        return None
    dev = fk.segments_to_device(segs, src.device) if len(segs) else torch.zeros(
        (0, 4), dtype=torch.int32, device=src.device)
    if layerwise:
        for layer in range(src.num_layers):
            fk.flowkv_transfer_layers(src, dst, dev, len(segs), total, layer, 1, stream=stream,
                                      **cfg)
    elif cfg:
        fk.flowkv_transfer_ex(src, dst, dev, len(segs), total, stream=stream, **cfg)
    else:
        fk.flowkv_transfer(src, dst, dev, len(segs), total, stream=stream)
    torch.cuda.synchronize()
    return dev


def plan_tables(tables, src_blocks, dst_blocks):
    off = np.concatenate(([0], np.cumsum([len(s) for s, _ in tables]))).astype(np.int64)
    S = np.concatenate([s for s, _ in tables]) if tables else np.zeros(0, np.int32)
    D = np.concatenate([d for _, d in tables]) if tables else np.zeros(0, np.int32)
    return fk.flowkv_plan_batch(off, S, D, src_blocks, dst_blocks), S, D


def check_full_pool(geom, sl, dl, src_blocks, dst_blocks, tables, seed=0, **cfg):
    """Whole-pool comparison (small pools): GPU result == oracle result."""
    src = device_pool(geom, sl, src_blocks, seed)
    dst = device_pool(geom, dl, dst_blocks, seed + 1)
    h_src, h_dst = download_all(src), download_all(dst)
    segs, S, D = plan_tables(tables, src_blocks, dst_blocks)
    run_transfer(src, dst, segs, **cfg)
    oracle.transfer_batch_fast(h_src, h_dst, [(s, d) for s, d in tables])
    got = download_all(dst)
    assert host_equal(got, h_dst), first_mismatch(got, h_dst)
    return segs


def gather_blocks(pool: fk.KVPool, idx: torch.Tensor) -> torch.Tensor:
    """Blocks `idx` of a device pool as bytes, (len(idx), L, 2, chunk), in
    either layout; torch's own indexing, nothing from the library."""
    n, L = idx.numel(), pool.num_layers
    if pool.layout == BM:
        return pool.tensors[0].index_select(0, idx).view(torch.uint8).reshape(n, L, 2, -1)
    per_layer = [t.index_select(1, idx).view(torch.uint8).reshape(2, n, -1) for t in pool.tensors]
    return torch.stack(per_layer, 0).permute(2, 0, 1, 3)


def moved_blocks_equal(src: fk.KVPool, dst: fk.KVPool, S, D) -> bool:
    """Every moved block, whole, on the device: receiver block D[i] equals
    sender block S[i] in every layer and both of K and V.  With whole-block
    semantics this is the copy's definition at block granularity, so it holds
    at any size; pieces of about 256 MiB per side keep it within free memory."""
    S_t = torch.as_tensor(np.asarray(S, dtype=np.int64), device=src.device)
    D_t = torch.as_tensor(np.asarray(D, dtype=np.int64), device=dst.device)
    step = max(1, (256 << 20) // src.block_bytes)
    for lo in range(0, S_t.numel(), step):
        if not torch.equal(gather_blocks(src, S_t[lo:lo + step]),
                           gather_blocks(dst, D_t[lo:lo + step])):
            return False
    return True


def block_checksums(pool: fk.KVPool, piece_bytes: int = 256 << 20) -> torch.Tensor:
    """Two checksums of every block of a device pool, computed on the device
    with torch: the sum of the block's 32-bit words, and the sum of each word
    times a weight that depends on its position in the block (1 .. 4093), both
    in int64 (no overflow for blocks under 2 GiB).  Returns (num_blocks, 2)
    int64 on the device.  A write into a block changes them unless it
    happens to preserve both sums."""
    B, dev = pool.num_blocks, pool.device
    out = torch.zeros((B, 2), dtype=torch.int64, device=dev)
    if pool.layout == BM:
        parts = [(pool.tensors[0].view(torch.int32).reshape(B, -1), 0)]
    else:   # chunk (layer l, K/V kv) of every block, at word offset (2 l + kv) x chunk words
        cw = pool.chunk_bytes // 4
        parts = [(t[kv].view(torch.int32).reshape(B, -1), (2 * l + kv) * cw)
                 for l, t in enumerate(pool.tensors) for kv in range(2)]
    for words, base in parts:
        w = ((torch.arange(words.shape[1], device=dev, dtype=torch.int64) + base) % 4093) + 1
        step = max(1, piece_bytes // (4 * words.shape[1]))
        for lo in range(0, B, step):
            x = words[lo:lo + step].to(torch.int64)
            out[lo:lo + step, 0] += x.sum(1)
            out[lo:lo + step, 1] += (x * w).sum(1)
            del x
    return out


def check_sampled(wl, wl_ref, sl, dl, max_blocks=1536, untouched_frac=0.01, max_untouched=1024,
                  seed_sample=7, inline=False, layerwise=False, **cfg):
    """Full-size comparison: a seeded sample of the moved blocks (all of them
    when there are at most max_blocks) against the oracle; every moved block
    against its sender block on the device (`moved_blocks_equal`); the guard
    blocks around every receiver run plus a seeded sample of the other
    receiver blocks against their pre-image, byte for byte; and every other
    receiver block of the whole pool against its pre-image by the two
    checksums of `block_checksums`.

    `wl` holds the block lists from the library's allocator (they drive the
    device path), `wl_ref` the same workload from the oracle's allocator
    (they pick what the oracle copies); the two must agree exactly."""
    assert len(wl.tables) == len(wl_ref.tables)
    for (s1, d1), (s2, d2) in zip(wl.tables, wl_ref.tables):
        assert np.array_equal(s1, s2) and np.array_equal(d1, d2)
    geom = wl.geom
    need = pool_bytes(geom, wl.src_pool_blocks) + pool_bytes(geom, wl.dst_pool_blocks)
    gc.collect()
    torch.cuda.empty_cache()
    free, _ = torch.cuda.mem_get_info()
    assert need < free, f"pools need {need / 2**30:.1f} GiB, {free / 2**30:.1f} GiB free"
    src = device_pool(geom, sl, wl.src_pool_blocks, 0)
    dst = device_pool(geom, dl, wl.dst_pool_blocks, 1)
    segs, S, D = plan_tables(wl.tables, wl.src_pool_blocks, wl.dst_pool_blocks)
    S_ref, D_ref = wl_ref.flat()
    pick = sample_indices(len(S_ref), max_blocks, seed_sample)
    h_src = download_blocks(src, S_ref[pick])
    # receiver blocks not written: one guard on each side of every run, and a
    # seeded sample of the rest
    touched = np.zeros(wl.dst_pool_blocks, dtype=bool)
    touched[D] = True
    ends = segs["dst_block"] + segs["n_blocks"]
    guards = np.concatenate((segs["dst_block"] - 1, ends))
    guards = guards[(guards >= 0) & (guards < wl.dst_pool_blocks)]
    guards = np.unique(guards[~touched[guards]])
    rest = np.flatnonzero(~touched)
    k = min(max_untouched, max(1, int(untouched_frac * rest.size))) if rest.size else 0
    rest = rest[sample_indices(rest.size, k, seed_sample + 1)] if k else rest[:0]
    keep = np.unique(np.concatenate((guards[:max_untouched], rest))).astype(np.int64)
    before = download_blocks(dst, keep)
    sums_before = block_checksums(dst)
    run_transfer(src, dst, segs, inline=inline, layerwise=layerwise, **cfg)
    untouched = torch.as_tensor(~touched, device=dst.device)
    sums_after = block_checksums(dst)
    changed = (sums_after != sums_before).any(1) & untouched
    assert not bool(changed.any()), \
        f"untouched receiver blocks changed: {torch.nonzero(changed)[:8].flatten().tolist()}"
    del sums_before, sums_after, untouched, changed
    # oracle on compact pools: sampled logical block i moves from compact
    # sender block i to compact receiver block i
    expect = oracle.HostPool.zeros(dl, geom.num_layers, len(pick), geom.block_size,
                                   geom.slot_bytes)
    oracle.transfer_fast(h_src, expect, np.arange(len(pick)), np.arange(len(pick)))
    got = download_blocks(dst, D_ref[pick])
    assert host_equal(got, expect), first_mismatch(got, expect)
    after = download_blocks(dst, keep)
    assert host_equal(after, before), first_mismatch(after, before)
    assert moved_blocks_equal(src, dst, S, D)
    del src, dst
    torch.cuda.empty_cache()
    return segs, len(pick), len(keep)
