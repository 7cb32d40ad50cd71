"""GPU parity: the one-launch transfer kernel against the oracle, byte-exact.

Small pools are compared whole.  At full size, a seeded sample of the moved
blocks is compared with the oracle, every moved block with its sender block
on the device, and every guard block around a receiver run plus a seeded 1%
sample of the untouched receiver blocks with their pre-image.  Every case goes through the C ABI
(allocator, planner, transfer) via the ctypes binding.
"""

import gc
import itertools
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2504_03775_amd import flowkv as fk
from workloads import TINY, LLAMA3_8B, Geometry, recipes
from tests.gpu_helpers import (BM, LM, check_full_pool, check_sampled, device_pool,
                               download_all, first_mismatch, host_equal, plan_tables,
                               run_transfer)

pytestmark = pytest.mark.gpu

LAYOUT_PAIRS = list(itertools.product([LM, BM], [LM, BM]))
NAMES = {LM: "layer", BM: "block"}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def lib_alloc(P, pol, seed):
    return fk.Allocator(P, pol, seed)


def ref_alloc(P, pol, seed):
    return oracle.RefAllocator(P, pol, seed)


@pytest.mark.parametrize("sl,dl", LAYOUT_PAIRS, ids=lambda x: NAMES[x])
def test_tiny_full_pool_against_literal_loop(sl, dl):
    wl = recipes.tiny()
    say("tiny", NAMES[sl], NAMES[dl])
    src = device_pool(wl.geom, sl, 64, 0)
    dst = device_pool(wl.geom, dl, 64, 1)
    h_src, h_dst = download_all(src), download_all(dst)
    segs, S, D = plan_tables(wl.tables, 64, 64)
    run_transfer(src, dst, segs)
    oracle.transfer_ref(h_src, h_dst, S, D)  # the pure-Python definition
    assert host_equal(download_all(dst), h_dst)
    assert len(segs) == len(oracle.plan_ref(S.tolist(), D.tolist()))


CONFIGS = [dict(), dict(threads=64), dict(threads=128, unroll=2), dict(threads=512, unroll=16),
           dict(threads=1024, unroll=4), dict(grid=1), dict(grid=3, unroll=2),
           dict(cache=1), dict(cache=2), dict(cache=3), dict(cache=4, unroll=16, grid=5),
           dict(order=2), dict(order=3), dict(order=2, grid=7, threads=256),
           dict(order=3, grid=2, unroll=4), dict(order=1, grid=4), dict(order=4),
           dict(order=4, grid=5, threads=256), dict(order=4, threads=128, unroll=2)]


def random_case(seed):
    g = np.random.default_rng(seed)
    L = int(g.choice([1, 2, 3, 7, 128]))
    bs = int(g.choice([1, 2, 5, 16]))
    hkv = int(g.choice([1, 2, 3]))
    dh = int(g.choice([8, 40, 64, 128]))
    geom = Geometry(f"rand{seed}", L, hkv, dh, bs, "float16")
    if geom.chunk_bytes % 16:
        geom = Geometry(f"rand{seed}", L, hkv, 64, bs, "float16")
    # keep the pools small: at most ~48 MiB each
    maxb = max(2, min(96, (48 << 20) // geom.block_bytes))
    Bs = int(g.integers(1, maxb + 1))
    Bd = int(g.integers(1, maxb + 1))
    kind = g.integers(4)
    n_req = int(g.integers(1, 4))
    tables = []
    if kind == 0:      # seeded permutations
        ps, pd = g.permutation(Bs), g.permutation(Bd)
    elif kind == 1:    # contiguous on both sides
        ps, pd = np.arange(Bs), np.arange(Bd)
    elif kind == 2:    # descending (never mergeable)
        ps, pd = np.arange(Bs)[::-1], np.arange(Bd)[::-1]
    else:              # ascending free blocks of a randomly occupied receiver
        ps = np.arange(Bs)
        busy = g.permutation(Bd)[: int(g.integers(0, Bd // 2 + 1))]
        pd = np.setdiff1d(np.arange(Bd), busy)
    n = int(g.integers(0, min(len(ps), len(pd)) + 1))
    cuts = np.sort(g.integers(0, n + 1, size=n_req - 1))
    bounds = np.concatenate(([0], cuts, [n]))
    for i in range(n_req):
        tables.append((ps[bounds[i]:bounds[i + 1]].astype(np.int32),
                       pd[bounds[i]:bounds[i + 1]].astype(np.int32)))
    return geom, Bs, Bd, tables


@pytest.mark.parametrize("seed", range(48))
def test_random_shapes_layouts_and_launch_shapes(seed):
    geom, Bs, Bd, tables = random_case(seed)
    sl, dl = LAYOUT_PAIRS[seed % 4]
    cfg = CONFIGS[seed % len(CONFIGS)]
    say(f"seed={seed} L={geom.num_layers} bs={geom.block_size} Hkv={geom.kv_heads} "
        f"Dh={geom.head_dim} H={geom.chunk_bytes} Bs={Bs} Bd={Bd} "
        f"n={sum(len(s) for s, _ in tables)} {NAMES[sl]}->{NAMES[dl]} cfg={cfg}")
    check_full_pool(geom, sl, dl, Bs, Bd, tables, seed=seed, **cfg)


def test_empty_plan_leaves_pool_unchanged():
    src = device_pool(TINY, BM, 8, 0)
    dst = device_pool(TINY, LM, 8, 1)
    before = download_all(dst)
    run_transfer(src, dst, fk.flowkv_plan([], [], 8, 8))
    assert host_equal(download_all(dst), before)


def test_last_block_ids_and_max_layers():
    """Block IDs at the very end of the pools, 128 layers, per-lane path
    (H = 16 * 3 * 40 * 2 = 3,840 bytes is not a multiple of the line)."""
    geom = Geometry("edge", 128, 3, 40, 16, "bfloat16")
    Bs, Bd = 9, 7
    tables = [(np.array([8, 0, 7], np.int32), np.array([6, 5, 0], np.int32))]
    for sl, dl in LAYOUT_PAIRS:
        check_full_pool(geom, sl, dl, Bs, Bd, tables)


@pytest.mark.parametrize("path", ["per_lane", "uniform"])
def test_blocks_just_under_the_2_gib_limit(path):
    """The largest block the launcher accepts (2 x layers x H < 2 GiB), where
    offsets inside a block use the top of 31 bits: one layer, H = 2^30 - 256
    (not a multiple of the 16 KiB line: per-lane path) or 2^30 - 16,384
    (uniform path); 3-block pools, both layouts."""
    if path == "per_lane":
        geom = Geometry("huge-lane", 1, 3, 128, 1398101, "bfloat16")    # H = 2^30 - 256
    else:
        geom = Geometry("huge-uni", 1, 64, 128, 65535, "bfloat16")      # H = 2^30 - 16384
    assert 2**31 - 2**15 <= geom.block_bytes < 2**31
    tables = [(np.array([2, 0], np.int32), np.array([1, 2], np.int32))]
    for sl, dl in ((BM, BM), (LM, BM)):
        say(f"{path}: block {geom.block_bytes} B, {NAMES[sl]}->{NAMES[dl]}")
        check_full_pool(geom, sl, dl, 3, 3, tables)
        gc.collect()
        torch.cuda.empty_cache()


def test_plan_records_outside_pools_are_skipped():
    """A hand-made record pointing past the receiver pool moves nothing and
    faults nothing; the valid record next to it still moves."""
    geom = TINY
    src = device_pool(geom, BM, 4, 0)
    dst = device_pool(geom, BM, 4, 1)
    h_src, h_dst = download_all(src), download_all(dst)
    segs = np.zeros(2, dtype=fk.SEGMENT_DTYPE)
    segs[0] = (1, 2, 1, 0)
    segs[1] = (0, 3, 4, 1)  # blocks 3..6 of a 4-block receiver: out of range
    dev = fk.segments_to_device(segs, src.device)
    fk.flowkv_transfer(src, dst, dev, 2, 5)
    torch.cuda.synchronize()
    got = download_all(dst)
    # record 0 moves block 1 -> 2; record 1's first block (0 -> 3) is inside
    # both pools and moves, its other three blocks would land past the end
    oracle.transfer_fast(h_src, h_dst, [1, 0], [2, 3])
    assert host_equal(got, h_dst)


def test_two_streams_two_plans():
    """Two plans on two streams into disjoint receiver blocks."""
    geom = LLAMA3_8B
    src = device_pool(geom, BM, 16, 0)
    dst = device_pool(geom, BM, 16, 1)
    h_src, h_dst = download_all(src), download_all(dst)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    p1 = fk.flowkv_plan([0, 1, 2], [10, 11, 3], 16, 16)
    p2 = fk.flowkv_plan([5, 9], [0, 1], 16, 16)
    d1 = fk.segments_to_device(p1, src.device, s1)
    d2 = fk.segments_to_device(p2, src.device, s2)
    fk.flowkv_transfer(src, dst, d1, len(p1), 3, stream=s1)
    fk.flowkv_transfer(src, dst, d2, len(p2), 2, stream=s2)
    torch.cuda.synchronize()
    oracle.transfer_fast(h_src, h_dst, [0, 1, 2, 5, 9], [10, 11, 3, 0, 1])
    assert host_equal(download_all(dst), h_dst)


def test_plan_stager_on_idle_and_busy_streams():
    """PlanStager copies a plan on the stream itself when it is idle and on
    its side stream behind running work; with more plans than ring slots and
    one plan above the ring's capacity (the ring grows), every transfer
    equals the oracle's."""
    geom = Geometry("stager", 2, 2, 64, 16, "float16")      # 16 KiB blocks
    B = 2048
    src = device_pool(geom, BM, B, 0)
    dst = device_pool(geom, BM, B, 1)
    h_src, h_dst = download_all(src), download_all(dst)
    stager = fk.PlanStager(src.device, capacity=8, slots=2)
    stream = torch.cuda.current_stream()
    filler = torch.empty(256 << 20, dtype=torch.uint8, device=src.device)
    g = np.random.default_rng(9)
    perm = g.permutation(B).astype(np.int32)
    pos, seen = 0, set()
    for i in range(12):
        n = 300 if i == 7 else int(g.integers(1, 100))
        S, D = g.permutation(B)[:n].astype(np.int32), perm[pos:pos + n]
        pos += n
        segs = fk.flowkv_plan(S, D, B, B)
        if i % 3 == 0:
            torch.cuda.synchronize()          # idle: the copy goes on the stream
        else:
            for _ in range(8):                # busy (about 0.3 ms of queued fills): the
                filler.fill_(i)               # copy goes on the side stream
        seen.add(stream.query())
        dev = stager.stage(segs, stream)
        fk.flowkv_transfer_ex(src, dst, dev, len(segs), n, stream=stream)
        stager.release(stream)
        oracle.transfer_fast(h_src, h_dst, S, D)
    torch.cuda.synchronize()
    assert seen == {True, False}
    got = download_all(dst)
    assert host_equal(got, h_dst), first_mismatch(got, h_dst)


def test_launches_from_four_host_threads():
    """The launcher is reentrant: four host threads each plan and enqueue
    transfers on a stream of their own at the same time (ctypes releases the
    interpreter lock during the calls), into disjoint receiver blocks, with
    both kernel-argument and device plans; the result equals the oracle's."""
    from concurrent.futures import ThreadPoolExecutor

    geom = Geometry("threads", 4, 2, 64, 16, "float16")     # 32 KiB blocks
    B = 4096
    src = device_pool(geom, BM, B, 0)
    dst = device_pool(geom, LM, B, 1)
    h_src, h_dst = download_all(src), download_all(dst)
    g = np.random.default_rng(3)
    perm_d = g.permutation(B).astype(np.int32)
    jobs = []   # per thread: 24 requests of 1..40 blocks, receiver blocks disjoint
    pos = 0
    for t in range(4):
        reqs = []
        for _ in range(24):
            n = int(g.integers(1, 41))
            S = (np.arange(n) + int(g.integers(0, B - n))).astype(np.int32) if g.random() < 0.5 \
                else g.permutation(B)[:n].astype(np.int32)
            reqs.append((S, perm_d[pos:pos + n]))
            pos += n
        jobs.append(reqs)

    def worker(t):
        stream = torch.cuda.Stream(src.device)
        keep = []
        for i, (S, D) in enumerate(jobs[t]):
            segs = fk.flowkv_plan(S, D, B, B)
            if i % 2 and len(segs) <= fk.INLINE_RUNS:
                fk.flowkv_transfer_inline(src, dst, segs, len(S), stream=stream)
            else:
                dev = fk.segments_to_device(segs, src.device, stream)
                keep.append(dev)
                fk.flowkv_transfer(src, dst, dev, len(segs), len(S), stream=stream)
        stream.synchronize()
        return len(keep)

    with ThreadPoolExecutor(4) as ex:
        list(ex.map(worker, range(4)))
    torch.cuda.synchronize()
    for reqs in jobs:
        for S, D in reqs:
            oracle.transfer_fast(h_src, h_dst, S, D)
    got = download_all(dst)
    assert host_equal(got, h_dst), first_mismatch(got, h_dst)


# ---- full-size workloads -----------------------------------------------------

def build(recipe, *args):
    return recipe(lib_alloc, *args), recipe(ref_alloc, *args)


@pytest.mark.parametrize("policy", ["fifo_sorted", "segment"])
@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, LM), (LM, BM), (BM, LM)],
                         ids=lambda x: NAMES[x])
def test_llama8b_13k_full_size(policy, sl, dl):
    wl, ref = build(recipes.llama8b_13k, policy)
    say(f"8b 13k {policy} {NAMES[sl]}->{NAMES[dl]}: {wl.n_blocks} blocks")
    segs, nb, nk = check_sampled(wl, ref, sl, dl)
    assert nb == 813  # every moved block checked
    say(f"  {len(segs)} runs, {nb} blocks checked, {nk} untouched checked")


@pytest.mark.parametrize("policy,sl,dl", [("segment", BM, BM), ("segment", LM, BM),
                                          ("fifo_sorted", BM, BM), ("fifo_sorted", LM, LM)])
def test_llama8b_13k_full_size_plan_in_kernel_arguments(policy, sl, dl):
    """The 13k request in the launch bench.py times for it: the plan carried
    in the kernel's arguments -- 43 runs from the segment-allocator receiver,
    255 from the free-list receiver (12-byte records beside one base pointer
    per side between block-major pools, beside 32 per side between
    layer-major ones)."""
    wl, ref = build(recipes.llama8b_13k, policy)
    say(f"8b 13k inline {policy} {NAMES[sl]}->{NAMES[dl]}")
    segs, nb, nk = check_sampled(wl, ref, sl, dl, inline=True)
    assert nb == 813
    cap = (fk.INLINE_RUNS_BLOCK_MAJOR if (sl, dl) == (BM, BM) else fk.INLINE_RUNS_LAYER_MAJOR)
    assert len(segs) <= cap
    if policy == "fifo_sorted":
        assert len(segs) > fk.INLINE_RUNS  # the compact form
    say(f"  inline: {len(segs)} runs, {nb} blocks checked, {nk} untouched checked")


@pytest.mark.parametrize("tokens", [500, 4000, 12000])
def test_table3_lengths_full_size_per_layer_launches(tokens):
    """Table 3's FlowKV-Layerwise column as bench.py --op table3 times it:
    the request at one of the table's input lengths, free-list receiver in
    the 65,536-block pools, moved as 32 per-layer launches from a device
    plan; sampled against the oracle like the other full-size cases."""
    wl, ref = build(recipes.llama8b_13k, "fifo_sorted", 65_536, tokens)
    say(f"table3 {tokens} tokens, per-layer launches: {wl.n_blocks} blocks")
    segs, nb, nk = check_sampled(wl, ref, BM, BM, layerwise=True)
    assert nb == wl.n_blocks
    say(f"  {len(segs)} runs, {nb} blocks checked, {nk} untouched checked")


@pytest.mark.parametrize("policy,sl,dl", [("segment", BM, BM), ("fifo_shuffled", BM, BM),
                                          ("segment", LM, LM)])
def test_batch32_full_size(policy, sl, dl):
    wl, ref = build(recipes.batch32, policy)
    say(f"batch32 {policy} {NAMES[sl]}->{NAMES[dl]}: {wl.n_blocks} blocks, "
        f"pools {wl.src_pool_blocks}/{wl.dst_pool_blocks}")
    segs, nb, nk = check_sampled(wl, ref, sl, dl)
    if policy == "segment":
        assert len(segs) == 32
    say(f"  {len(segs)} runs, {nb} blocks checked")


@pytest.mark.parametrize("policy,sl,dl", [("segment", BM, BM), ("fifo_shuffled", LM, LM),
                                          ("segment", BM, LM)])
def test_llama70b_tp8_full_size(policy, sl, dl):
    wl, ref = build(recipes.llama70b_tp8, policy)
    say(f"70b tp8 {policy} {NAMES[sl]}->{NAMES[dl]}: {wl.n_blocks} blocks")
    segs, nb, nk = check_sampled(wl, ref, sl, dl, max_blocks=4096)
    if policy == "segment":
        assert len(segs) == 16
    say(f"  {len(segs)} runs, {nb} blocks checked")


@pytest.mark.parametrize("variant,sl,dl", [("segment", BM, BM), ("shuffled", BM, BM),
                                           ("stride2", BM, BM), ("shuffled", LM, BM)])
def test_churn_full_size(variant, sl, dl):
    wl, ref = build(recipes.churn, variant)
    say(f"churn {variant} {NAMES[sl]}->{NAMES[dl]}: {wl.n_blocks} blocks")
    segs, nb, nk = check_sampled(wl, ref, sl, dl)
    if variant == "stride2":
        assert len(segs) == wl.n_blocks
    say(f"  {len(segs)} runs, {nb} blocks checked")


# ---- layer-wise variant (section 4.4, Table 3: FlowKV-Layerwise) -------------

@pytest.mark.parametrize("seed", range(16))
def test_layer_ranges_against_oracle(seed):
    geom, Bs, Bd, tables = random_case(1000 + seed)
    sl, dl = LAYOUT_PAIRS[seed % 4]
    g = np.random.default_rng(seed)
    l0 = int(g.integers(0, geom.num_layers))
    lc = int(g.integers(1, geom.num_layers - l0 + 1))
    cfg = CONFIGS[seed % len(CONFIGS)]
    say(f"layers seed={seed} L={geom.num_layers} [{l0}, {l0 + lc}) H={geom.chunk_bytes} "
        f"{NAMES[sl]}->{NAMES[dl]} cfg={cfg}")
    src = device_pool(geom, sl, Bs, seed)
    dst = device_pool(geom, dl, Bd, seed + 1)
    h_src, h_dst = download_all(src), download_all(dst)
    segs, S, D = plan_tables(tables, Bs, Bd)
    dev = fk.segments_to_device(segs, src.device) if len(segs) else torch.zeros(
        (0, 4), dtype=torch.int32, device=src.device)
    fk.flowkv_transfer_layers(src, dst, dev, len(segs), fk.plan_total_blocks(segs), l0, lc, **cfg)
    torch.cuda.synchronize()
    for s_, d_ in tables:
        oracle.transfer_fast(h_src, h_dst, s_, d_, layers=range(l0, l0 + lc))
    assert host_equal(download_all(dst), h_dst)


@pytest.mark.parametrize("l0,lc", [(127, 1), (0, 128), (64, 64)],
                         ids=["last-layer", "all-layers", "upper-half"])
def test_layer_ranges_of_the_deepest_pools(l0, lc):
    """Layer ranges at the top of 128-layer pools, in all four layout pairs,
    on both address paths (H = 3,840 B: per-lane; H = 4 KiB at 256 threads:
    uniform), against the oracle over the whole receiver pool."""
    tables = [(np.array([8, 0, 7, 1], np.int32), np.array([6, 5, 0, 1], np.int32))]
    for geom, cfg in ((Geometry("deep-lane", 128, 3, 40, 16, "bfloat16"), {}),
                      (Geometry("deep-uni", 128, 1, 128, 16, "bfloat16"), dict(threads=256))):
        for sl, dl in LAYOUT_PAIRS:
            say(f"layers [{l0}, {l0 + lc}) of 128, H={geom.chunk_bytes} {NAMES[sl]}->{NAMES[dl]}")
            src = device_pool(geom, sl, 9, 3)
            dst = device_pool(geom, dl, 7, 4)
            h_src, h_dst = download_all(src), download_all(dst)
            segs, S, D = plan_tables(tables, 9, 7)
            dev = fk.segments_to_device(segs, src.device)
            fk.flowkv_transfer_layers(src, dst, dev, len(segs), fk.plan_total_blocks(segs), l0,
                                      lc, **cfg)
            torch.cuda.synchronize()
            for s_, d_ in tables:
                oracle.transfer_fast(h_src, h_dst, s_, d_, layers=range(l0, l0 + lc))
            got = download_all(dst)
            assert host_equal(got, h_dst), first_mismatch(got, h_dst)


def test_pools_of_different_element_types_are_refused():
    """bf16 into fp16 has the same byte geometry, which is all the library
    compares; the binding refuses the pair before any launch."""
    a = device_pool(Geometry("bf", 2, 2, 64, 16, "bfloat16"), BM, 8, 0)
    b = device_pool(Geometry("fp", 2, 2, 64, 16, "float16"), BM, 8, 1)
    before = b.tensors[0].clone()
    segs = fk.flowkv_plan([0, 1], [2, 3], 8, 8)
    dev = fk.segments_to_device(segs, a.device)
    for call in (lambda: fk.flowkv_transfer_inline(a, b, segs, 2),
                 lambda: fk.flowkv_transfer(a, b, dev, len(segs), 2),
                 lambda: fk.flowkv_transfer_layers(b, a, dev, len(segs), 2, 0, 1),
                 lambda: fk.flowkv_transfer_request(a, b, [0, 1], [2, 3])):
        with pytest.raises(ValueError, match="element types"):
            call()
    torch.cuda.synchronize()
    assert torch.equal(b.tensors[0], before)


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, BM)], ids=lambda x: NAMES[x])
def test_concurrent_requests_on_separate_streams(sl, dl):
    """The copy keeps no state between launches: four requests moved at once
    on four streams (plans in the kernel arguments, disjoint receiver blocks)
    leave the receiver exactly as the oracle moving them one after another."""
    geom = Geometry("streams", 4, 2, 64, 16, "bfloat16")
    B = 160
    g = np.random.default_rng(77)
    src_ids = g.permutation(B).astype(np.int32)
    dst_ids = g.permutation(B).astype(np.int32)
    sizes = [40, 1, 23, 60]
    tables, pos = [], 0
    for k in sizes:
        tables.append((src_ids[pos:pos + k], dst_ids[pos:pos + k]))
        pos += k
    src = device_pool(geom, sl, B, 5)
    dst = device_pool(geom, dl, B, 6)
    h_src, h_dst = download_all(src), download_all(dst)
    streams = [torch.cuda.Stream() for _ in tables]    # default priority
    torch.cuda.synchronize()
    for (s_, d_), st in zip(tables, streams):
        segs = fk.flowkv_plan(s_, d_, B, B)
        fk.flowkv_transfer_inline(src, dst, segs, len(s_), stream=st)
    torch.cuda.synchronize()
    for s_, d_ in tables:
        oracle.transfer_fast(h_src, h_dst, s_, d_)
    got = download_all(dst)
    assert host_equal(got, h_dst), first_mismatch(got, h_dst)


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, LM)], ids=lambda x: NAMES[x])
def test_one_launch_per_layer_equals_one_launch(sl, dl):
    """The 8B geometry (32 layers): 32 per-layer launches give the same
    receiver pool as one whole-plan launch."""
    geom = LLAMA3_8B
    src = device_pool(geom, sl, 24, 0)
    d1 = device_pool(geom, dl, 24, 1)
    d2 = device_pool(geom, dl, 24, 1)
    segs = fk.flowkv_plan([3, 4, 5, 9, 1], [0, 1, 2, 20, 7], 24, 24)
    dev = fk.segments_to_device(segs, src.device)
    fk.flowkv_transfer(src, d1, dev, len(segs), 5)
    for l in range(geom.num_layers):
        fk.flowkv_transfer_layers(src, d2, dev, len(segs), 5, l, 1)
    torch.cuda.synchronize()
    assert host_equal(download_all(d1), download_all(d2))


# ---- plans carried in the kernel arguments -----------------------------------

@pytest.mark.parametrize("seed", range(12))
def test_inline_plans_against_oracle(seed):
    geom, Bs, Bd, tables = random_case(2000 + seed)
    sl, dl = LAYOUT_PAIRS[seed % 4]
    cfg = CONFIGS[seed % len(CONFIGS)]
    segs, S, D = plan_tables(tables, Bs, Bd)
    if len(segs) > fk.INLINE_RUNS:
        pytest.skip("plan longer than the inline limit")
    say(f"inline seed={seed} runs={len(segs)} n={len(S)} {NAMES[sl]}->{NAMES[dl]} cfg={cfg}")
    src = device_pool(geom, sl, Bs, seed)
    dst = device_pool(geom, dl, Bd, seed + 1)
    h_src, h_dst = download_all(src), download_all(dst)
    fk.flowkv_transfer_inline(src, dst, segs, fk.plan_total_blocks(segs), **cfg)
    torch.cuda.synchronize()
    oracle.transfer_batch_fast(h_src, h_dst, [(s_, d_) for s_, d_ in tables])
    assert host_equal(download_all(dst), h_dst)


@pytest.mark.parametrize("seed", range(16))
def test_compact_inline_plans_against_oracle(seed):
    """Plans of 65 runs up to the compact capacity, carried in the kernel
    arguments as 12-byte records: 300 between block-major pools, 264 when a
    pool is layer-major (at most 32 layers); every layout pair, random
    geometries (the uniform and the per-lane path, 1 to 32 layers), runs of
    1 to 3 blocks, random launch shapes."""
    g = np.random.default_rng(5000 + seed)
    geoms = [Geometry("c1", 2, 2, 64, 16, "float16"), Geometry("c2", 3, 3, 40, 16, "bfloat16"),
             Geometry("c3", 1, 1, 128, 5, "float16"), Geometry("c4", 32, 1, 32, 2, "bfloat16")]
    geom = geoms[seed % len(geoms)]
    sl, dl = LAYOUT_PAIRS[(seed // len(geoms)) % 4]
    cap = fk.INLINE_RUNS_BLOCK_MAJOR if (sl, dl) == (BM, BM) else fk.INLINE_RUNS_LAYER_MAJOR
    k = int(g.integers(fk.INLINE_RUNS + 1, cap + 1))
    if seed < 4:
        k = cap
    lens = g.integers(1, 4, size=k)
    n = int(lens.sum())
    B = 2 * n + 8
    # runs that cannot merge: each run's sender start jumps ahead
    S, D, s0, d0 = [], [], 0, int(g.integers(0, 4))
    for m in lens:
        S.extend(range(s0, s0 + m))
        D.extend(range(d0, d0 + m))
        s0 += m + 1
        d0 += m + int(g.integers(0, 2))
    S, D = np.array(S, np.int32), np.array(D, np.int32)
    assert S.max() < B and D.max() < B
    segs = fk.flowkv_plan(S, D, B, B)
    assert len(segs) == k
    cfg = CONFIGS[seed % len(CONFIGS)]
    say(f"compact inline seed={seed} {NAMES[sl]}->{NAMES[dl]} runs={k} blocks={n} "
        f"geom={geom.name} cfg={cfg}")
    src = device_pool(geom, sl, B, seed)
    dst = device_pool(geom, dl, B, seed + 1)
    assert fk.inline_capacity(src, dst) == cap
    h_src, h_dst = download_all(src), download_all(dst)
    fk.flowkv_transfer_inline(src, dst, segs, n, **cfg)
    torch.cuda.synchronize()
    oracle.transfer_fast(h_src, h_dst, S, D)
    got = download_all(dst)
    assert host_equal(got, h_dst), first_mismatch(got, h_dst)


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, LM), (LM, BM)], ids=lambda x: NAMES[x])
def test_transfer_request_plans_and_moves_one_request(sl, dl):
    """flowkv_transfer_request (plan and launch in one call) on a request
    whose lists are runs of consecutive IDs with random breaks: the receiver
    pool equals the oracle's, byte for byte, and the run count is the
    planner's.  A plan past the inline capacity raises ECAP and moves
    nothing."""
    geom = Geometry("req", 4, 2, 64, 16, "bfloat16")
    B = 700                        # room for the stride-2 lists of 301 blocks below
    g = np.random.default_rng(77 + sl * 2 + dl)
    def table(n):
        out, x, used = [], int(g.integers(0, B)), set()
        while len(out) < n:
            if g.random() < 0.08 or x >= B or x in used:
                x = int(g.integers(0, B))
                continue
            out.append(x)
            used.add(x)
            x += 1
        return np.asarray(out, dtype=np.int32)
    S, D = table(200), table(200)
    want_runs = len(fk.flowkv_plan(S, D, B, B))
    src = device_pool(geom, sl, B, 5)
    dst = device_pool(geom, dl, B, 6)
    cap = fk.inline_capacity(src, dst)
    assert want_runs <= cap, (want_runs, cap)
    h_src, h_dst = download_all(src), download_all(dst)
    say(f"request {NAMES[sl]}->{NAMES[dl]}: {len(S)} blocks, {want_runs} runs, capacity {cap}")
    assert fk.flowkv_transfer_request(src, dst, S, D) == want_runs
    torch.cuda.synchronize()
    oracle.transfer_fast(h_src, h_dst, S, D)
    after = download_all(dst)
    assert host_equal(after, h_dst)
    # past the capacity: ECAP with the run count, and the receiver untouched
    k = cap + 1
    with pytest.raises(fk.FlowKVError) as e:
        fk.flowkv_transfer_request(src, dst, 2 * np.arange(k), 2 * np.arange(k) + 1)
    assert e.value.code == fk.ECAP
    torch.cuda.synchronize()
    assert host_equal(download_all(dst), after)


def test_inline_plan_at_the_limit_equals_device_plan():
    """64 one-block runs (the inline limit) at the 8B geometry: the inline and
    the device-memory plan give the same receiver pool, and match the oracle."""
    geom = LLAMA3_8B
    src = device_pool(geom, BM, 130, 0)
    d1 = device_pool(geom, LM, 130, 1)
    d2 = device_pool(geom, LM, 130, 1)
    h_src, h_dst = download_all(src), download_all(d1)
    S = 2 * np.arange(64, dtype=np.int32)
    D = 2 * np.arange(64, dtype=np.int32) + 1
    segs = fk.flowkv_plan(S, D, 130, 130)
    assert len(segs) == fk.INLINE_RUNS
    fk.flowkv_transfer_inline(src, d1, segs, 64)
    fk.flowkv_transfer(src, d2, fk.segments_to_device(segs, src.device), len(segs), 64)
    torch.cuda.synchronize()
    oracle.transfer_fast(h_src, h_dst, S, D)
    got = download_all(d1)
    assert host_equal(got, h_dst)
    assert host_equal(got, download_all(d2))


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, LM), (BM, LM)], ids=lambda x: NAMES[x])
def test_compact_inline_plan_at_the_limit_equals_device_plan(sl, dl):
    """One-block runs up to the compact limit (300 between block-major
    pools, 264 with a layer-major pool) at the 8B geometry, whose 32 layers
    fill the layer-major form's base pointers: the compact inline plan and
    the device-memory plan give the same receiver pool, and match the
    oracle."""
    geom = LLAMA3_8B
    assert geom.num_layers == fk.INLINE_LAYERS
    k = fk.INLINE_RUNS_BLOCK_MAJOR if (sl, dl) == (BM, BM) else fk.INLINE_RUNS_LAYER_MAJOR
    B = 2 * k + 2
    src = device_pool(geom, sl, B, 0)
    d1 = device_pool(geom, dl, B, 1)
    d2 = device_pool(geom, dl, B, 1)
    assert fk.inline_capacity(src, d1) == k
    h_src, h_dst = download_all(src), download_all(d1)
    S = 2 * np.arange(k, dtype=np.int32)
    D = 2 * np.arange(k, dtype=np.int32) + 1
    segs = fk.flowkv_plan(S, D, B, B)
    assert len(segs) == k
    say(f"compact inline at the limit {NAMES[sl]}->{NAMES[dl]}: {k} runs")
    fk.flowkv_transfer_inline(src, d1, segs, k)
    fk.flowkv_transfer(src, d2, fk.segments_to_device(segs, src.device), len(segs), k)
    torch.cuda.synchronize()
    oracle.transfer_fast(h_src, h_dst, S, D)
    got = download_all(d1)
    assert host_equal(got, h_dst)
    assert host_equal(got, download_all(d2))
