"""Pins for the transfer oracle (``oracle.kvcopy``), CPU only.

The oracle computes pool offsets with its own explicit formulas.  These tests
read and write the pools only through numpy's shaped-array indexing of the
Eq. 5 layouts -- (2, B, bs, slot) per layer for (L, 2, B, H), and
(B, L, 2, bs, slot) for (B, L, 2, H) -- so a wrong stride, a swapped index or
a dropped term in the oracle shows up as a wrong tag.  The same views give the
slot addresses that pin Eq. 5's point: a request's aligned runs are one
contiguous copy each block-major and 2L each layer-major.
"""

import itertools

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import (BLOCK_MAJOR, LAYER_MAJOR, HostPool, transfer_fast,
                    transfer_ref, transfer_batch_fast)

LAYOUTS = [LAYER_MAJOR, BLOCK_MAJOR]


def shaped(pool: HostPool, dtype=np.int32):
    """numpy views of a pool indexed as [l][kv, b, s, w] or [b, l, kv, s, w]."""
    w = pool.slot_bytes // np.dtype(dtype).itemsize
    if pool.layout == LAYER_MAJOR:
        return [buf.view(dtype).reshape(2, pool.num_blocks, pool.block_size, w)
                for buf in pool.buffers]
    return pool.buffers[0].view(dtype).reshape(
        pool.num_blocks, pool.num_layers, 2, pool.block_size, w)


def get_slot(pool, views, b, l, kv, s):
    if pool.layout == LAYER_MAJOR:
        return views[l][kv, b, s]
    return views[b, l, kv, s]


def tag_pool(pool: HostPool, marker: int):
    """Write (b, l, kv, s, marker, ...) into the int32 words of every slot."""
    v = shaped(pool)
    B, L, bs = pool.num_blocks, pool.num_layers, pool.block_size
    b = np.arange(B)[:, None]
    s = np.arange(bs)[None, :]
    for l in range(L):
        for kv in (0, 1):
            if pool.layout == LAYER_MAJOR:
                tgt = v[l][kv]
            else:
                tgt = v[:, l, kv]
            tgt[..., 0] = b
            tgt[..., 1] = l
            tgt[..., 2] = kv
            tgt[..., 3] = s
            tgt[..., 4:] = marker
    return pool


def make_pool(layout, L, B, bs, slot_bytes, marker):
    return tag_pool(HostPool.zeros(layout, L, B, bs, slot_bytes), marker)


def check_tags(src, dst_before, dst, S, D):
    """Every slot of every receiver block D[i] carries sender block S[i]'s tag
    for the same (layer, K/V, slot); every other receiver slot is unchanged."""
    vd, vb = shaped(dst), shaped(dst_before)
    Dmap = {int(d): int(s) for s, d in zip(S, D)}
    for b in range(dst.num_blocks):
        for l in range(dst.num_layers):
            for kv in (0, 1):
                for s in range(dst.block_size):
                    got = get_slot(dst, vd, b, l, kv, s)
                    if b in Dmap:
                        assert tuple(got[:4]) == (Dmap[b], l, kv, s), (b, l, kv, s)
                        assert np.all(got[4:] == 0x51C0), (b, l, kv, s)
                    else:
                        assert np.array_equal(got, get_slot(dst_before, vb, b, l, kv, s))


@pytest.mark.parametrize("sl,dl", list(itertools.product(LAYOUTS, LAYOUTS)))
@pytest.mark.parametrize("fn", [transfer_ref, transfer_fast])
def test_tags_land_in_receiver_blocks(sl, dl, fn):
    rng = np.random.default_rng(7)
    L, bs, slot = 3, 4, 32
    src = make_pool(sl, L, 9, bs, slot, 0x51C0)
    dst = make_pool(dl, L, 11, bs, slot, 0xD57)
    before = dst.copy()
    S = rng.permutation(9)[:5]
    D = rng.permutation(11)[:5]
    fn(src, dst, S, D)
    check_tags(src, before, dst, S, D)


@pytest.mark.parametrize("fn", [transfer_ref, transfer_fast])
def test_layout_equivalence(fn):
    """Same logical K/V moved through any pair of layouts reads back the same."""
    rng = np.random.default_rng(3)
    L, bs, slot, n = 2, 4, 16, 6
    logical = rng.integers(0, 2**31, size=(n, L, 2, bs, slot // 4), dtype=np.int32)
    S = rng.permutation(10)[:n]
    D = rng.permutation(12)[:n]
    results = []
    for sl, dl in itertools.product(LAYOUTS, LAYOUTS):
        src = HostPool.zeros(sl, L, 10, bs, slot)
        dst = HostPool.zeros(dl, L, 12, bs, slot)
        vs = shaped(src)
        for i in range(n):
            for l in range(L):
                for kv in (0, 1):
                    if sl == LAYER_MAJOR:
                        vs[l][kv, S[i]] = logical[i, l, kv]
                    else:
                        vs[S[i], l, kv] = logical[i, l, kv]
        fn(src, dst, S, D)
        vd = shaped(dst)
        back = np.zeros_like(logical)
        for i in range(n):
            for l in range(L):
                for kv in (0, 1):
                    back[i, l, kv] = vd[l][kv, D[i]] if dl == LAYER_MAJOR else vd[D[i], l, kv]
        results.append(back)
    for r in results:
        assert np.array_equal(r, logical)


def test_contiguous_block_major_is_one_memcpy():
    """Both lists contiguous, both pools block-major: the result is one plain
    byte copy of n whole blocks (Figure 3's ideal case moves as one op)."""
    rng = np.random.default_rng(11)
    L, bs, slot, n = 4, 2, 48, 5
    B = 13
    src = HostPool.zeros(BLOCK_MAJOR, L, B, bs, slot)
    dst = HostPool.zeros(BLOCK_MAJOR, L, B, bs, slot)
    src.buffers[0][:] = rng.integers(0, 256, src.buffers[0].size, dtype=np.uint8)
    dst.buffers[0][:] = rng.integers(0, 256, dst.buffers[0].size, dtype=np.uint8)
    expect = bytearray(dst.buffers[0].tobytes())
    bb = L * 2 * bs * slot
    s0, d0 = 6, 2
    expect[d0 * bb:(d0 + n) * bb] = src.buffers[0].tobytes()[s0 * bb:(s0 + n) * bb]
    transfer_fast(src, dst, range(s0, s0 + n), range(d0, d0 + n))
    assert dst.buffers[0].tobytes() == bytes(expect)


def test_partial_last_block_tokens_arrive():
    """A request of T tokens that ends mid-block: every token t < T arrives,
    for every layer and K/V (the paper's per-token K and V of section 3.1)."""
    L, bs, slot = 2, 16, 16
    T = 40  # 2.5 blocks
    n = -(-T // bs)
    src = make_pool(LAYER_MAJOR, L, 8, bs, slot, 0x51C0)
    dst = make_pool(BLOCK_MAJOR, L, 8, bs, slot, 0xD57)
    S, D = [5, 2, 7], [1, 6, 3]
    transfer_fast(src, dst, S, D)
    vs, vd = shaped(src), shaped(dst)
    for t in range(T):
        for l in range(L):
            for kv in (0, 1):
                a = vs[l][kv, S[t // bs], t % bs]
                b = vd[D[t // bs], l, kv, t % bs]
                assert np.array_equal(a, b)
    assert n == 3


def test_batch_union_and_rejects_shared_receiver_block():
    L, bs, slot = 2, 2, 16
    src = make_pool(BLOCK_MAJOR, L, 8, bs, slot, 0x51C0)
    dst = make_pool(BLOCK_MAJOR, L, 8, bs, slot, 0xD57)
    before = dst.copy()
    tables = [([1, 2], [5, 6]), ([1, 7], [0, 3])]  # sender block 1 shared
    transfer_batch_fast(src, dst, tables)
    check_tags(src, before, dst, [1, 2, 1, 7], [5, 6, 0, 3])
    with pytest.raises(ValueError):
        transfer_batch_fast(src, dst, [([1], [5]), ([2], [5])])


def test_rejects_bad_tables():
    src = HostPool.zeros(BLOCK_MAJOR, 1, 4, 1, 16)
    dst = HostPool.zeros(BLOCK_MAJOR, 1, 4, 1, 16)
    for S, D in (([4], [0]), ([0], [4]), ([0, 1], [2, 2]), ([0], [0, 1]), ([-1], [0])):
        with pytest.raises(ValueError):
            transfer_fast(src, dst, S, D)


@settings(max_examples=200, deadline=None)
@given(st.data())
def test_loop_and_vectorised_forms_agree(data):
    L = data.draw(st.integers(1, 3))
    bs = data.draw(st.integers(1, 4))
    slot = 16 * data.draw(st.integers(1, 2))
    Bs = data.draw(st.integers(1, 8))
    Bd = data.draw(st.integers(1, 8))
    n = data.draw(st.integers(0, min(Bs, Bd)))
    sl = data.draw(st.sampled_from(LAYOUTS))
    dl = data.draw(st.sampled_from(LAYOUTS))
    seed = data.draw(st.integers(0, 2**32 - 1))
    rng = np.random.default_rng(seed)
    src = HostPool.zeros(sl, L, Bs, bs, slot)
    for buf in src.buffers:
        buf[:] = rng.integers(0, 256, buf.size, dtype=np.uint8)
    dst = HostPool.zeros(dl, L, Bd, bs, slot)
    for buf in dst.buffers:
        buf[:] = rng.integers(0, 256, buf.size, dtype=np.uint8)
    S = rng.permutation(Bs)[:n]
    D = rng.permutation(Bd)[:n]
    a, b = dst.copy(), dst.copy()
    transfer_ref(src, a, S, D)
    transfer_fast(src, b, S, D)
    for x, y in zip(a.buffers, b.buffers):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("sl,dl", list(itertools.product(LAYOUTS, LAYOUTS)))
def test_layer_subset_moves_only_those_layers(sl, dl):
    """The layer-at-a-time variant: a layer subset moves exactly those layers'
    K and V slots; every other receiver slot keeps its tag."""
    rng = np.random.default_rng(5)
    L, bs, slot = 5, 2, 32
    src = make_pool(sl, L, 7, bs, slot, 0x51C0)
    dst = make_pool(dl, L, 8, bs, slot, 0xD57)
    before = dst.copy()
    S, D = rng.permutation(7)[:4], rng.permutation(8)[:4]
    moved = [1, 3]
    transfer_fast(src, dst, S, D, layers=moved)
    vd, vb = shaped(dst), shaped(before)
    Dmap = {int(d): int(s) for s, d in zip(S, D)}
    for b in range(8):
        for l in range(L):
            for kv in (0, 1):
                for s in range(bs):
                    got = get_slot(dst, vd, b, l, kv, s)
                    if b in Dmap and l in moved:
                        assert tuple(got[:4]) == (Dmap[b], l, kv, s)
                    else:
                        assert np.array_equal(got, get_slot(before, vb, b, l, kv, s))


@pytest.mark.parametrize("fn", [transfer_ref, transfer_fast])
def test_layer_by_layer_composes_to_the_whole_transfer(fn):
    rng = np.random.default_rng(9)
    L, bs, slot = 4, 3, 16
    src = HostPool.zeros(BLOCK_MAJOR, L, 6, bs, slot)
    src.buffers[0][:] = rng.integers(0, 256, src.buffers[0].size, dtype=np.uint8)
    dst = HostPool.zeros(LAYER_MAJOR, L, 6, bs, slot)
    for buf in dst.buffers:
        buf[:] = rng.integers(0, 256, buf.size, dtype=np.uint8)
    S, D = rng.permutation(6)[:5], rng.permutation(6)[:5]
    whole, parts = dst.copy(), dst.copy()
    fn(src, whole, S, D)
    for l in reversed(range(L)):
        fn(src, parts, S, D, layers=[l])
    for a, b in zip(whole.buffers, parts.buffers):
        assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        fn(src, parts, S, D, layers=[L])


# ---- Eq. 5's claim: the restructured layout cuts transfer operations by 2L ------

def byte_address(pool: HostPool, b, l, kv, s):
    """(buffer, byte offset) of one slot, read off numpy's shaped views."""
    v = shaped(pool, np.uint8)
    if pool.layout == LAYER_MAJOR:
        buf, row = l, v[l][kv, b, s]
    else:
        buf, row = 0, v[b, l, kv, s]
    return buf, row.ctypes.data - pool.buffers[buf].ctypes.data


def contiguous_copies(src: HostPool, dst: HostPool, S, D) -> int:
    """The fewest contiguous (sender range -> receiver range) copies that
    perform the transfer's slot copies: the number of slot copies that no
    other slot copy continues on both sides at once."""
    sb = src.slot_bytes
    copies = set()
    for b_s, b_d in zip(S, D):
        for l in range(src.num_layers):
            for kv in (0, 1):
                for s in range(src.block_size):
                    copies.add(byte_address(src, int(b_s), l, kv, s) +
                               byte_address(dst, int(b_d), l, kv, s))
    return sum(1 for (i, o, j, p) in copies if (i, o - sb, j, p - sb) not in copies)


@pytest.mark.parametrize("seed", range(24))
def test_block_major_needs_one_copy_per_run_layer_major_2L(seed):
    """Section 3.3, Eq. 5: in the per-layer layout (L, 2, B, H) each aligned
    run of blocks is 2L separate ranges (one per layer and K/V); in the
    restructured layout (B, L, 2, H) it is one.  With ascending block lists
    (as the allocators hand out) the fewest contiguous copies are exactly
    the plan's runs block-major and 2L times as many layer-major; a fully
    contiguous request is one copy."""
    from oracle import plan_ref

    g = np.random.default_rng(300 + seed)
    L = int(g.integers(1, 4))
    bs = int(g.choice([1, 2, 4]))
    B = 40
    n = int(g.integers(1, 14))
    if seed % 6 == 0:                               # one contiguous run on both sides
        s0, d0 = int(g.integers(1, B - n - 1)), int(g.integers(1, B - n - 1))
        S, D = np.arange(s0, s0 + n), np.arange(d0, d0 + n)
    else:                                           # ascending, gaps at random
        S = np.sort(g.choice(np.arange(1, B - 1), n, replace=False))
        D = np.sort(g.choice(np.arange(1, B - 1), n, replace=False))
    runs = len(plan_ref(S.tolist(), D.tolist()))
    if seed % 6 == 0:
        assert runs == 1
    for layout, per_run in ((BLOCK_MAJOR, 1), (LAYER_MAJOR, 2 * L)):
        src = HostPool.zeros(layout, L, B, bs, 8)
        dst = HostPool.zeros(layout, L, B, bs, 8)
        assert contiguous_copies(src, dst, S, D) == per_run * runs, (layout, L, runs)
