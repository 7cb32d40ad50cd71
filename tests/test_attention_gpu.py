"""GPU parity of paged decode attention against the float64 oracle.

Every output element must lie within its own bound (tests/attn_tolerance.py):
the float32 rounding of its scores, weights and sums, scaled by what the
oracle returns beside the output -- sum_t p_t |V_t|, the spread
sqrt(sum_t p_t^2 (V_t - o)^2) and the largest score magnitude -- plus, in the
matrix-core pass (8 query heads per KV head, head_dim 128), the relative
2^-16 of weights carried into P.V as two bfloat16 parts.  Each test prints
its worst error and its worst ratio of error to bound.
"""

import gc
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.attention import decode_attention_scales
from paper_2504_03775_amd import flowkv as fk
from workloads import Geometry, make_device_pool, recipes
from tests import attn_tolerance
from tests.gpu_helpers import BM, LM, download_blocks

pytestmark = pytest.mark.gpu
NAMES = {LM: "layer", BM: "block"}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bf16_to_f64(t: torch.Tensor) -> np.ndarray:
    u = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16).astype(np.uint32)
    return (u << 16).view(np.float32).astype(np.float64)


def run_case(geom: Geometry, layout, pool_blocks, lens, q_heads, seed, split=0, layer=None,
             max_seq=None, check=True, host_lens=False):
    g = np.random.default_rng(seed)
    layer = int(g.integers(geom.num_layers)) if layer is None else layer
    pool = fk.KVPool(layout, make_device_pool(geom, layout, pool_blocks, "cuda", seed))
    bs = geom.block_size
    nblk = [max(1, -(-T // bs)) for T in lens]
    perm = g.permutation(pool_blocks)
    assert sum(nblk) <= pool_blocks
    tables, pos = [], 0
    for k in nblk:
        tables.append(perm[pos:pos + k].astype(np.int32))
        pos += k
    max_blocks = max(nblk)
    tab = np.full((len(lens), max_blocks), -1, dtype=np.int32)
    for r, t in enumerate(tables):
        tab[r, :len(t)] = t
    n = len(lens)
    q = torch.randn((n, q_heads, geom.head_dim), generator=torch.Generator("cuda").manual_seed(
        seed + 7), device="cuda").to(torch.bfloat16)
    max_seq = max(lens) if max_seq is None else max_seq
    ws = torch.empty(fk.flowkv_decode_attention_workspace(n, q_heads, geom.head_dim, max_seq,
                                                          split), dtype=torch.uint8, device="cuda")
    out = torch.full((n, q_heads, geom.head_dim), float("nan"), dtype=torch.float32, device="cuda")
    scale = 1.0 / np.sqrt(geom.head_dim)
    fk.flowkv_decode_attention(pool, layer, q, torch.as_tensor(tab, device="cuda"),
                               torch.as_tensor(np.asarray(lens, np.int32), device="cuda"),
                               max_seq, scale, out, ws, split,
                               seq_lens_host=np.asarray(lens, np.int32) if host_lens else None)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    if not check:
        return got, None
    # oracle on a compact host copy of exactly the blocks the requests use
    used = np.concatenate(tables)
    host = download_blocks(pool, used)
    lut = {int(b): i for i, b in enumerate(used)}
    ctabs = [[lut[int(b)] for b in t] for t in tables]
    eff = [min(T, max_seq) for T in lens]
    want, w1, w2, s1 = decode_attention_scales(host, bf16_to_f64(q), ctabs, eff, layer,
                                               geom.kv_heads, geom.head_dim, scale)
    err, ratio = attn_tolerance.check(
        got, want, w1, w2, s1, eff, split or fk.flowkv_decode_attention_split(n, max_seq),
        attn_tolerance.matrix_core_pass(q_heads, geom.kv_heads, geom.head_dim))
    say(f"  worst error / bound {ratio:.3f}")
    return got, err


SHAPES = [  # (layers, kv heads, head dim, block size, q heads)
    (2, 2, 64, 16, 4), (3, 1, 128, 16, 8), (2, 8, 128, 16, 32), (1, 4, 64, 5, 4),
    (2, 2, 128, 1, 16), (4, 1, 64, 7, 1),
]


@pytest.mark.parametrize("seed", range(18))
def test_random_cases_against_oracle(seed):
    L, hkv, dh, bs, hq = SHAPES[seed % len(SHAPES)]
    layout = (LM, BM)[seed % 2]
    geom = Geometry(f"attn{seed}", L, hkv, dh, bs, "bfloat16")
    g = np.random.default_rng(100 + seed)
    n = int(g.integers(1, 5))
    lens = [int(x) for x in g.integers(1, 700, size=n)]
    if seed % 3 == 0:
        lens[0] = 1
    split = [0, 16, 64, 1, 300, 1024][seed % 6]
    blocks = sum(max(1, -(-T // bs)) for T in lens) + int(g.integers(0, 20))
    say(f"attn seed={seed} L={L} Hkv={hkv} Hq={hq} Dh={dh} bs={bs} {NAMES[layout]} "
        f"lens={lens} split={split}")
    _, err = run_case(geom, layout, blocks, lens, hq, seed, split)
    say(f"  max error {err:.2e}")


@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
def test_llama8b_geometry_long_requests(layout):
    """Llama-3-8B geometry (32 query heads on 8 KV heads, head_dim 128, block
    16): requests of 1 to 20,000 tokens, ragged last blocks."""
    geom = Geometry("llama8b", 32, 8, 128, 16, "bfloat16")
    lens = [20000, 1, 13000, 4097, 16]
    blocks = sum(-(-T // 16) for T in lens) + 64
    say(f"8b attention {NAMES[layout]} lens={lens}")
    _, err = run_case(geom, layout, blocks, lens, 32, 11, layer=17)
    say(f"  max error {err:.2e}")


@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
def test_blocks_beyond_4_gib_into_the_pool(layout):
    """A 140,000-block pool of 8.5 GiB (one layer, 32 KiB chunks) with the
    requests' blocks drawn at random from all of it: most K/V reads sit past
    4 GiB from the pool's base (in the layer-major layout the V half starts
    at 4.3 GiB), so block offsets must be formed in 64 bits."""
    geom = Geometry("far", 1, 8, 128, 16, "bfloat16")
    B = 140_000
    assert B * geom.block_bytes > 2**32 and B * geom.chunk_bytes > 2**32
    lens = [2000, 1500, 777]
    say(f"far blocks {NAMES[layout]}: pool {B * geom.block_bytes / 2**30:.1f} GiB")
    _, err = run_case(geom, layout, B, lens, 32, 31, layer=0)
    say(f"  max error {err:.2e}")


def test_llama70b_share_geometry():
    """One GPU's share of Llama-3-70B at TP=8: 1 KV head, 8 query heads."""
    geom = Geometry("llama70b-tp8", 80, 1, 128, 16, "bfloat16")
    lens = [32000, 777]
    blocks = sum(-(-T // 16) for T in lens) + 16
    _, err = run_case(geom, BM, blocks, lens, 8, 12, layer=79)
    say(f"  max error {err:.2e}")


def test_both_layouts_give_identical_outputs():
    """The same K/V stored in the two Eq. 5 layouts gives bit-identical
    outputs: the kernel's arithmetic does not depend on the layout."""
    geom = Geometry("same", 4, 2, 128, 16, "bfloat16")
    B, layer, hq = 60, 2, 8
    bm = make_device_pool(geom, BM, B, "cuda", 9)[0]            # (B, L, 2, bs, Hkv, Dh)
    lm = [bm[:, l].transpose(0, 1).contiguous() for l in range(geom.num_layers)]  # (2, B, ...)
    pools = [fk.KVPool(BM, [bm]), fk.KVPool(LM, lm)]
    lens = [333, 700]
    tab = torch.as_tensor(np.array([np.arange(0, 44), np.arange(16, 60)], np.int32), device="cuda")
    sl = torch.as_tensor(np.asarray(lens, np.int32), device="cuda")
    q = torch.randn((2, hq, 128), device="cuda").to(torch.bfloat16)
    outs = []
    for pool in pools:
        ws = torch.empty(fk.flowkv_decode_attention_workspace(2, hq, 128, 700), dtype=torch.uint8,
                         device="cuda")
        out = torch.empty((2, hq, 128), dtype=torch.float32, device="cuda")
        fk.flowkv_decode_attention(pool, layer, q, tab, sl, 700, 0.088, out, ws)
        torch.cuda.synchronize()
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1])


HOST_LENS_SHAPES = [  # (layers, kv heads, head dim, block size, q heads): every pass
    (2, 2, 64, 16, 2), (2, 2, 64, 16, 4), (2, 1, 64, 16, 8), (2, 4, 128, 16, 4),
    (2, 2, 128, 16, 16), (2, 1, 128, 7, 1), (2, 2, 128, 16, 4),
]


@pytest.mark.parametrize("shape", range(len(HOST_LENS_SHAPES)))
@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
def test_host_lengths_give_identical_outputs(layout, shape):
    """Lengths passed on the host travel in the kernel arguments: splits past
    a request's end then leave no record and the merge reads only the live
    ones.  The arithmetic is the same, so the outputs are bit-identical to the
    device-lengths call, for every pass (vector at 1, 2, 4 and 8 query heads
    per KV head, both head dims; matrix-core at 8 over head_dim 128), mixed
    lengths with empty requests, lengths past max_seq_len and past the block
    table; and they pass the oracle."""
    L, hkv, dh, bs, hq = HOST_LENS_SHAPES[shape]
    geom = Geometry(f"hl{shape}", L, hkv, dh, bs, "bfloat16")
    g = np.random.default_rng(700 + shape)
    lens = [int(x) for x in g.integers(1, 900, size=5)] + [0, 1, 1500]
    split = [0, 64, 128, 300][shape % 4]
    max_seq = 1200          # the 1,500-token request is cut at 1,200 tokens
    blocks = sum(max(1, -(-T // bs)) for T in lens) + 8
    say(f"host lengths {NAMES[layout]} L={L} Hkv={hkv} Hq={hq} Dh={dh} bs={bs} lens={lens} "
        f"split={split}")
    dev_out, _ = run_case(geom, layout, blocks, lens, hq, 40 + shape, split, max_seq=max_seq,
                          check=False)
    host_out, _ = run_case(geom, layout, blocks, lens, hq, 40 + shape, split, max_seq=max_seq,
                           check=False, host_lens=True)
    assert np.array_equal(dev_out, host_out, equal_nan=False)
    assert np.all(host_out[5] == 0)          # the empty request
    # the oracle takes no empty request: the same lengths without it
    live = lens[:5] + lens[6:]
    _, err = run_case(geom, layout, blocks, live, hq, 40 + shape, split, max_seq=max_seq,
                      host_lens=True)
    say(f"  identical to the device-lengths call; max error {err:.2e}")


@pytest.mark.parametrize("n_req", [fk.ATTN_INLINE_LENS, fk.ATTN_INLINE_LENS + 1])
def test_host_lengths_at_the_argument_capacity(n_req):
    """At most ATTN_INLINE_LENS host lengths ride in the kernel arguments;
    one request more and the call reads the lengths on the device instead.
    Either way the outputs equal the device-lengths call bit for bit and
    pass the oracle."""
    geom = Geometry("cap", 2, 2, 64, 16, "bfloat16")
    g = np.random.default_rng(n_req)
    lens = [int(x) for x in g.integers(1, 48, size=n_req)]
    blocks = sum(-(-T // 16) for T in lens) + 4
    say(f"host lengths at capacity: {n_req} requests, {sum(lens)} tokens")
    dev_out, _ = run_case(geom, BM, blocks, lens, 4, 90, check=False)
    host_out, err = run_case(geom, BM, blocks, lens, 4, 90, host_lens=True)
    assert np.array_equal(dev_out, host_out)
    say(f"  identical to the device-lengths call; max error {err:.2e}")


@pytest.mark.parametrize("hq,hkv,dh", [(8, 1, 128), (4, 2, 64)],
                         ids=["matrix-core-pass", "vector-pass"])
def test_most_requests_one_token_each(hq, hkv, dh):
    """65,535 requests (the grid's limit) of one token each: a softmax over
    one token weighs it exactly 1, so every output is that token's V, bit
    for bit (bf16 values are exact in float32), gathered here with torch's
    own indexing."""
    n = 65535
    geom = Geometry("many", 1, hkv, dh, 16, "bfloat16")
    B = n + 3
    g = np.random.default_rng(5)
    blk = g.permutation(B)[:n].astype(np.int32)
    pool = fk.KVPool(BM, make_device_pool(geom, BM, B, "cuda", 5))
    tab = torch.as_tensor(blk.reshape(n, 1), device="cuda")
    lens = torch.ones(n, dtype=torch.int32, device="cuda")
    q = torch.randn((n, hq, dh), generator=torch.Generator("cuda").manual_seed(6),
                    device="cuda").to(torch.bfloat16)
    ws = torch.empty(fk.flowkv_decode_attention_workspace(n, hq, dh, 1), dtype=torch.uint8,
                     device="cuda")
    out = torch.full((n, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
    say(f"{n} one-token requests, {hq} query heads on {hkv}, head_dim {dh}")
    fk.flowkv_decode_attention(pool, 0, q, tab, lens, 1, 0.1, out, ws)
    torch.cuda.synchronize()
    # block-major pool: (B, L, 2, bs, Hkv, Dh); V of layer 0, slot 0
    v = pool.tensors[0].view(B, 1, 2, 16, hkv, dh)[torch.as_tensor(blk.astype(np.int64),
                                                                   device="cuda"), 0, 1, 0]
    want = v.float().repeat_interleave(hq // hkv, dim=1)   # query head h reads KV head h // G
    assert torch.equal(out, want)


@pytest.mark.parametrize("host_lens", [False, True], ids=["lengths-on-device", "lengths-on-host"])
@pytest.mark.parametrize("hq,hkv,dh", [(8, 1, 128), (4, 2, 64)],
                         ids=["matrix-core-pass", "vector-pass"])
def test_most_splits_constant_values(hq, hkv, dh, host_lens):
    """One 65,535-token request in one-token splits: 65,535 pass-1 workgroups
    per KV head (the grid's limit) and as many records for the merge.  With a
    zero query every weight is exactly 1, and with V constant per KV head
    every partial sum is an exact multiple of that constant, so each output
    is the constant, bit for bit."""
    T = 65535
    geom = Geometry("splits", 1, hkv, dh, 16, "bfloat16")
    B = -(-T // 16) + 2
    pool = fk.KVPool(BM, make_device_pool(geom, BM, B, "cuda", 8))
    consts = torch.tensor([0.75, -3.0][:hkv], dtype=torch.bfloat16, device="cuda")
    kv = pool.tensors[0].view(B, 1, 2, 16, hkv, dh)
    kv[:, 0, 1] = consts.view(1, 1, hkv, 1)          # V of every slot: its head's constant
    blk = np.random.default_rng(8).permutation(B)[:-(-T // 16)].astype(np.int32)
    tab = torch.as_tensor(blk.reshape(1, -1), device="cuda")
    lens = torch.tensor([T], dtype=torch.int32, device="cuda")
    q = torch.zeros((1, hq, dh), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(fk.flowkv_decode_attention_workspace(1, hq, dh, T, 1), dtype=torch.uint8,
                     device="cuda")
    out = torch.full((1, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
    say(f"one {T}-token request in {T} splits, {hq} query heads on {hkv}, head_dim {dh}")
    fk.flowkv_decode_attention(pool, 0, q, tab, lens, T, 0.1, out, ws, 1,
                               seq_lens_host=np.array([T], np.int32) if host_lens else None)
    torch.cuda.synchronize()
    want = consts.float().repeat_interleave(hq // hkv).view(1, hq, 1).expand(1, hq, dh)
    assert torch.equal(out, want)


@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
@pytest.mark.parametrize("layer", [0, fk.MAX_LAYERS - 1], ids=["first-layer", "last-layer"])
def test_deepest_pool_first_and_last_layer(layout, layer):
    """Pools of the most layers the library takes: the last layer's base
    pointer (layer-major) or its offset inside a block (block-major) against
    the oracle."""
    geom = Geometry("deep", fk.MAX_LAYERS, 2, 64, 16, "bfloat16")
    say(f"{fk.MAX_LAYERS}-layer {NAMES[layout]} pool, layer {layer}")
    run_case(geom, layout, 24, [37, 150, 1], 4, 11, layer=layer)


def test_pool_of_another_type_is_refused():
    """The kernels read bf16 K/V; an fp16 pool of the same byte size (the
    transfer moves either) is refused by the binding, not misread."""
    geom = Geometry("fp16", 2, 2, 64, 16, "float16")
    pool = fk.KVPool(BM, make_device_pool(geom, BM, 8, "cuda", 1))
    q = torch.zeros((1, 4, 64), dtype=torch.bfloat16, device="cuda")
    tab = torch.zeros((1, 1), dtype=torch.int32, device="cuda")
    lens = torch.ones(1, dtype=torch.int32, device="cuda")
    out = torch.empty((1, 4, 64), dtype=torch.float32, device="cuda")
    ws = torch.empty(fk.flowkv_decode_attention_workspace(1, 4, 64, 1), dtype=torch.uint8,
                     device="cuda")
    with pytest.raises(ValueError, match="bfloat16"):
        fk.flowkv_decode_attention(pool, 0, q, tab, lens, 1, 0.1, out, ws)
    with pytest.raises(ValueError, match="bfloat16"):
        fk.flowkv_decode_attention_noalloc(pool, 0, q, tab, lens, 1, 0.1, out)


def test_length_caps_and_empty_request():
    """Tokens past max_seq_len are not read; a zero-length request gives zeros."""
    geom = Geometry("caps", 2, 2, 64, 16, "bfloat16")
    got, err = run_case(geom, BM, 40, [300, 120], 4, 3, max_seq=200)
    assert err is not None
    z, _ = run_case(geom, LM, 40, [0, 50], 4, 4, check=False)
    assert np.all(z[0] == 0)
    # max_seq_len 0: no token is read, every output is zero, and the
    # workspace has 0 bytes (a NULL pointer is accepted)
    z, _ = run_case(geom, BM, 40, [30, 50], 4, 5, max_seq=0, check=False)
    assert np.all(z == 0)


@pytest.mark.parametrize("hq", [8, 16], ids=["vector-pass", "matrix-core-pass"])
@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
def test_blocks_outside_the_pool_contribute_nothing(layout, hq):
    """A block ID outside the pool (negative or >= the pool's size) inside a
    request's length is skipped: the output equals attention over the tokens
    of the valid blocks alone (attention does not depend on token order).
    8 query heads on 2 KV heads run the vector pass, 16 the matrix-core pass
    (where a hole falls inside a 32-token tile, split 64: two tiles)."""
    geom = Geometry("holes", 3, 2, 128, 16, "bfloat16")
    B, layer, bs = 50, 1, 16
    pool = fk.KVPool(layout, make_device_pool(geom, layout, B, "cuda", 21))
    g = np.random.default_rng(21)
    perm = g.permutation(B).astype(np.int32)
    full = [perm[0:10], perm[10:30]]           # 10 and 20 blocks
    lens = [10 * bs - 5, 20 * bs - 9]          # ragged last blocks
    holes = [[3], [0, 7, 8, 15]]               # positions replaced, never the last block
    bad = [-1, B, B + 1000, -7]
    tab = np.full((2, 20), -1, dtype=np.int32)
    valid_tables, valid_lens = [], []
    for r in range(2):
        t = full[r].copy()
        for i, pos in enumerate(holes[r]):
            t[pos] = bad[i % len(bad)]
        tab[r, :len(t)] = t
        keep = [int(b) for b in t if 0 <= b < B]
        valid_tables.append(keep)
        valid_lens.append(lens[r] - bs * len(holes[r]))
    q = torch.randn((2, hq, 128), generator=torch.Generator("cuda").manual_seed(5),
                    device="cuda").to(torch.bfloat16)
    max_seq = max(lens)
    ws = torch.empty(fk.flowkv_decode_attention_workspace(2, hq, 128, max_seq, 64),
                     dtype=torch.uint8, device="cuda")
    out = torch.empty((2, hq, 128), dtype=torch.float32, device="cuda")
    scale = 1.0 / np.sqrt(128)
    fk.flowkv_decode_attention(pool, layer, q, torch.as_tensor(tab, device="cuda"),
                               torch.as_tensor(np.asarray(lens, np.int32), device="cuda"),
                               max_seq, scale, out, ws, 64)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    used = np.array(sorted({b for t in valid_tables for b in t}), dtype=np.int64)
    host = download_blocks(pool, used)
    lut = {int(b): i for i, b in enumerate(used)}
    want, w1, w2, s1 = decode_attention_scales(
        host, bf16_to_f64(q), [[lut[b] for b in t] for t in valid_tables], valid_lens, layer,
        geom.kv_heads, geom.head_dim, scale)
    # the kernel's chains run over the full lengths, holes included
    err, ratio = attn_tolerance.check(got, want, w1, w2, s1, lens, 64,
                                      attn_tolerance.matrix_core_pass(hq, 2, 128))
    say(f"holes {NAMES[layout]} hq={hq}: max error {err:.2e}, worst error / bound {ratio:.3f}")


@pytest.mark.parametrize("layout", [BM, LM], ids=lambda x: NAMES[x])
@pytest.mark.parametrize("split", [32, 64, 128, 160, 256, 384, 1024])
def test_matrix_core_pass_tile_counts(layout, split):
    """The matrix-core pass (8 query heads per KV head, head_dim 128) takes
    32-token tiles, 4 waves a workgroup, and issues each tile's loads one tile
    ahead into alternating buffers.  Lengths around tile and step edges
    (1, 31..33, 127..129, 255, 257, 1000) under these split lengths give waves
    0 to 8 tiles, odd and even counts, full and ragged last tiles."""
    geom = Geometry("tiles", 2, 2, 128, 16, "bfloat16")
    lens = [1, 31, 32, 33, 127, 128, 129, 255, 257, 1000]
    blocks = sum(-(-T // 16) for T in lens) + 8
    say(f"matrix-core tiles {NAMES[layout]} split={split}")
    _, err = run_case(geom, layout, blocks, lens, 16, 40 + split, split, layer=1)
    say(f"  max error {err:.2e}")


# ---- the bench's attention workloads at full size ------------------------------

def download_layer(pool: fk.KVPool, ids, layer: int) -> oracle.HostPool:
    """K and V of one layer of blocks `ids` of a device pool (either layout),
    as a compact one-layer block-major host pool (block i = block ids[i])."""
    idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device=pool.device)
    slot = pool.kv_heads * pool.head_dim * pool.elem_bytes
    hp = oracle.HostPool.zeros(BM, 1, len(ids), pool.block_size, slot)
    out = hp.buffers[0].reshape(len(ids), -1)
    for lo in range(0, len(ids), 4096):
        if pool.layout == BM:   # (B, L, 2, bs, Hkv, Dh) -> (k, 2, bs, Hkv, Dh)
            sub = pool.tensors[0].index_select(0, idx[lo:lo + 4096])[:, layer].contiguous()
        else:                   # layer tensor (2, B, bs, Hkv, Dh) -> (k, 2, bs, Hkv, Dh)
            sub = pool.tensors[layer].index_select(1, idx[lo:lo + 4096]).transpose(0, 1)
            sub = sub.contiguous()
        out[lo:lo + 4096] = sub.view(torch.uint8).reshape(sub.shape[0], -1).cpu().numpy()
    return hp


BENCH_ATTN = {  # as bench.py --op attention builds them: recipe, query heads
    "batch": (lambda mk: recipes.batch32(mk, "segment"), 32),
    "8b": (lambda mk: recipes.llama8b_13k(mk, "segment"), 32),
    "70b": (lambda mk: recipes.llama70b_tp8(mk, "segment"), 8),
}


@pytest.mark.parametrize("name,layout", [(w, BM) for w in sorted(BENCH_ATTN)] + [("batch", LM)],
                         ids=lambda x: NAMES.get(x, x) if isinstance(x, int) else x)
def test_bench_attention_workloads_full_size(name, layout):
    """Each --op attention workload exactly as bench.py runs it: its recipe's
    block lists, the full receiver pool (block-major, and for the batch also
    layer-major as --layout layer runs it; seeded N(0,1)), every request in
    one call with the lengths on the host, the default split, the middle
    layer; the outputs of a sample of requests (shortest, longest and two
    between) against the oracle on just those requests' blocks of that
    layer, and every output against the same call with the lengths read on
    the device."""
    make, q_heads = BENCH_ATTN[name]
    wl = make(lambda P, pol, seed: fk.Allocator(P, pol, seed))
    geom = wl.geom
    gc.collect()
    torch.cuda.empty_cache()
    pool = fk.KVPool(layout, make_device_pool(geom, layout, wl.dst_pool_blocks, "cuda", 1))
    lens = np.asarray(wl.tokens, dtype=np.int32)
    n, max_seq = len(lens), int(lens.max())
    max_blocks = max(len(d) for _, d in wl.tables)
    tab = np.full((n, max_blocks), -1, dtype=np.int32)
    for r, (_, d) in enumerate(wl.tables):
        tab[r, :len(d)] = d
    q = torch.randn((n, q_heads, geom.head_dim), generator=torch.Generator("cuda").manual_seed(3),
                    device="cuda").to(torch.bfloat16)
    layer, scale = geom.num_layers // 2, 1.0 / geom.head_dim ** 0.5
    ws = torch.empty(fk.flowkv_decode_attention_workspace(n, q_heads, geom.head_dim, max_seq),
                     dtype=torch.uint8, device="cuda")
    out = torch.full((n, q_heads, geom.head_dim), float("nan"), dtype=torch.float32, device="cuda")
    fk.flowkv_decode_attention(pool, layer, q, torch.as_tensor(tab, device="cuda"),
                               torch.as_tensor(lens, device="cuda"), max_seq, scale, out, ws,
                               seq_lens_host=lens)
    torch.cuda.synchronize()
    # the same call with the lengths read on the device: bit-identical
    out_dev = torch.empty_like(out)
    fk.flowkv_decode_attention(pool, layer, q, torch.as_tensor(tab, device="cuda"),
                               torch.as_tensor(lens, device="cuda"), max_seq, scale, out_dev, ws)
    torch.cuda.synchronize()
    assert torch.equal(out, out_dev)
    del out_dev
    order = np.argsort(lens, kind="stable")
    pick = sorted({int(order[0]), int(order[-1]), int(order[n // 3]), int(order[(2 * n) // 3])})
    say(f"{name}: {n} requests, {int(lens.sum())} tokens, pool {wl.dst_pool_blocks} blocks, "
        f"split {fk.flowkv_decode_attention_split(n, max_seq)}; checking requests {pick}")
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    ids = np.concatenate([wl.tables[r][1] for r in pick]).astype(np.int64)
    host = download_layer(pool, ids, layer)
    ctabs, pos = [], 0
    for r in pick:
        k = len(wl.tables[r][1])
        ctabs.append(list(range(pos, pos + k)))
        pos += k
    picked = [int(lens[r]) for r in pick]
    want, w1, w2, s1 = decode_attention_scales(host, bf16_to_f64(q[pick]), ctabs, picked, 0,
                                               geom.kv_heads, geom.head_dim, scale)
    err, ratio = attn_tolerance.check(
        got[pick], want, w1, w2, s1, picked, fk.flowkv_decode_attention_split(n, max_seq),
        attn_tolerance.matrix_core_pass(q_heads, geom.kv_heads, geom.head_dim))
    say(f"  max error {err:.2e}, worst error / bound {ratio:.3f}")
    del pool
    torch.cuda.empty_cache()
