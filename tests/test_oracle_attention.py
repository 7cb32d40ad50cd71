"""Pins for the decode-attention oracle (``oracle.attention``), CPU only.

The oracle gathers K and V slot by slot with the pool's own address formulas
and runs softmax attention per query head.  These tests build pools through
numpy's shaped views of the Eq. 5 layouts and check the oracle against
closed forms and against a separate dense computation (np.repeat for the
grouped heads, scipy's logsumexp for the normaliser, einsum for the products).
"""

import numpy as np
import pytest
from scipy.special import logsumexp

from oracle import BLOCK_MAJOR, LAYER_MAJOR, HostPool
from oracle.attention import decode_attention

LAYOUTS = [LAYER_MAJOR, BLOCK_MAJOR]


def to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float values to bfloat16 (nearest-even); returns uint16 patterns."""
    f = np.asarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def from_bf16(u: np.ndarray) -> np.ndarray:
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def build_pool(layout, L, B, bs, hkv, dh, layer, tables, kv_tokens):
    """Pool whose blocks hold, for layer `layer`, the bf16 patterns
    kv_tokens[r][kv, t, g, d] of each request's token t at its slot."""
    pool = HostPool.zeros(layout, L, B, bs, hkv * dh * 2)
    if layout == BLOCK_MAJOR:
        v = pool.buffers[0].view(np.uint16).reshape(B, L, 2, bs, hkv, dh)
    else:
        v = [b.view(np.uint16).reshape(2, B, bs, hkv, dh) for b in pool.buffers]
    for table, kvt in zip(tables, kv_tokens):
        for t in range(kvt.shape[1]):
            b, s = table[t // bs], t % bs
            for kv in (0, 1):
                if layout == BLOCK_MAJOR:
                    v[b, layer, kv, s] = kvt[kv, t]
                else:
                    v[layer][kv, b, s] = kvt[kv, t]
    return pool


def dense_reference(q, kv_f64, hq, hkv, scale):
    """Softmax attention on contiguous (2, T, hkv, dh) K/V of one request."""
    K = np.repeat(kv_f64[0], hq // hkv, axis=1)   # (T, hq, dh)
    V = np.repeat(kv_f64[1], hq // hkv, axis=1)
    s = scale * np.einsum("hd,thd->ht", q, K)
    p = np.exp(s - logsumexp(s, axis=1, keepdims=True))
    return np.einsum("ht,thd->hd", p, V)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_matches_dense_attention(layout):
    rng = np.random.default_rng(1)
    L, B, bs, hkv, dh, hq = 3, 12, 4, 2, 16, 8
    layer = 2
    lens = [1, 7, 13]
    # requests' blocks are distinct
    tables = []
    perm = rng.permutation(B)
    pos = 0
    for T in lens:
        nb = -(-T // bs)
        tables.append(perm[pos:pos + nb])
        pos += nb
    kv_bits = [to_bf16(rng.standard_normal((2, T, hkv, dh))) for T in lens]
    pool = build_pool(layout, L, B, bs, hkv, dh, layer, tables, kv_bits)
    q = from_bf16(to_bf16(rng.standard_normal((len(lens), hq, dh))))
    scale = 1 / np.sqrt(dh)
    got = decode_attention(pool, q, tables, lens, layer, hkv, dh, scale)
    for r, T in enumerate(lens):
        want = dense_reference(q[r], from_bf16(kv_bits[r]), hq, hkv, scale)
        np.testing.assert_allclose(got[r], want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_closed_forms(layout):
    rng = np.random.default_rng(2)
    L, B, bs, hkv, dh, hq = 2, 6, 2, 1, 8, 2
    scale = 0.5
    # one token: the output is that token's V exactly
    kv = to_bf16(rng.standard_normal((2, 1, hkv, dh)))
    pool = build_pool(layout, L, B, bs, hkv, dh, 1, [[4]], [kv])
    q = rng.standard_normal((1, hq, dh))
    got = decode_attention(pool, q, [[4]], [1], 1, hkv, dh, scale)
    assert np.array_equal(got[0, 0], from_bf16(kv[1, 0, 0]))
    # a zero query scores every key equally: the output is the mean of V
    T = 5
    kv = to_bf16(rng.standard_normal((2, T, hkv, dh)))
    pool = build_pool(layout, L, B, bs, hkv, dh, 0, [[3, 0, 5]], [kv])
    got = decode_attention(pool, np.zeros((1, hq, dh)), [[3, 0, 5]], [T], 0, hkv, dh, scale)
    np.testing.assert_allclose(got[0, 1], from_bf16(kv[1, :, 0]).mean(axis=0), rtol=1e-12)
    # a query that singles out key j returns V[j] (up to exp(-big) weights)
    keys = np.zeros((T, hkv, dh))
    for t in range(T):
        keys[t, 0, t] = 1.0
    kv = np.stack([to_bf16(keys), to_bf16(rng.standard_normal((T, hkv, dh)))])
    pool = build_pool(layout, L, B, bs, hkv, dh, 0, [[3, 0, 5]], [kv])
    j = 3
    qj = np.zeros((1, hq, dh))
    qj[0, :, j] = 200.0
    got = decode_attention(pool, qj, [[3, 0, 5]], [T], 0, hkv, dh, scale)
    np.testing.assert_allclose(got[0, 0], from_bf16(kv[1, j, 0]), rtol=1e-12, atol=1e-30)
    # scores far beyond exp's range (s = 1000) still give a finite, exact
    # answer: the normaliser is taken relative to the largest score
    qj[0, :, j] = 2000.0
    got = decode_attention(pool, qj, [[3, 0, 5]], [T], 0, hkv, dh, scale)
    assert np.all(np.isfinite(got))
    np.testing.assert_allclose(got[0, 0], from_bf16(kv[1, j, 0]), rtol=1e-12, atol=1e-30)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_query_heads_read_their_group_kv_head(layout):
    """Grouped KV heads: query head h reads KV head h // (Hq / Hkv).  With
    every token's V of KV head g equal to the constant g + 1, query head h's
    output is (h // G) + 1 whatever q and K are: the weights sum to one."""
    rng = np.random.default_rng(4)
    L, B, bs, hkv, dh, hq = 2, 8, 4, 4, 8, 8       # G = 2
    T = 11
    k = rng.standard_normal((T, hkv, dh))
    v = np.broadcast_to((np.arange(hkv) + 1.0)[None, :, None], (T, hkv, dh))
    kv = np.stack([to_bf16(k), to_bf16(v)])
    table = [5, 2, 7]
    pool = build_pool(layout, L, B, bs, hkv, dh, 1, [table], [kv])
    q = rng.standard_normal((1, hq, dh)) * 3.0
    got = decode_attention(pool, q, [table], [T], 1, hkv, dh, 0.7)
    want = (np.arange(hq) // (hq // hkv) + 1.0)[:, None] * np.ones(dh)
    np.testing.assert_allclose(got[0], want, rtol=1e-13, atol=0)


def test_block_relabelling_does_not_change_the_result():
    rng = np.random.default_rng(3)
    L, B, bs, hkv, dh, hq = 2, 10, 4, 2, 8, 4
    T = 15
    kv = to_bf16(rng.standard_normal((2, T, hkv, dh)))
    q = rng.standard_normal((1, hq, dh))
    outs = []
    for seed in range(3):
        table = np.random.default_rng(seed).permutation(B)[:4]
        pool = build_pool(BLOCK_MAJOR, L, B, bs, hkv, dh, 1, [table], [kv])
        outs.append(decode_attention(pool, q, [table], [T], 1, hkv, dh, 0.3))
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])


def test_rejects_bad_inputs():
    pool = HostPool.zeros(BLOCK_MAJOR, 1, 4, 2, 16)
    with pytest.raises(ValueError):
        decode_attention(pool, np.zeros((1, 2, 8)), [[0]], [1], 0, 2, 8, 1.0)  # slot size
    pool = HostPool.zeros(BLOCK_MAJOR, 1, 4, 2, 2 * 8 * 2)
    with pytest.raises(ValueError):
        decode_attention(pool, np.zeros((1, 3, 8)), [[0]], [1], 0, 2, 8, 1.0)  # 3 % 2
    with pytest.raises(ValueError):
        decode_attention(pool, np.zeros((1, 2, 8)), [[0]], [3], 0, 2, 8, 1.0)  # T > blocks
    with pytest.raises(ValueError):
        decode_attention(pool, np.zeros((1, 2, 8)), [[0]], [0], 0, 2, 8, 1.0)  # T = 0


# ---- the GPU tests' tolerance: it rejects plausible kernel errors -----------------
#
# tests/attn_tolerance.py bounds |kernel - oracle| per output element from the
# scales decode_attention_scales returns.  Here, in numpy, float32 evaluations
# of attention stand in for kernels: two that are right (the vector pass's
# arithmetic, and the matrix-core pass's weights carried as two bf16 parts)
# must pass, and two with bugs a loose bound would let through must fail.

from tests import attn_tolerance  # noqa: E402


def long_request(T, hkv, hq, dh, seed):
    """One request of T tokens on a one-layer block-major pool with N(0, 1)
    bf16 K, V and q; returns the oracle's output and scales, K and V as
    float32, q, and the scale."""
    from oracle.attention import decode_attention_scales, gather_kv

    rng = np.random.default_rng(seed)
    bs, B = 16, -(-T // 16)
    pool = HostPool.zeros(BLOCK_MAJOR, 1, B, bs, hkv * dh * 2)
    pool.buffers[0].view(np.uint16)[:] = to_bf16(rng.standard_normal(pool.buffers[0].size // 2))
    q = from_bf16(to_bf16(rng.standard_normal((1, hq, dh))))
    scale = 1 / np.sqrt(dh)
    table = list(range(B))
    out, w1, w2, s1 = decode_attention_scales(pool, q, [table], [T], 0, hkv, dh, scale)
    kv = gather_kv(pool, table, T, 0, hkv, dh).astype(np.float32)
    return out, w1, w2, s1, kv, q, scale


def float32_attention(kv, q, scale, hq, hkv, weights="f32", drop=None):
    """Attention of one request evaluated in float32: scores, exp2 weights
    against the largest score, their sum L, and sum_t w_t V_t / L with the
    weights w_t taken as float32 ('f32'), as bf16(p) + bf16(p - bf16(p))
    ('hi+lo'), or as bf16(p) alone ('hi').  `drop` leaves the 32 tokens from
    that index out of the weighted sum (a skipped tile)."""
    K, V = kv[0], kv[1]
    o = np.zeros((1, hq, K.shape[2]))
    for h in range(hq):
        g = h // (hq // hkv)
        s = (K[:, g, :] @ q[0, h].astype(np.float32)) * np.float32(scale * np.log2(np.e))
        p = np.exp2(s - s.max()).astype(np.float32)
        L = p.sum(dtype=np.float32)
        if drop is not None:
            p[drop:drop + 32] = 0
        hi = from_bf16(to_bf16(p)).astype(np.float32)
        if weights == "f32":
            num = p @ V[:, g, :]
        elif weights == "hi":
            num = hi @ V[:, g, :]
        else:
            lo = from_bf16(to_bf16(p - hi)).astype(np.float32)
            num = (hi @ V[:, g, :]).astype(np.float32) + (lo @ V[:, g, :]).astype(np.float32)
        o[0, h] = num.astype(np.float32) / L
    return o


HQ, HKV, DH = 8, 1, 128     # the matrix-core pass's shape (one 70B TP=8 share)


@pytest.mark.parametrize("T", [50, 300, 4097, 20000])
def test_tolerance_accepts_float32_evaluations(T):
    out, w1, w2, s1, kv, q, scale = long_request(T, HKV, HQ, DH, T)
    for weights, mc in (("f32", False), ("hi+lo", True)):
        got = float32_attention(kv, q, scale, HQ, HKV, weights)
        attn_tolerance.check(got, out, w1, w2, s1, [T], 256, mc)


@pytest.mark.parametrize("T", [300, 4097, 20000])
def test_tolerance_rejects_weights_carried_as_bf16_alone(T):
    """Dropping the low bf16 part of the matrix-core pass's weights (errors
    near 1e-4 at these lengths) fails the bound."""
    out, w1, w2, s1, kv, q, scale = long_request(T, HKV, HQ, DH, T)
    got = float32_attention(kv, q, scale, HQ, HKV, "hi")
    tol = attn_tolerance.tolerance(w1, w2, s1, [T], 256, True)
    assert np.any(np.abs(got - out) > tol)
    with pytest.raises(AssertionError):
        attn_tolerance.check(got, out, w1, w2, s1, [T], 256, True)


def test_tolerance_rejects_a_skipped_tile_in_every_head():
    """Leaving one interior 32-token tile out of a 32,000-token request
    fails the bound in every query head."""
    T = 32000
    out, w1, w2, s1, kv, q, scale = long_request(T, HKV, HQ, DH, 7)
    got = float32_attention(kv, q, scale, HQ, HKV, "hi+lo", drop=16000)
    tol = attn_tolerance.tolerance(w1, w2, s1, [T], 1024, True)
    bad = np.abs(got - out) > tol
    assert bad.any(axis=2).all(), bad.any(axis=2)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_error_scales_closed_forms(layout):
    """decode_attention_scales returns decode_attention's output and, for one
    token, w1 = |V|, w2 = 0 and s1 = scale * sum |q K|; for any request
    |o| <= w1 (a weighted mean of V under weights summing to one)."""
    from oracle.attention import decode_attention_scales

    rng = np.random.default_rng(8)
    L, B, bs, hkv, dh, hq = 2, 9, 4, 2, 8, 4
    kv1 = to_bf16(rng.standard_normal((2, 1, hkv, dh)))
    kvT = to_bf16(rng.standard_normal((2, 13, hkv, dh)))
    tables = [[6], [2, 0, 8, 5]]
    pool = build_pool(layout, L, B, bs, hkv, dh, 1, tables, [kv1, kvT])
    q = from_bf16(to_bf16(rng.standard_normal((2, hq, dh))))
    out, w1, w2, s1 = decode_attention_scales(pool, q, tables, [1, 13], 1, hkv, dh, 0.3)
    assert np.array_equal(out, decode_attention(pool, q, tables, [1, 13], 1, hkv, dh, 0.3))
    V1, K1 = from_bf16(kv1[1, 0]), from_bf16(kv1[0, 0])
    for h in range(hq):
        g = h // (hq // hkv)
        assert np.array_equal(w1[0, h], np.abs(V1[g]))
        assert np.all(w2[0, h] == 0)
        assert s1[0, h] == pytest.approx(0.3 * np.abs(K1[g]) @ np.abs(q[0, h]), rel=1e-15)
    assert np.all(np.abs(out) <= w1 * (1 + 1e-12))
    assert np.all(w2[1] > 0)
