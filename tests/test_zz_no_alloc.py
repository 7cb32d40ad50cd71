"""The allocation-free decode attention (flowkv_decode_attention_noalloc)
against the workspace form (flowkv_decode_attention), through the C ABI.

Both run the same kernels on the same inputs, so their outputs must be
bit-identical.  Each case makes two calls in a row on one GPU, the second with
a smaller input, so the second runs over scratch contents the first left
behind; a third case fills the scratch to within a few percent of its size.
"""

import sys

import numpy as np
import pytest
import torch

from paper_2504_03775_amd import flowkv as fk
from workloads import Geometry, make_device_pool
from tests.gpu_helpers import BM, LM

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def inputs(geom, layout, lens, q_heads, seed, split=0):
    g = np.random.default_rng(seed)
    bs = geom.block_size
    nblk = [max(1, -(-T // bs)) for T in lens]
    B = sum(nblk) + 8
    pool = fk.KVPool(layout, make_device_pool(geom, layout, B, "cuda", seed))
    perm = g.permutation(B).astype(np.int32)
    tab = np.full((len(lens), max(nblk)), -1, dtype=np.int32)
    pos = 0
    for r, k in enumerate(nblk):
        tab[r, :k] = perm[pos:pos + k]
        pos += k
    q = torch.randn((len(lens), q_heads, geom.head_dim),
                    generator=torch.Generator("cuda").manual_seed(seed), device="cuda")
    return (pool, q.to(torch.bfloat16), torch.as_tensor(tab, device="cuda"),
            torch.as_tensor(np.asarray(lens, np.int32), device="cuda"), max(lens), split)


def both(geom, args, scale, layer):
    pool, q, tab, sl, max_seq, split = args
    n, hq, dh = q.shape
    ws = torch.empty(fk.flowkv_decode_attention_workspace(n, hq, dh, max_seq, split),
                     dtype=torch.uint8, device="cuda")
    want = torch.full((n, hq, dh), float("nan"), dtype=torch.float32, device="cuda")
    got = torch.full_like(want, float("nan"))
    got_host = torch.full_like(want, float("nan"))
    fk.flowkv_decode_attention(pool, layer, q, tab, sl, max_seq, scale, want, ws, split)
    fk.flowkv_decode_attention_noalloc(pool, layer, q, tab, sl, max_seq, scale, got, split)
    # and with the lengths on the host (carried in the kernel arguments)
    fk.flowkv_decode_attention_noalloc(pool, layer, q, tab, sl, max_seq, scale, got_host, split,
                                       seq_lens_host=sl.cpu().numpy())
    torch.cuda.synchronize()
    assert torch.equal(got.cpu(), got_host.cpu()), "host-lengths call differs"
    return want.cpu(), got.cpu()


CASES = {
    # vector pass: 32 query heads on 8 KV heads (Llama-3-8B), block-major
    "vector-pass": (Geometry("8b", 4, 8, 128, 16, "bfloat16"), BM, 32,
                    [[5000, 1, 2345, 777], [700]]),
    # matrix-core pass: 8 query heads on 1 KV head (the 70B TP=8 share), layer-major
    "matrix-core-pass": (Geometry("70b", 3, 1, 128, 16, "bfloat16"), LM, 8,
                         [[3000, 40, 4097], [100]]),
    # head_dim 64, two query heads per KV head, odd block size
    "head-dim-64": (Geometry("d64", 2, 4, 64, 7, "bfloat16"), BM, 8, [[1500, 333], [65]]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_noalloc_matches_workspace_form_on_two_calls(name):
    geom, layout, hq, calls = CASES[name]
    for i, lens in enumerate(calls):
        say(f"no-alloc attention {name} call {i + 1}: lens={lens}")
        want, got = both(geom, inputs(geom, layout, lens, hq, 50 + i), 1 / np.sqrt(geom.head_dim),
                         geom.num_layers - 1)
        assert torch.isfinite(want).all()
        assert torch.equal(want, got), f"call {i + 1}: outputs differ"


def test_noalloc_fills_the_scratch_then_a_small_call():
    """12 requests of 20,000 tokens with 32 query heads at split 256 need
    12 x 32 x 79 x 130 floats = 15.8 MB of partial results, 94% of the
    scratch; then a 1-request call must still agree with the workspace form."""
    geom = Geometry("8b-1layer", 1, 8, 128, 16, "bfloat16")
    lens = [20000] * 12
    need = fk.flowkv_decode_attention_workspace(12, 32, 128, 20000, 256)
    assert 0.9 * fk.ATTN_SCRATCH_BYTES < need <= fk.ATTN_SCRATCH_BYTES
    say(f"no-alloc attention, scratch nearly full: {need} of {fk.ATTN_SCRATCH_BYTES} bytes")
    want, got = both(geom, inputs(geom, BM, lens, 32, 60, split=256), 0.088, 0)
    assert torch.equal(want, got)
    say("no-alloc attention, then one 333-token request")
    want, got = both(geom, inputs(geom, BM, [333], 32, 61, split=256), 0.088, 0)
    assert torch.equal(want, got)
