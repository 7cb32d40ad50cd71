"""The library's launches captured in a HIP graph and replayed (GPU).

Callers that cannot allocate -- code under graph capture among them -- use
flowkv_decode_attention_noalloc, and a transfer whose plan rides in the
kernel arguments needs no device buffer either.  Both are captured here with
torch's graph capture (hipStreamBeginCapture underneath), then replayed
several times with eager work on the same memory between replays; every
replay must reproduce the eager result exactly.  Lengths passed on the host
and the plan's records are copied into the kernel arguments at capture, so a
replay repeats the captured call.
"""

import sys

import numpy as np
import pytest
import torch

from paper_2504_03775_amd import flowkv as fk
from workloads import Geometry, make_device_pool

pytestmark = pytest.mark.gpu

BM, LM = fk.LAYOUT_BLOCK_MAJOR, fk.LAYOUT_LAYER_MAJOR


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("host_lens", [False, True], ids=["lengths-on-device", "lengths-on-host"])
@pytest.mark.parametrize("hq", [8, 32], ids=["matrix-core-pass", "vector-pass"])
def test_noalloc_attention_replays_in_a_graph(hq, host_lens):
    hkv = 1 if hq == 8 else 8
    geom = Geometry("graph-attn", 2, hkv, 128, 16, "bfloat16")
    lens = np.array([3000, 1, 777, 1500], np.int32)
    nblk = [-(-int(T) // 16) for T in lens]
    B = sum(nblk) + 4
    g = np.random.default_rng(11)
    pool = fk.KVPool(LM, make_device_pool(geom, LM, B, "cuda", 11))
    perm = g.permutation(B).astype(np.int32)
    tab = np.full((len(lens), max(nblk)), -1, np.int32)
    pos = 0
    for r, k in enumerate(nblk):
        tab[r, :k] = perm[pos:pos + k]
        pos += k
    tab_d = torch.as_tensor(tab, device="cuda")
    lens_d = torch.as_tensor(lens, device="cuda")
    q = torch.randn((len(lens), hq, 128), generator=torch.Generator("cuda").manual_seed(3),
                    device="cuda").to(torch.bfloat16)
    hl = lens if host_lens else None
    say(f"graph capture: no-alloc attention, {hq} query heads on {hkv}, host lengths {host_lens}")

    # eager first (this also looks up the library's scratch on this GPU)
    eager = torch.empty((len(lens), hq, 128), dtype=torch.float32, device="cuda")
    fk.flowkv_decode_attention_noalloc(pool, 1, q, tab_d, lens_d, int(lens.max()), 0.088, eager,
                                       seq_lens_host=hl)
    torch.cuda.synchronize()
    assert torch.isfinite(eager).all()

    out = torch.full_like(eager, float("nan"))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fk.flowkv_decode_attention_noalloc(pool, 1, q, tab_d, lens_d, int(lens.max()), 0.088,
                                           out, seq_lens_host=hl)
    for i in range(4):
        out.fill_(float("nan"))                 # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {i} differs from the eager call"
        # an eager call of the same attention between replays shares the
        # scratch; the next replay must still be right
        other = torch.empty_like(eager)
        fk.flowkv_decode_attention_noalloc(pool, 0, q, tab_d, lens_d, int(lens.max()), 0.088,
                                           other, seq_lens_host=hl)
        torch.cuda.synchronize()
    say("  4 replays equal the eager call")


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, BM)], ids=["block-block", "layer-block"])
def test_inline_transfer_replays_in_a_graph(sl, dl):
    """A 255-run plan in the kernel arguments (the compact form between
    block-major pools, the general form's 64-run limit does not apply) or a
    40-run plan from a layer-major sender, captured and replayed: each replay
    copies the same blocks again after the receiver was overwritten."""
    geom = Geometry("graph-xfer", 4, 2, 64, 16, "bfloat16")
    k = 255 if (sl, dl) == (BM, BM) else 40
    B = 2 * k + 8
    S = 2 * np.arange(k, dtype=np.int32)
    D = 2 * np.arange(k, dtype=np.int32) + 1
    segs = fk.flowkv_plan(S, D, B, B)
    assert len(segs) == k
    src = fk.KVPool(sl, make_device_pool(geom, sl, B, "cuda", 21))
    dst = fk.KVPool(dl, make_device_pool(geom, dl, B, "cuda", 22))
    say(f"graph capture: inline transfer, {k} runs")

    def blocks(pool, ids):
        idx = torch.as_tensor(ids.astype(np.int64), device="cuda")
        if pool.layout == BM:
            return pool.tensors[0].index_select(0, idx).view(torch.uint8).reshape(len(ids), -1)
        per = [t.index_select(1, idx).view(torch.uint8).reshape(2, len(ids), -1)
               for t in pool.tensors]
        return torch.stack(per, 0).permute(2, 0, 1, 3).reshape(len(ids), -1)

    want = blocks(src, S).clone()
    if sl != dl:   # block-major receiver: a block is (L, 2, chunk); build that order
        idx = torch.as_tensor(S.astype(np.int64), device="cuda")
        want = torch.stack([t.index_select(1, idx) for t in src.tensors], 0) \
            .permute(2, 0, 1, 3, 4, 5).contiguous().view(torch.uint8).reshape(k, -1)
    untouched = np.setdiff1d(np.arange(B), D)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        fk.flowkv_transfer_inline(src, dst, segs, k)
    for i in range(3):
        for t in dst.tensors:                   # eager work between replays
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(blocks(dst, D), want), f"replay {i}: moved blocks differ"
        assert not blocks(dst, untouched).any(), f"replay {i}: wrote outside the plan"
    say("  3 replays move the plan's blocks and nothing else")


@pytest.mark.parametrize("sl,dl", [(BM, BM), (LM, BM), (BM, LM)],
                         ids=["block-block", "layer-block", "block-layer"])
def test_per_layer_launches_replay_in_a_graph(sl, dl):
    """The form the Table 3 sweep replays: one launch per layer with the plan
    in device memory, all of them captured in one graph.  Each replay, after
    the receiver was cleared, moves every layer of the plan's blocks and
    nothing else."""
    geom = Geometry("graph-layers", 6, 2, 64, 16, "bfloat16")
    k = 37
    B = 3 * k + 5
    S = np.random.default_rng(31).permutation(B)[:2 * k].astype(np.int32)
    D = (np.arange(2 * k, dtype=np.int32) // 2) * 3 + (np.arange(2 * k) % 2)
    segs = fk.flowkv_plan(S, D.astype(np.int32), B, B)
    n = len(S)
    src = fk.KVPool(sl, make_device_pool(geom, sl, B, "cuda", 41))
    dst = fk.KVPool(dl, make_device_pool(geom, dl, B, "cuda", 42))
    segs_dev = fk.segments_to_device(segs, src.device)
    torch.cuda.synchronize()
    say(f"graph capture: {geom.num_layers} per-layer launches, {len(segs)} runs")

    def blocks(pool, ids):   # (len(ids), L, 2, chunk) bytes in either layout
        idx = torch.as_tensor(np.asarray(ids, dtype=np.int64), device="cuda")
        if pool.layout == BM:
            return pool.tensors[0].index_select(0, idx).view(torch.uint8).reshape(
                len(ids), geom.num_layers, 2, -1)
        per = [t.index_select(1, idx).view(torch.uint8).reshape(2, len(ids), -1)
               for t in pool.tensors]
        return torch.stack(per, 0).permute(2, 0, 1, 3)

    want = blocks(src, S).clone()
    untouched = np.setdiff1d(np.arange(B), D)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for layer in range(geom.num_layers):
            fk.flowkv_transfer_layers(src, dst, segs_dev, len(segs), n, layer, 1)
    for i in range(3):
        for t in dst.tensors:                   # eager work between replays
            t.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(blocks(dst, D), want), f"replay {i}: moved blocks differ"
        assert not blocks(dst, untouched).any(), f"replay {i}: wrote outside the plan"
    say("  3 replays move every layer of the plan's blocks and nothing else")


def test_request_and_workspace_attention_replay_in_a_graph():
    """Two more entry points that allocate nothing during the call: the
    one-call request transfer (its plan is built on the host stack and
    rides in the kernel arguments) and attention with the caller's
    workspace.  Captured together, replayed after the receiver and the
    output were cleared, each replay reproduces the eager results."""
    geom = Geometry("graph-both", 3, 2, 128, 16, "bfloat16")
    B = 96
    g = np.random.default_rng(51)
    S = g.permutation(B)[:40].astype(np.int32)
    D = g.permutation(B)[:40].astype(np.int32)
    src = fk.KVPool(BM, make_device_pool(geom, BM, B, "cuda", 52))
    dst = fk.KVPool(BM, make_device_pool(geom, BM, B, "cuda", 53))
    lens = np.array([600, 17], np.int32)
    tab = torch.as_tensor(np.stack([D[:38], np.r_[D[38:], -np.ones(36, np.int32)]]),
                          device="cuda")
    lens_d = torch.as_tensor(lens, device="cuda")
    q = torch.randn((2, 8, 128), generator=torch.Generator("cuda").manual_seed(54),
                    device="cuda").to(torch.bfloat16)
    ws = torch.empty(fk.flowkv_decode_attention_workspace(2, 8, 128, 600), dtype=torch.uint8,
                     device="cuda")
    say("graph capture: request transfer, then attention over the moved blocks")

    def both(out):
        fk.flowkv_transfer_request(src, dst, S, D)
        fk.flowkv_decode_attention(dst, 1, q, tab, lens_d, 600, 0.088, out, ws)

    pre = dst.tensors[0].clone()
    eager = torch.empty((2, 8, 128), dtype=torch.float32, device="cuda")
    both(eager)
    torch.cuda.synchronize()
    moved = dst.tensors[0].clone()
    out = torch.empty_like(eager)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        both(out)
    for i in range(3):
        dst.tensors[0].copy_(pre)               # eager work between replays
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(dst.tensors[0], moved), f"replay {i}: receiver differs"
        assert torch.equal(out, eager), f"replay {i}: attention differs"
    say("  3 replays equal the eager calls")
