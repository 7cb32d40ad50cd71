"""CPU checks of the full-size tests' receiver-pool checksums
(``tests/gpu_helpers.block_checksums``), on CPU tensors in both layouts."""

from types import SimpleNamespace

import numpy as np
import torch

from tests.gpu_helpers import BM, LM, block_checksums


def fake_pool(layout, L=3, B=7, chunk_words=24, seed=0):
    g = torch.Generator().manual_seed(seed)
    if layout == BM:
        ts = [torch.randint(-2**31, 2**31 - 1, (B, L, 2, chunk_words), generator=g,
                            dtype=torch.int64).to(torch.int32)]
    else:
        ts = [torch.randint(-2**31, 2**31 - 1, (2, B, chunk_words), generator=g,
                            dtype=torch.int64).to(torch.int32) for _ in range(L)]
    return SimpleNamespace(layout=layout, num_blocks=B, num_layers=L, tensors=ts,
                           chunk_bytes=4 * chunk_words, device=torch.device("cpu"))


def block_words(pool, b):
    """Block b's 32-bit words in block order: (layer, K/V, chunk)."""
    if pool.layout == BM:
        return pool.tensors[0][b].reshape(-1).numpy().astype(np.int64)
    return np.concatenate([t[kv, b].numpy() for t in pool.tensors for kv in range(2)]
                          ).astype(np.int64)


def test_checksums_match_their_definition_in_both_layouts():
    for layout in (BM, LM):
        pool = fake_pool(layout)
        got = block_checksums(pool, piece_bytes=200).numpy()
        for b in range(pool.num_blocks):
            x = block_words(pool, b)
            w = np.arange(x.size) % 4093 + 1
            assert got[b, 0] == x.sum() and got[b, 1] == (x * w).sum()


def test_checksums_see_a_changed_or_moved_word():
    for layout in (BM, LM):
        pool = fake_pool(layout, seed=1)
        base = block_checksums(pool)
        t = pool.tensors[0] if layout == BM else pool.tensors[2]
        idx = (4, 1, 1, 5) if layout == BM else (1, 4, 5)
        t[idx] += 1                                        # one word of block 4 changes
        after = block_checksums(pool)
        assert not torch.equal(after[4], base[4])
        assert torch.equal(torch.cat((after[:4], after[5:])), torch.cat((base[:4], base[5:])))
        t[idx] -= 1
        row = t[4] if layout == BM else t[1, 4]
        row.view(-1)[[0, 1]] = row.view(-1)[[1, 0]].clone()   # two words swap places
        assert block_checksums(pool)[4, 0] == base[4, 0]
        assert block_checksums(pool)[4, 1] != base[4, 1]
