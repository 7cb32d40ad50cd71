"""The library driven through its C ABI alone, without Python or torch.

``tests/native/abi_transfer`` (built by the package's build step) allocates
two block-major pools with hipMalloc, places two requests with the library's
allocators, plans them and moves one with flowkv_transfer (plan in device
memory), one with flowkv_transfer_inline (plan in the kernel arguments) and
one with flowkv_transfer_request (planned and launched in one call), then
writes the pools and block lists out.  The receiver pool after the
transfers must equal the oracle's result on the sender pool and the
receiver's pre-image, byte for byte.
"""

import os
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "native", "abi_transfer")

pytestmark = pytest.mark.gpu


def host_pool(raw: np.ndarray, layers, blocks, bs, slot) -> oracle.HostPool:
    hp = oracle.HostPool.zeros(oracle.BLOCK_MAJOR, layers, blocks, bs, slot)
    hp.buffers[0][:] = raw
    return hp


def test_transfer_through_the_c_abi_alone(tmp_path):
    assert os.path.exists(EXE), "tests/native/abi_transfer is not built (run the build step)"
    print("running", EXE, flush=True)
    r = subprocess.run([EXE, str(tmp_path)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi ok" in r.stdout
    lines = (tmp_path / "tables.txt").read_text().splitlines()
    L, bs, slot, src_blocks, dst_blocks, runs_a, runs_b, runs_c = map(int, lines[0].split())
    lists = {ln.split()[0]: np.array(ln.split()[1:], dtype=np.int64) for ln in lines[1:]}
    read = lambda name: np.fromfile(tmp_path / name, dtype=np.uint8)  # noqa: E731
    src = host_pool(read("src.bin"), L, src_blocks, bs, slot)
    want = host_pool(read("dst_before.bin"), L, dst_blocks, bs, slot)
    got = host_pool(read("dst_after.bin"), L, dst_blocks, bs, slot)
    for req in ("A", "B", "C"):
        oracle.transfer_fast(src, want, lists["S" + req], lists["D" + req])
    assert np.array_equal(got.buffers[0], want.buffers[0])
    # the run counts the program used are the oracle's plan sizes
    assert runs_a == len(oracle.plan_ref(lists["SA"].tolist(), lists["DA"].tolist()))
    assert runs_b == len(oracle.plan_ref(lists["SB"].tolist(), lists["DB"].tolist()))
    assert runs_c == len(oracle.plan_ref(lists["SC"].tolist(), lists["DC"].tolist()))
    # and the transfers changed something: A, B and C are 52 of 80 blocks
    assert not np.array_equal(got.buffers[0], read("dst_before.bin"))
