"""The matrix-core attention pass's explicit vector-memory wait against the
gfx950 code the compiler emits (CPU: hipcc cross-compiles without a GPU).

Inside its tile loop, decode_attn_split_mfma waits with s_waitcnt
vmcnt(kIssueVm) for the current tile's V, which it loaded into LDS with
global_load_lds: the compiler does not track those loads for LDS reads.  That
wait is right only if the loop issues exactly kIssueVm vector-memory
instructions per iteration -- the next tile's loads -- and nothing else that
counts against the same counter (a register spill to scratch would).  The
immediate comes from the constexpr counts that size the issue loop; this test
checks the emitted code against it, for both layouts.

The transfer kernels are checked the same way for what the library claims
of them: every instantiation runs without scratch memory.
"""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "paper_2504_03775_amd", "csrc", "flowkv_attention.hip")
VM = re.compile(r"^\s+(global_|buffer_|flat_|scratch_)\w+")


def hipcc():
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    return None


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    cc = hipcc()
    if cc is None:
        pytest.skip("hipcc not found")
    out = tmp_path_factory.mktemp("asm") / "attn.s"
    from paper_2504_03775_amd.build import HIP_FLAGS, INCLUDE, CSRC
    flags = [f for f in HIP_FLAGS if f not in ("-fPIC", "-Wall")]
    subprocess.run([cc, *flags, "--cuda-device-only", "-S", "-I", INCLUDE, "-I", CSRC, SRC,
                    "-o", str(out)], check=True, capture_output=True, timeout=600)
    return out.read_text()


def kernel_text(asm, pattern):
    m = re.search(rf"^({pattern}):[^\n]*\n(.*?)\n\s+s_endpgm", asm, re.S | re.M)
    assert m, pattern
    return m.group(1), m.group(2)


def metadata(asm, name):
    m = re.search(rf"\.name:\s+{re.escape(name)}\n(.*?)(?=\n  - \.|\Z)", asm, re.S)
    assert m, name
    return m.group(1)


@pytest.mark.parametrize("lens", ["Lb0", "Lb1"], ids=["lengths-on-device", "lengths-in-arguments"])
@pytest.mark.parametrize("layout", ["Lb0", "Lb1"], ids=["block-major", "layer-major"])
def test_mfma_wait_matches_the_loads_the_loop_issues(asm, layout, lens):
    name, body = kernel_text(asm, rf"_ZN\w*decode_attn_split_mfmaILi8E{layout}E{lens}EEEvN\w+")
    waits = [int(x) for x in re.findall(r"s_waitcnt vmcnt\((\d+)\)", body)]
    explicit = [w for w in waits if w > 0]
    assert len(explicit) == 1, waits
    n = explicit[0]
    # the basic blocks of the loop that holds the explicit wait: LLVM marks
    # each with its loop header
    blocks = re.split(r"\n(?=\.LBB\d+_\d+:)", body)
    holder = next(b for b in blocks if f"s_waitcnt vmcnt({n})" in b)
    header = re.search(r"(?:Header=|=>This Inner Loop Header)", holder.split("\n")[0])
    assert header, "the explicit wait is not inside a loop"
    m = re.search(r"Header=(BB\d+_\d+)", holder.split("\n")[0])
    head = m.group(1) if m else holder.split(":")[0].lstrip(".")
    in_loop = [b for b in blocks
               if f"Header={head} " in b.split("\n")[0] or b.startswith(f".L{head}:")]
    assert len(in_loop) >= 2
    vm = [ln.strip() for b in in_loop for ln in b.split("\n") if VM.match(ln)]
    assert len(vm) == n, (n, vm)
    assert sum("global_load_lds" in x for x in vm) == n // 2     # V into LDS
    assert not any("store" in x or "atomic" in x for x in vm)
    meta = metadata(asm, name)
    assert re.search(r"\.private_segment_fixed_size:\s+0\b", meta)
    assert re.search(r"\.vgpr_spill_count:\s+0\b", meta)


# ---- the transfer kernels: no scratch memory, no spills ------------------------

XFER_SRC = os.path.join(ROOT, "paper_2504_03775_amd", "csrc", "flowkv_transfer.hip")


@pytest.fixture(scope="module")
def xfer_asm(tmp_path_factory):
    cc = hipcc()
    if cc is None:
        pytest.skip("hipcc not found")
    out = tmp_path_factory.mktemp("asm") / "xfer.s"
    from paper_2504_03775_amd.build import HIP_FLAGS, INCLUDE, CSRC
    flags = [f for f in HIP_FLAGS if f not in ("-fPIC", "-Wall")]
    subprocess.run([cc, *flags, "--cuda-device-only", "-S", "-I", INCLUDE, "-I", CSRC, XFER_SRC,
                    "-o", str(out)], check=True, capture_output=True, timeout=900)
    return out.read_text()


def test_transfer_kernels_use_no_scratch_and_spill_nothing(xfer_asm):
    """Every instantiation of kv_segment_copy -- both layouts on each side,
    every unroll and cache policy, both address paths, the device-plan form
    and the three argument forms -- keeps its state in registers: no private
    (scratch) segment and no vector registers spilled.  So the transfer needs
    no device memory beyond the pools and the caller's plan, which is why it
    has no variant that allocates nothing.  The default launch shape (unroll
    4) spills no scalar registers either; some unroll-16 forms spill a few
    into vector-register lanes, which costs no memory."""
    names = re.findall(r"\.name:\s+(\S*kv_segment_copy\S*)", xfer_asm)
    # 4 layout pairs x 4 unroll x 4 cache x 2 paths x (device plan, general
    # inline form), 32 between block-major pools and 96 with a layer-major
    # pool in the compact forms
    assert len(names) == 4 * 4 * 4 * 2 * 2 + 32 + 96, len(names)
    assert sum("XferArgsCompactILi1E" in n for n in names) == 32
    assert sum("XferArgsCompactILi32E" in n for n in names) == 96
    # the code object's kernel list, one YAML entry per kernel
    entries = [e for e in re.split(r"\n  - ", xfer_asm) if "kv_segment_copy" in e
               and re.search(r"\.name:\s+\S*kv_segment_copy", e)]
    assert len(entries) == len(names)
    for e in entries:
        n = re.search(r"\.name:\s+(\S+)", e).group(1)
        assert re.search(r"\.private_segment_fixed_size:\s+0\b", e), n
        assert re.search(r"\.vgpr_spill_count:\s+0\b", e), n
        if "ELi4ELi" in n:    # unroll 4, the default
            assert re.search(r"\.sgpr_spill_count:\s+0\b", e), n
        size = int(re.search(r"\.kernarg_segment_size:\s+(\d+)", e).group(1))
        assert size <= 4096, (n, size)
