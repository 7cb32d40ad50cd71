"""Benchmark of the KV-cache transfer hot path on one MI355X.

Default workload: one Llama-3-8B-shape request of 13,000 tokens (813 blocks
of 2 MiB: 32 layers x K/V x 16 tokens x 8 KV heads x 128 dims, bf16) moved
between two 65,536-block pools.  The sender's blocks come from the segment
allocator on a fresh pool (one run); the receiver's table comes from a seeded
free list (free IDs ascending) of a pool with 30% of its blocks held at
random, which gives 255 runs.  A step is one pass of the hot path for that
request:
  1. bidirectional segment alignment of the sender's and receiver's block
     lists (host),
  2. the plan goes to the device: in the kernel's arguments when it fits
     there (64 runs, or 300 between block-major pools in the planner's
     form), else staged through a ring of pinned buffers (one small copy on
     a side stream, overlapping the previous kernel),
  3. one kernel launch moves every run's K and V of all 32 layers.
With --dst-policy segment the receiver's segment allocator also runs inside
every step: it places the request's 813 blocks in the 30%-occupied pool (43
runs, so the plan rides in the kernel's arguments) and releases them after
the launch, so every step sees the same pool state.  The default run also
times that receiver the same way and reports it under context.
The other workloads (--workload) take their block lists from the allocators
at setup, as their recipes describe; their step is plan + stage + one launch
for the whole batch.  Steps are enqueued back to back on one stream; host work
overlaps the previous step's kernel.  Inputs are resident in HBM before timing
starts.

Prints one JSON line.  `value` is the effective transfer rate (payload bytes
of K and V moved per second over the timed steps); `roofline` prices the
transfer kernel's own launches (events around each launch -- or, with
--layerwise, around each step's per-layer launches -- on their stream)
against the 8 TB/s HBM peak with 2x payload (read + write) of traffic;
`cpu_baseline` is the oracle (numpy, one thread) moving the same blocks on the
host.  The timed launches are bracketed by HIP events made for timing only
(see TimingEvent).
"""

from __future__ import annotations

import argparse
import ctypes
import gc
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "effective KV transfer GB/s (% of HBM peak); ms per 13k-token request transfer"
KERNEL_SRC = os.path.join(ROOT, "paper_2504_03775_amd", "csrc", "flowkv_transfer.hip")
PMC_SUMMARY = os.path.join(ROOT, "profiles", "kv_segment_copy_llama3-8b-13k_pmc.txt")
# counter summaries per (workload, layout) of the transfer kernel
PMC_SUMMARIES = {
    ("8b", "block"): PMC_SUMMARY,
    ("8b", "layer"): os.path.join(ROOT, "profiles",
                                  "kv_segment_copy_llama3-8b-13k_layer-major_pmc.txt"),
    ("70b-shuffled", "layer"): os.path.join(ROOT, "profiles",
                                            "kv_segment_copy_70b-shuffled_layer-major_pmc.txt"),
}
ATTN_SRC = os.path.join(ROOT, "paper_2504_03775_amd", "csrc", "flowkv_attention.hip")

# hipEventDisableSystemFence (hip_runtime_api.h): recording the event skips
# the system-scope fence (an L2 write-back and invalidation) that an ordinary
# event adds after the work it follows
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000
_HIP_RT = []


def _hip_runtime():
    """The HIP runtime torch loaded (one per process), with the event calls."""
    if not _HIP_RT:
        paths = sorted({ln.split()[-1] for ln in open("/proc/self/maps")
                        if "libamdhip64" in ln})
        if len(paths) != 1:
            raise RuntimeError(f"expected one HIP runtime in the process, found {paths}")
        lib = ctypes.CDLL(paths[0])
        lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                            ctypes.c_void_p]
        lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        _HIP_RT.append(lib)
    return _HIP_RT[0]


class TimingEvent:
    """A HIP event for timing only, with torch.cuda.Event's record() and
    elapsed_time().  It is created with hipEventDisableSystemFence: an
    ordinary event's completion fence writes back and invalidates the caches
    between back-to-back kernels, which measurably lengthens both the step
    and the interval the events bracket (about 3 us per 0.55 ms step)."""

    def __init__(self):
        self._rt = _hip_runtime()
        self._h = ctypes.c_void_p()
        rc = self._rt.hipEventCreateWithFlags(ctypes.byref(self._h),
                                              HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags returned {rc}")

    def record(self, stream=None):
        import torch

        s = stream if stream is not None else torch.cuda.current_stream()
        rc = self._rt.hipEventRecord(self._h, ctypes.c_void_p(s.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord returned {rc}")

    def elapsed_time(self, end: "TimingEvent") -> float:
        ms = ctypes.c_float()
        rc = self._rt.hipEventElapsedTime(ctypes.byref(ms), self._h, end._h)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime returned {rc}")
        return ms.value

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h:
            self._rt.hipEventDestroy(h)


TIMING = {"events": "hip, system fence disabled"}


def timing_pairs(k: int):
    """k (start, end) timing-event pairs: TimingEvent, or torch's events
    where the runtime refuses the flag (TIMING says which)."""
    import torch

    try:
        return [(TimingEvent(), TimingEvent()) for _ in range(k)]
    except (RuntimeError, OSError, AttributeError) as e:
        TIMING["events"] = f"torch ({e})"
        return [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(k)]
ATTN_PMC_SUMMARY = {
    "batch": os.path.join(ROOT, "profiles", "decode_attn_llama3-8b-batch32_pmc.txt"),
    "70b": os.path.join(ROOT, "profiles", "decode_attn_llama3-70b-tp8-share_pmc.txt"),
}

WORKLOADS = {
    # name: (recipe, args, description)
    "8b": ("llama8b_13k", (), "llama3-8b-kv-13k-token-request"),
    "tiny": ("tiny", (), "tiny-2-layer-fp16-256-token-request"),
    "batch": ("batch32", ("segment",), "llama3-8b-kv-batch-32-requests-2k-20k/segment-allocator"),
    "batch-shuffled": ("batch32", ("fifo_shuffled",),
                       "llama3-8b-kv-batch-32-requests-2k-20k/shuffled-free-list"),
    "70b": ("llama70b_tp8", ("segment",), "llama3-70b-tp8-share-16x32k-tokens/segment-allocator"),
    "70b-shuffled": ("llama70b_tp8", ("fifo_shuffled",),
                     "llama3-70b-tp8-share-16x32k-tokens/shuffled-free-list"),
    "churn": ("churn", ("segment",), "llama3-8b-kv-churn-128-live/segment-allocator"),
    "churn-shuffled": ("churn", ("shuffled",), "llama3-8b-kv-churn-128-live/shuffled-free-list"),
    "churn-stride2": ("churn", ("stride2",), "llama3-8b-kv-churn/stride-2-one-block-runs"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1,
                    help="GPUs to use: 1 only (the path runs on one device)")
    ap.add_argument("--op", choices=["transfer", "attention", "schedule", "overlap", "table3"],
                    default="transfer",
                    help="transfer: the KV transfer hot path (default); attention: one decode "
                         "step of paged attention over the receiver pool of the batch workload; "
                         "schedule: the load-aware scheduler (host) at 1,024 nodes, and the "
                         "cluster model's three load mixes with fixed and load-aware roles; "
                         "overlap: the 13k request's transfer after, or layer by layer beside, "
                         "a prefill stand-in; table3: one launch against 32 per-layer launches "
                         "at Table 3's input lengths")
    ap.add_argument("--lengths", default="",
                    help="table3: comma-separated input lengths in tokens (default: Table 3's "
                         "500, 1000, 2000, 4000, 8000, 10000, 12000)")
    ap.add_argument("--steps", type=int, default=100, help="timed steps")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before them (default: 200 for attention, whose "
                         "step needs about 25 ms of work to reach steady clocks, else 10)")
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="8b")
    ap.add_argument("--layout", choices=["block", "layer"], default="block",
                    help="pool layout of both sides: Eq. 5 block-major or per-layer")
    ap.add_argument("--dst-policy", choices=["segment", "fifo_sorted", "fifo_shuffled"],
                    default="fifo_sorted", help="receiver allocator of the 8b workload")
    ap.add_argument("--dst-occupied", type=float, default=0.30,
                    help="8b workload: fraction of the receiver's blocks held at random before "
                         "the request arrives")
    ap.add_argument("--layerwise", action="store_true",
                    help="move each plan as one launch per layer (the paper's layer-wise "
                         "ablation) instead of one launch for all layers")
    ap.add_argument("--staged-plan", action="store_true",
                    help="always stage the plan in device memory (no kernel-argument plans)")
    ap.add_argument("--no-cpu-baseline", action="store_true",
                    help="skip timing the oracle on the host")
    ap.add_argument("--no-context", action="store_true",
                    help="skip the memcpy comparators and the flushed-cache timing")
    ap.add_argument("--threads", type=int, default=0,
                    help="transfer workgroup size, 64..1024 (0 = library default)")
    ap.add_argument("--unroll", type=int, default=0,
                    help="16-byte vectors per thread per tile: 2, 4, 8, 16 (0 = default)")
    ap.add_argument("--grid", type=int, default=0,
                    help="transfer workgroups (0 = one per tile, capped per CU)")
    ap.add_argument("--cache", type=int, default=0,
                    help="1 plain, 2 nontemporal loads, 3 nontemporal stores, "
                         "4 both (0 = default)")
    ap.add_argument("--order", type=int, default=0,
                    help="tile visiting order: 1 plan order, 2 blocks scattered, 3 tiles "
                         "scattered (0 = library default)")
    ap.add_argument("--attn-workload", choices=["batch", "8b", "70b"], default="batch",
                    help="attention: receiver pool and block lists of the batch (32 requests), "
                         "8b (one 13,000-token request) or 70b (the TP=8 share, 16 x 32,000 "
                         "tokens) workload")
    ap.add_argument("--split", type=int, default=0,
                    help="attention: tokens per pass-1 workgroup (0 = library default)")
    ap.add_argument("--calibrate-copy-gib", type=float, default=1.0,
                    help="size of the plain copy run beside the kernel (HBM counter scale)")
    ap.add_argument("--calibration-only", action="store_true",
                    help="of the context rows run only the plain copy (for counter runs)")
    args = ap.parse_args()
    if args.warmup is None:
        args.warmup = 200 if args.op == "attention" else 10
    return args


def kernel_hash(src: str = KERNEL_SRC) -> str:
    return hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]


def traffic_from_profile(summary: str = PMC_SUMMARY, src: str = KERNEL_SRC, split=None,
                         runs=None):
    """HBM bytes per launch from the committed counter summary, scaled by the
    plain-copy calibration recorded with it; None if absent, if the kernel
    source changed since the counters were taken, or if they were taken on
    another plan (run count) or (attention) at another split length."""
    if not summary or not os.path.exists(summary):
        return None
    text = open(summary).read()
    if runs is not None:
        mr = re.search(r"(\d+) runs x 16 B plan", text)
        if not mr or int(mr.group(1)) != runs:
            return None
    if split is not None:
        ms = re.search(r"split_tokens:\s*(\d+)", text)
        if not ms or int(ms.group(1)) != split:
            return None
    m = re.search(r"kernel_source_sha256_16:\s*(\w+)", text)
    if not m or m.group(1) != kernel_hash(src):
        return None
    t = re.search(r"hbm_bytes_per_launch:\s*([0-9.eE+]+)", text)
    return float(t.group(1)) if t else None


ATTN_WORKLOADS = {
    # name: (recipe, args, query heads, workload label)
    "batch": ("batch32", ("segment",), 32, "llama3-8b-decode-attention-batch-32-requests-2k-20k"),
    "8b": ("llama8b_13k", ("segment",), 32, "llama3-8b-decode-attention-one-13k-request"),
    "70b": ("llama70b_tp8", ("segment",), 8, "llama3-70b-tp8-share-decode-attention-16x32k"),
}


RESERVE_BYTES = 4 << 30   # device memory left free beside the pools


def fit_receiver_blocks(free_bytes: int, src_blocks: int, dst_blocks: int,
                        block_bytes: int, reserve: int = RESERVE_BYTES) -> int:
    """Receiver-pool size that fits beside the sender's pool: dst_blocks if
    both fit in free_bytes - reserve, else the largest multiple of 4,096
    blocks that does (0 if not even 4,096 fit)."""
    room = free_bytes - reserve - src_blocks * block_bytes
    if room >= dst_blocks * block_bytes:
        return dst_blocks
    return max(0, room // block_bytes // 4096 * 4096)


def attention_setup(attn_workload: str, layout_name: str, split: int):
    """Decode attention (one layer, one new token per request) over the
    receiver pool and block lists of a transfer workload: the step, with the
    lengths carried on the host when they fit, and its algorithmic bytes."""
    import types

    import numpy as np
    import torch

    from paper_2504_03775_amd import flowkv as fk
    from workloads import make_device_pool, recipes

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = fk.LAYOUT_BLOCK_MAJOR if layout_name == "block" else fk.LAYOUT_LAYER_MAJOR
    recipe, rargs, q_heads, label = ATTN_WORKLOADS[attn_workload]
    wl = getattr(recipes, recipe)(lambda P, pol, seed: fk.Allocator(P, pol, seed), *rargs)
    geom = wl.geom
    pool = fk.KVPool(layout, make_device_pool(geom, layout, wl.dst_pool_blocks, dev, seed=1))
    lens = np.asarray(wl.tokens, dtype=np.int32)
    max_blocks = max(len(d) for _, d in wl.tables)
    tab = np.full((len(lens), max_blocks), -1, dtype=np.int32)
    for r, (_, d) in enumerate(wl.tables):
        tab[r, :len(d)] = d
    tab_d = torch.as_tensor(tab, device=dev)
    lens_d = torch.as_tensor(lens, device=dev)
    q = torch.randn((len(lens), q_heads, geom.head_dim), device=dev).to(torch.bfloat16)
    out = torch.empty((len(lens), q_heads, geom.head_dim), dtype=torch.float32, device=dev)
    max_seq = int(lens.max())
    ws = torch.empty(fk.flowkv_decode_attention_workspace(len(lens), q_heads, geom.head_dim,
                                                          max_seq, split),
                     dtype=torch.uint8, device=dev)
    scale = 1.0 / geom.head_dim ** 0.5
    layer = geom.num_layers // 2

    # the lengths travel on the host too, as a serving loop that keeps them
    # there passes them (they then ride in the kernel arguments)
    host_lens = lens if len(lens) <= fk.ATTN_INLINE_LENS else None

    def step(host=True):
        fk.flowkv_decode_attention(pool, layer, q, tab_d, lens_d, max_seq, scale, out, ws,
                                   split, seq_lens_host=host_lens if host else None)

    split_used = split or fk.flowkv_decode_attention_split(len(lens), max_seq)
    kv_bytes = int(lens.sum()) * 2 * geom.kv_heads * geom.head_dim * 2
    # workspace: written by pass 1 and read by pass 2, for the splits that exist
    used_splits = int(sum(-(-int(T) // split_used) for T in lens))
    ws_bytes = 2 * used_splits * q_heads * (geom.head_dim + 2) * 4
    algo = kv_bytes + q.numel() * 2 + out.numel() * 4 + ws_bytes + tab.nbytes
    return types.SimpleNamespace(step=step, algo=algo, label=label, split=split_used,
                                 pool=pool, geom=geom, layer=layer, q=q, wl=wl, lens=lens,
                                 scale=scale, q_heads=q_heads, host_lens=host_lens,
                                 layout=layout_name, dev=dev)


def attention_time(step, steps: int, warmup: int):
    """Mean kernel time (ms, HIP events around each step) and wall time (s)
    of `steps` back-to-back steps after `warmup` untimed ones."""
    import torch

    # the interpreter's garbage is collected before the warmup, not between
    # it and the timed steps: after the GPU idles for a few tens of ms this
    # step runs about 3% slower for the next ~25 ms of work
    evs = timing_pairs(steps)
    gc.collect()
    gc.disable()
    try:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for e in evs:
            e[0].record()
            step()
            e[1].record()
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t0
    finally:
        gc.enable()
    ts = [a.elapsed_time(b) for a, b in evs]
    return statistics.fmean(ts), elapsed, ts


def attention_context(steps: int) -> dict:
    """The attention bench's default step (the 32-request batch over a
    block-major pool), timed the same way, for the transfer bench's line."""
    try:
        a = attention_setup("batch", "block", 0)
        ms, elapsed, ts = attention_time(a.step, steps, 200)
        import numpy as np
        row = {"workload": a.label, "split_tokens": a.split, "steps": steps, "warmup": 200,
               "kernel_ms_avg": round(ms, 4),
               "kernel_ms_p10_p50_p90": [round(float(x), 4)
                                         for x in np.percentile(ts, [10, 50, 90])],
               "hbm_gbps": round(a.algo / (ms * 1e-3) / 1e9, 1),
               "roofline_frac": round(a.algo / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
               "note": "bench.py --op attention's step in the same run (decode_attn_split + "
                       "decode_attn_merge), after the transfer pools were freed"}
        del a
        return row
    except Exception as e:  # reported in the line, never a reason to lose it
        row = {"error": f"{type(e).__name__}: {e}"[:300]}
        try:
            import torch
            row["allocated_gib"] = round(torch.cuda.memory_allocated() / 2**30, 2)
        except Exception:
            pass
        return row


def bench_attention(args):
    """Decode attention (one layer, one new token per request) over the
    receiver pool and block lists of a transfer workload: by default the
    32-request batch (32 query heads on 8 KV heads, head_dim 128, block 16,
    2,000-20,000 tokens per request); also the 13,000-token request and one
    GPU's share of Llama-3-70B at TP=8 (8 query heads on 1 KV head)."""
    import numpy as np
    import torch

    a = attention_setup(args.attn_workload, args.layout, args.split)
    step, algo, split, host_lens = a.step, a.algo, a.split, a.host_lens
    pool, geom, layer, q, wl, lens, scale = a.pool, a.geom, a.layer, a.q, a.wl, a.lens, a.scale
    q_heads, label, dev = a.q_heads, a.label, a.dev
    ms, elapsed, ts = attention_time(step, args.steps, args.warmup)

    context = {}
    ab = None
    if not args.no_context and host_lens is not None:
        # the same step with the lengths in the kernel arguments and read from
        # device memory, alternated step by step so that both see the same
        # clocks and caches
        evs_h, evs_d = timing_pairs(args.steps), timing_pairs(args.steps)
        torch.cuda.synchronize()
        for eh, ed in zip(evs_h, evs_d):
            eh[0].record()
            step(host=True)
            eh[1].record()
            ed[0].record()
            step(host=False)
            ed[1].record()
        torch.cuda.synchronize()
        ab = (statistics.fmean(a.elapsed_time(b) for a, b in evs_h),
              statistics.fmean(a.elapsed_time(b) for a, b in evs_d))
    if not args.no_context:
        # plain contiguous device-to-device copy: context, and the kernel that
        # scales HBM counters taken from this process
        nbytes = int(args.calibrate_copy_gib * (1 << 30))
        a_ = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        b_ = torch.empty_like(a_)
        for _ in range(3):
            b_.copy_(a_)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            b_.copy_(a_)
        e1.record()
        torch.cuda.synchronize()
        context.update({"contiguous_copy_gbps": round(2 * nbytes / (e0.elapsed_time(e1) / 10
                                                                     * 1e-3) / 1e9, 1),
                        "contiguous_copy_bytes": nbytes})
        del a_, b_

    cpu = None
    if not args.no_cpu_baseline:
        cpu = attention_cpu_baseline(pool, geom, layer, q, wl, lens, scale, np, torch)

    achieved = algo / (ms * 1e-3) / 1e9
    if ab is not None:
        context["lengths_in_arguments_vs_device"] = {
            "kernel_ms_avg": [round(ab[0], 4), round(ab[1], 4)],
            "roofline_frac": [round(algo / (x * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4) for x in ab],
            "note": "the step with the lengths in the kernel arguments, then read from "
                    "device memory, alternated step by step"}
    line = {
        "metric": "decode attention HBM GB/s (one layer, one token per request)",
        "value": round(achieved, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed * 1e3 / args.steps, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": label,
                   "requests": len(lens), "tokens": int(lens.sum()), "q_heads": q_heads,
                   "kv_heads": geom.kv_heads, "head_dim": geom.head_dim,
                   "block_size": geom.block_size, "kv_dtype": "bf16",
                   "layout": f"{args.layout}-major", "layer": layer, "split_tokens": split,
                   "lengths_in": ("kernel-arguments" if host_lens is not None
                                  else "device-memory")},
        "kernel_ms_avg": round(ms, 4),
        "kernel_ms_p10_p50_p90": [round(float(x), 4) for x in np.percentile(ts, [10, 50, 90])],
        "timing_events": TIMING["events"],
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic_from_profile(ATTN_PMC_SUMMARY.get(args.attn_workload)
                                                     if args.layout == "block" else None,
                                                     ATTN_SRC, split)},
        "cpu_baseline": cpu,
        "context": context,
    }
    print(json.dumps(line), flush=True)


def attention_cpu_baseline(pool, geom, layer, q, wl, lens, scale, np, torch):
    """The float64 oracle on the host, on a bounded sample: the workload's
    shortest request (its blocks downloaded to a compact host pool), run
    repeatedly for about 10 s; reported as K/V bytes read per second."""
    import oracle
    from oracle.attention import decode_attention

    r = int(np.argmin(lens))
    ids = np.asarray(wl.tables[r][1], dtype=np.int64)
    T = int(lens[r])
    idx = torch.as_tensor(ids, device=pool.device)
    slot = pool.kv_heads * pool.head_dim * pool.elem_bytes
    hp = oracle.HostPool.zeros(pool.layout, pool.num_layers, len(ids), pool.block_size, slot)
    if pool.layout == 1:    # block-major: one tensor, rows are blocks
        hp.buffers[0][:] = pool.tensors[0].index_select(0, idx).view(torch.uint8).cpu() \
            .numpy().reshape(-1)
    else:                   # layer-major: per layer (2, B, ...)
        for l_, t in enumerate(pool.tensors):
            hp.buffers[l_][:] = t.index_select(1, idx).contiguous().view(torch.uint8).cpu() \
                .numpy().reshape(-1)
    qh = q[r:r + 1].float().cpu().numpy().astype(np.float64)
    reps, dt = 0, 0.0
    while dt < 10.0 and reps < 1000:
        t0 = time.perf_counter()
        decode_attention(hp, qh, [list(range(len(ids)))], [T], layer, geom.kv_heads,
                         geom.head_dim, scale)
        dt += time.perf_counter() - t0
        reps += 1
    kv = T * 2 * geom.kv_heads * geom.head_dim * 2
    return {"value": round(kv * reps / dt / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"request {r} of the workload ({T} tokens, {kv} K/V bytes), one layer, "
                      f"repeated {reps}x ({dt:.1f} s), float64 numpy with a per-slot gather, "
                      f"one thread; {os.cpu_count()} host cores visible"}


def bench_schedule(args):
    """Load-aware scheduler (section 3.4, Algorithm 1), host code: evaluations
    per second at 1,024 nodes (512 prefill, 512 decode, window 8), routing
    calls per second, and the seeded cluster model's outcomes with fixed and
    load-aware roles.  No device kernel runs in this mode."""
    import numpy as np

    from paper_2504_03775_amd import flowkv as fk
    from workloads.cluster_sim import (STATUS_SCALE, Cluster, ClusterConfig, NativeScheduler,
                                       Workload)

    n, window = 1024, 8
    w = [0.25, 0.25, 0.125, 0.125, 0.0625, 0.0625, 0.0625, 0.0625]
    pargs = (window, STATUS_SCALE, w, w, 0.5, 0.5, 1.0, 1.0, 0.1, 3)
    roles = [i % 2 for i in range(n)]
    rng = np.random.default_rng(0)
    samples = rng.uniform(0, 4, size=(64, n, 12))
    nat = fk.Scheduler(fk.sched_params(*pargs), roles)

    def evals(sched, k):
        for i in range(k):
            sched.observe(samples[i % len(samples)])
            sched.evaluate()

    evals(nat, args.warmup)
    t0 = time.perf_counter()
    evals(nat, args.steps)
    t_eval = (time.perf_counter() - t0) / args.steps
    zeros = np.zeros(n, dtype=np.int64)
    queued = rng.integers(0, 100_000, n)
    rate = np.where(np.asarray(roles) == 0, 40_000.0, 0.0)
    spb = np.full((n, n), 2e-11)
    lat = np.full((n, n), 5e-5)
    free = np.full(n, 1 << 40, dtype=np.int64)
    t0 = time.perf_counter()
    for _ in range(args.steps):
        nat.route(8000, zeros, queued, rate, 8000 * 131072, spb, lat, free)
    t_route = (time.perf_counter() - t0) / args.steps

    cpu = None
    if not args.no_cpu_baseline:
        from oracle.scheduler import Params, RefScheduler
        ref = RefScheduler(Params(window, STATUS_SCALE, w, w, 0.5, 0.5, 1.0, 1.0, 0.1, 3), roles)
        as_lists = [s_.tolist() for s_ in samples]
        k, t_sum = 0, 0.0
        while t_sum < 10.0 and k < 10_000:        # about 10 s of host work
            t0 = time.perf_counter()
            ref.observe(as_lists[k % len(as_lists)])
            ref.evaluate()
            t_sum += time.perf_counter() - t0
            k += 1
        t_ref = t_sum / k
        cpu = {"value": round(1.0 / t_ref, 2), "unit": "evaluations/s", "cores": 1,
               "kind": "oracle", "sample": f"{k} evaluations at {n} nodes, window {window}, "
                                          f"pure Python ({t_sum:.1f} s)"}

    mixes = {"balanced": Workload(6.0, 400, [1000, 5000, 10000], [256], seed=1),
             "prefill-heavy": Workload(5.0, 300, [12000, 16000, 20000], [32], seed=2),
             "decode-heavy": Workload(30.0, 600, [500, 1000], [1024], seed=3)}
    sim = {}
    for name, wl in mixes.items():
        row = {}
        for label, sw in (("fixed", False), ("load_aware", True)):
            r4 = [0, 0, 1, 1]
            c = Cluster(ClusterConfig(roles=r4, switching=sw),
                        NativeScheduler(fk, fk.sched_params(4, *pargs[1:]), r4))
            out = c.run(wl)
            row[label] = {k_: (round(v, 4) if isinstance(v, float) else v)
                          for k_, v in out.items()
                          if k_ in ("requests_per_s", "ttft_mean_s", "e2e_mean_s",
                                    "role_switches", "scenario_ticks")}
        sim[name] = row
    # the extreme scenarios' scaling (low load read as the lower thresholds
    # eps_min = 0.05): a busy phase then a quiet one, 2 prefill + 2 decode
    # nodes and 2 offline spares, against four fixed nodes
    from workloads.cluster_sim import DECODE, OFFLINE, PREFILL
    phased = Workload(0.5, 300, [1000, 4000, 8000], [128, 512], seed=4,
                      phases=((20.0, 12.0), (60.0, 0.5)))
    row = {}
    for label, r6, scaling in (("four_fixed_nodes", [PREFILL, PREFILL, DECODE, DECODE], False),
                               ("scaling_with_spares", [PREFILL, PREFILL, DECODE, DECODE,
                                                        OFFLINE, OFFLINE], True)):
        c = Cluster(ClusterConfig(roles=r6, scaling=scaling),
                    NativeScheduler(fk, fk.sched_params(4, *pargs[1:], 0.05, 0.05), r6))
        out = c.run(phased)
        row[label] = {k_: (round(v, 4) if isinstance(v, float) else v) for k_, v in out.items()
                      if k_ in ("requests_per_s", "ttft_mean_s", "e2e_mean_s", "node_seconds",
                                "scale_requests", "scale_downs", "scenario_ticks")}
    sim["busy-then-quiet"] = row
    line = {
        "metric": "load-aware scheduler evaluations per second (1,024 nodes, window 8)",
        "value": round(1.0 / t_eval, 1), "unit": "evaluations/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(t_eval * 1e3, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": "load-aware-scheduler-1024-nodes", "nodes": n, "window": window,
                   "prefill_nodes": n // 2, "decode_nodes": n // 2},
        "route_us": round(t_route * 1e6, 2),
        "roofline": None,
        "cpu_baseline": cpu,
        "context": {"cluster_model_2p2d": sim},
    }
    print(json.dumps(line), flush=True)


def bench_overlap(args):
    """Layer-wise transfer overlapped with prefill (section 4.4 and Table 3:
    FlowKV-Layerwise).  A step prefills one 13,000-token Llama-3-8B prompt
    and moves its KV cache (the 13k request's plan), in four forms:
      prefill           the prefill stand-in alone;
      one_launch_after  prefill, then the whole transfer in one launch;
      layerwise_overlap each layer's transfer launched on a transfer stream as
                        soon as that layer's prefill work is done;
      layerwise_after   prefill, then 32 per-layer launches.
With layer-major pools two comparators run beside them, copying the same
runs with the copy engines instead of a kernel (hipMemcpyAsync of kind
hipMemcpyDeviceToDeviceNoCU, one call per run, layer and K-or-V):
      sdma_layerwise_overlap  per layer, as soon as that layer's prefill
                              work is done, on the transfer stream;
      sdma_after              all of them after the prefill.
    The prefill stand-in is each layer's four projection products over the
    prompt (q/k/v, output, gate and up, down: 5.67 TFLOP per layer in bf16,
    torch.matmul); attention over the prompt, norms and activations are left
    out, so the stand-in is shorter than a real prefill.  `value` is the
    transfer time the layer-wise overlap leaves exposed after the prefill:
    the median over rounds of (overlapped step - prefill-alone step), the
    four forms running interleaved, once per round."""
    import torch

    from paper_2504_03775_amd import flowkv as fk
    from workloads import make_device_pool, recipes

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = fk.LAYOUT_BLOCK_MAJOR if args.layout == "block" else fk.LAYOUT_LAYER_MAJOR
    wl = recipes.llama8b_13k(lambda P, pol, seed: fk.Allocator(P, pol, seed), args.dst_policy)
    geom = wl.geom
    S, D = wl.flat()
    n = len(S)
    src = fk.KVPool(layout, make_device_pool(geom, layout, wl.src_pool_blocks, dev, seed=0))
    dst = fk.KVPool(layout, make_device_pool(geom, layout, wl.dst_pool_blocks, dev, seed=1))
    segs = fk.flowkv_plan(S, D, wl.src_pool_blocks, wl.dst_pool_blocks)
    segs_dev = fk.segments_to_device(segs, dev)

    T, d, ff, kvd = sum(wl.tokens), 4096, 14336, 1024   # Llama-3-8B layer shapes
    g = torch.Generator(device=dev).manual_seed(9)

    def weight(k, m):
        return (torch.randn((k, m), generator=g, device=dev) * k ** -0.5).to(torch.bfloat16)

    x = torch.randn((T, d), generator=g, device=dev).to(torch.bfloat16)
    w_q, w_kv, w_o = weight(d, d), weight(d, 2 * kvd), weight(d, d)
    w_g, w_u, w_d = weight(d, ff), weight(d, ff), weight(ff, d)
    flops_layer = 2 * T * (d * d + d * 2 * kvd + d * d + 2 * d * ff + ff * d)

    def prefill_layer():
        q = x @ w_q
        _kv = x @ w_kv
        o = q @ w_o
        _u = o @ w_u
        return (o @ w_g) @ w_d

    main_s = torch.cuda.current_stream()
    xfer_s = torch.cuda.Stream(dev)            # default priority, like every stream here
    layer_done = [torch.cuda.Event() for _ in range(geom.num_layers)]

    def run(mode):
        for layer in range(geom.num_layers):
            prefill_layer()
            if mode == "layerwise_overlap":
                layer_done[layer].record(main_s)
                xfer_s.wait_event(layer_done[layer])
                fk.flowkv_transfer_layers(src, dst, segs_dev, len(segs), n, layer, 1,
                                          stream=xfer_s)
            elif mode == "sdma_layerwise_overlap":
                layer_done[layer].record(main_s)
                xfer_s.wait_event(layer_done[layer])
                sdma_layer(layer, xfer_s)
        if mode == "sdma_after":
            for layer in range(geom.num_layers):
                sdma_layer(layer, main_s)
        elif mode == "one_launch_after":
            if len(segs) <= fk.inline_capacity(src, dst):
                fk.flowkv_transfer_inline(src, dst, segs, n, stream=main_s)
            else:
                fk.flowkv_transfer_ex(src, dst, segs_dev, len(segs), n, stream=main_s)
        elif mode == "layerwise_after":
            for layer in range(geom.num_layers):
                fk.flowkv_transfer_layers(src, dst, segs_dev, len(segs), n, layer, 1,
                                          stream=main_s)
        elif mode in ("layerwise_overlap", "sdma_layerwise_overlap"):
            main_s.wait_stream(xfer_s)

    modes = ["prefill", "one_launch_after", "layerwise_overlap", "layerwise_after"]
    sdma_calls = []
    if layout == fk.LAYOUT_LAYER_MAJOR:
        # copy-engine comparators: one 1-D copy per (layer, K or V, run); a
        # layer tensor is (2, B, H) bytes, so K/V piece kv of blocks
        # [b, b + k) is the contiguous range ((kv * B + b) * H, k * H)
        hip = ctypes.CDLL(fk._hip_runtimes_loaded()[0])
        hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                       ctypes.c_int, ctypes.c_void_p]
        hip.hipMemcpyAsync.restype = ctypes.c_int
        H = geom.chunk_bytes
        for layer in range(geom.num_layers):
            calls = []
            for rec in segs:
                b_s, b_d, k = int(rec["src_block"]), int(rec["dst_block"]), int(rec["n_blocks"])
                assert 0 <= b_s and b_s + k <= src.num_blocks and 0 <= b_d
                assert b_d + k <= dst.num_blocks
                for kv in range(2):
                    calls.append((dst.tensors[layer].data_ptr() + (kv * dst.num_blocks + b_d) * H,
                                  src.tensors[layer].data_ptr() + (kv * src.num_blocks + b_s) * H,
                                  k * H))
            sdma_calls.append(calls)
        modes += ["sdma_layerwise_overlap", "sdma_after"]

    def sdma_layer(layer, stream):
        for d_ptr, s_ptr, nbytes in sdma_calls[layer]:
            rc = hip.hipMemcpyAsync(d_ptr, s_ptr, nbytes, 1024, stream.cuda_stream)
            assert rc == 0, f"hipMemcpyAsync: error {rc}"
    for _ in range(max(1, args.warmup)):
        for m in modes:
            run(m)
    torch.cuda.synchronize()
    # every block moved, in the last form run (spot check of the first, a
    # middle and the last block)
    for i in sorted({0, n // 2, n - 1}):
        if layout == fk.LAYOUT_BLOCK_MAJOR:
            ok = torch.equal(src.tensors[0][int(S[i])], dst.tensors[0][int(D[i])])
        else:
            ok = all(torch.equal(a[:, int(S[i])], b[:, int(D[i])])
                     for a, b in zip(src.tensors, dst.tensors))
        assert ok, f"block {i} not moved"

    times = {m: [] for m in modes}
    gc.collect()
    gc.disable()
    t0 = time.perf_counter()
    for r in range(args.steps):
        # interleaved, in an order rotated every round, and each form started
        # after two untimed prefill layers: a form that leaves the compute
        # units idle (the copy-engine form runs 50 ms on them alone) must not
        # slow down whichever form follows it
        for m in modes[r % len(modes):] + modes[:r % len(modes)]:
            prefill_layer()
            prefill_layer()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(main_s)
            run(m)
            e1.record(main_s)
            e1.synchronize()
            times[m].append(e0.elapsed_time(e1))
    elapsed = time.perf_counter() - t0
    gc.enable()
    med = {m: statistics.median(v) for m, v in times.items()}
    # exposed transfer time per round: a form minus the prefill-alone run of
    # the same round (pairing removes the drift of the prefill's own time,
    # which varies by about half a millisecond from round to round)
    diffs = {m: sorted(a - b for a, b in zip(times[m], times["prefill"])) for m in modes[1:]}
    exposed = {m: round(statistics.median(d), 4) for m, d in diffs.items()}
    spread = {m: [round(d[len(d) // 4], 4), round(d[(3 * len(d)) // 4], 4)]
              for m, d in diffs.items()}
    line = {
        "metric": "KV transfer time exposed after a 13,000-token prefill, layer-wise overlap",
        "value": exposed["layerwise_overlap"], "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(elapsed * 1e3 / args.steps, 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": "llama3-8b-13k-prefill-then-kv-transfer", "tokens": T,
                   "layers": geom.num_layers, "blocks": n, "runs": len(segs),
                   "layout": f"{args.layout}-major",
                   "prefill_stand_in": "4 projection products per layer (q, kv, o, gate/up, "
                                       "down), bf16 torch.matmul",
                   "prefill_tflop": round(flops_layer * geom.num_layers / 1e12, 2)},
        "median_ms": {m: round(v, 4) for m, v in med.items()},
        "exposed_ms": exposed,
        "exposed_ms_p25_p75": spread,
        "prefill_tflops": round(flops_layer * geom.num_layers / (med["prefill"] * 1e-3) / 1e12,
                                1),
        "roofline": None,
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


TABLE3_LENGTHS = [500, 1000, 2000, 4000, 8000, 10000, 12000]
# Table 3's FlowKV and FlowKV-Layerwise transfer latencies in seconds, single
# L20 server (NVIDIA, NCCL): context only, another machine and another link
TABLE3_PAPER_S = {500: (0.0044, 0.0678), 1000: (0.0075, 0.1309), 2000: (0.0126, 0.2565),
                  4000: (0.0236, 0.5338), 8000: (0.0447, 1.1173), 10000: (0.0555, 1.4121),
                  12000: (0.0681, 1.7218)}


def bench_table3(args):
    """FlowKV vs FlowKV-Layerwise across input lengths (section 4.4, Table
    3) on one MI355X: Llama-3-8B KV of one request of T tokens for each of
    the table's lengths, moved between the bench's two 65,536-block pools
    (sender blocks from the segment allocator, receiver blocks from the
    seeded free list of the 30%-occupied pool), in two forms:
      one_launch  the whole plan in one launch (plan in the kernel arguments
                  when it fits there, else staged);
      layerwise   32 launches, one per layer (K and V of that layer);
    and, by kernel time only, the layerwise launches replayed from a HIP
    graph captured once (layerwise_graph).
    Per form and length: the median kernel time (HIP events around the
    launches), the step time back to back, and the synchronised request
    latency (plan, staging, launches and kernels, synchronised; median of
    20).  `value` is the mean synchronised one-launch latency over the
    lengths (the paper's column mean, 0.0309 s on one L20 server)."""
    import torch

    from paper_2504_03775_amd import flowkv as fk
    from workloads import make_device_pool, recipes

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = fk.LAYOUT_BLOCK_MAJOR if args.layout == "block" else fk.LAYOUT_LAYER_MAJOR
    lengths = [int(x) for x in args.lengths.split(",")] if args.lengths else TABLE3_LENGTHS
    make_alloc = lambda P, pol, seed: fk.Allocator(P, pol, seed)  # noqa: E731
    wl0 = recipes.llama8b_13k(make_alloc, args.dst_policy, tokens=max(lengths),
                              occupied=args.dst_occupied)
    geom = wl0.geom
    src = fk.KVPool(layout, make_device_pool(geom, layout, wl0.src_pool_blocks, dev, seed=0))
    dst = fk.KVPool(layout, make_device_pool(geom, layout, wl0.dst_pool_blocks, dev, seed=1))
    stream = torch.cuda.current_stream()
    stager = fk.PlanStager(dev, capacity=4096)
    rows = []
    gc.collect()
    for T in lengths:
        wl = recipes.llama8b_13k(make_alloc, args.dst_policy, tokens=T,
                                 occupied=args.dst_occupied)
        (S, D), = wl.tables
        n = len(S)

        def step(form, ev=None):
            segs = fk.flowkv_plan(S, D, src.num_blocks, dst.num_blocks)
            inline = form == "one_launch" and len(segs) <= fk.inline_capacity(src, dst)
            segs_dev = None if inline else stager.stage(segs, stream)
            if ev is not None:
                ev[0].record(stream)
            if inline:
                fk.flowkv_transfer_inline(src, dst, segs, n, stream=stream)
            elif form == "one_launch":
                fk.flowkv_transfer_ex(src, dst, segs_dev, len(segs), n, stream=stream)
            else:
                for layer in range(geom.num_layers):
                    fk.flowkv_transfer_layers(src, dst, segs_dev, len(segs), n, layer, 1,
                                              stream=stream)
            if ev is not None:
                ev[1].record(stream)
            if not inline:
                stager.release(stream)
            return len(segs)

        row = {"tokens": T, "blocks": n, "payload_bytes": n * geom.block_bytes}
        for form in ("one_launch", "layerwise"):
            runs = step(form)
            torch.cuda.synchronize()
            i = n // 2
            if layout == fk.LAYOUT_BLOCK_MAJOR:
                assert torch.equal(src.tensors[0][int(S[i])], dst.tensors[0][int(D[i])])
            for _ in range(args.warmup):
                step(form)
            evs = timing_pairs(args.steps)
            torch.cuda.synchronize()
            gc.disable()
            t0 = time.perf_counter()
            for e in evs:
                step(form, e)
            torch.cuda.synchronize()
            el = time.perf_counter() - t0
            lat = []
            for _ in range(20):
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                step(form)
                torch.cuda.synchronize()
                lat.append((time.perf_counter() - t1) * 1e3)
            gc.enable()
            k_ms = statistics.median(a.elapsed_time(b) for a, b in evs)
            row[form] = {"kernel_ms_median": round(k_ms, 4),
                         "ms_per_step": round(el * 1e3 / args.steps, 4),
                         "latency_ms_median": round(statistics.median(lat), 4),
                         "launches": 1 if form == "one_launch" else geom.num_layers,
                         "hbm_frac": round(2 * n * geom.block_bytes / (k_ms * 1e-3) / 1e9
                                           / HBM_PEAK_GBPS, 4)}
            row["runs"] = runs
        row["layerwise_over_one_launch"] = {
            k: round(row["layerwise"][k] / row["one_launch"][k], 2)
            for k in ("kernel_ms_median", "ms_per_step", "latency_ms_median")}
        # the same 32 per-layer launches captured once in a HIP graph and
        # replayed: what the gaps between dispatches cost.  The plan is fixed
        # at capture, so only the kernel time compares.
        segs = fk.flowkv_plan(S, D, src.num_blocks, dst.num_blocks)
        segs_g = fk.segments_to_device(segs, dev)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for layer in range(geom.num_layers):
                fk.flowkv_transfer_layers(src, dst, segs_g, len(segs), n, layer, 1)
        for _ in range(max(1, args.warmup)):
            graph.replay()
        evs = timing_pairs(args.steps)
        torch.cuda.synchronize()
        for e in evs:
            e[0].record(stream)
            graph.replay()
            e[1].record(stream)
        torch.cuda.synchronize()
        k_g = statistics.median(a.elapsed_time(b) for a, b in evs)
        row["layerwise_graph"] = {"kernel_ms_median": round(k_g, 4),
                                  "launches": geom.num_layers,
                                  "over_one_launch": round(
                                      k_g / row["one_launch"]["kernel_ms_median"], 2)}
        del graph, segs_g
        if T in TABLE3_PAPER_S:
            row["paper_s_single_l20"] = dict(zip(("flowkv", "flowkv_layerwise"),
                                                 TABLE3_PAPER_S[T]))
        rows.append(row)
        print(f"table3 {T} tokens: one launch {row['one_launch']['latency_ms_median']} ms, "
              f"per-layer {row['layerwise']['latency_ms_median']} ms", file=sys.stderr,
              flush=True)
    mean_lat = statistics.fmean(r["one_launch"]["latency_ms_median"] for r in rows)
    line = {
        "metric": "KV transfer latency per request, one launch (Table 3 FlowKV column, mean "
                  "over input lengths)",
        "value": round(mean_lat, 4), "unit": "ms", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(statistics.fmean(
            r["one_launch"]["ms_per_step"] for r in rows), 4),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic",
        "config": {"workload": "llama3-8b-kv-one-request-table3-lengths", "lengths": lengths,
                   "layers": geom.num_layers, "kv_heads": geom.kv_heads,
                   "head_dim": geom.head_dim, "block_size": geom.block_size,
                   "kv_dtype": "bf16", "pool_blocks": [src.num_blocks, dst.num_blocks],
                   "layout": f"{args.layout}-major", "receiver_policy": args.dst_policy,
                   "receiver_occupied": args.dst_occupied},
        "timing_events": TIMING["events"],
        "rows": rows,
        "roofline": None,
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): both pools of "
              "the transfer live on one device.", file=sys.stderr)
        sys.exit(2)
    if args.op == "attention":
        bench_attention(args)
        return
    if args.op == "schedule":
        bench_schedule(args)
        return
    if args.op == "overlap":
        bench_overlap(args)
        return
    if args.op == "table3":
        bench_table3(args)
        return

    import numpy as np
    import torch

    from paper_2504_03775_amd import flowkv as fk
    from workloads import (SEED_DST_TABLE, SEED_OCCUPANCY, make_device_pool,
                           occupied_blocks, recipes)
    from workloads.recipes import POLICIES

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    layout = fk.LAYOUT_BLOCK_MAJOR if args.layout == "block" else fk.LAYOUT_LAYER_MAJOR
    single = args.workload == "8b"

    # ---- setup (untimed): block lists, pools ------------------------------------
    make_alloc = lambda P, pol, seed: fk.Allocator(P, pol, seed)  # noqa: E731
    recipe, rargs, wl_desc = WORKLOADS[args.workload]
    shrunk = None
    if single:
        wl = recipes.llama8b_13k(make_alloc, args.dst_policy, occupied=args.dst_occupied)
        # a device without room for both 65,536-block pools gets a smaller
        # receiver pool (the request's 813 blocks still fit at 30% occupancy)
        free, _ = torch.cuda.mem_get_info()
        fit = fit_receiver_blocks(free, wl.src_pool_blocks, wl.dst_pool_blocks,
                                  wl.geom.block_bytes)
        if 0 < fit < wl.dst_pool_blocks:
            shrunk = {"receiver_pool_blocks_from": wl.dst_pool_blocks, "to": fit,
                      "reason": f"{free / 2**30:.1f} GiB of device memory free"}
            print(f"receiver pool shrunk to {fit} blocks: {shrunk['reason']}", file=sys.stderr)
            wl = recipes.llama8b_13k(make_alloc, args.dst_policy, dst_pool_blocks=fit,
                                     occupied=args.dst_occupied)
    elif recipe == "tiny":
        wl = recipes.tiny()
    else:
        wl = getattr(recipes, recipe)(make_alloc, *rargs)
    geom = wl.geom
    S_all, D_all = wl.flat()
    n = len(S_all)
    offsets = wl.offsets()
    payload = n * geom.block_bytes
    src_blocks, dst_blocks = wl.src_pool_blocks, wl.dst_pool_blocks

    free, _ = torch.cuda.mem_get_info()
    need = (src_blocks + dst_blocks) * geom.block_bytes
    if need > free - RESERVE_BYTES:
        raise SystemExit(f"pools need {need / 2**30:.1f} GiB, {free / 2**30:.1f} GiB free")
    t0 = time.perf_counter()
    src = fk.KVPool(layout, make_device_pool(geom, layout, src_blocks, dev, seed=0))
    dst = fk.KVPool(layout, make_device_pool(geom, layout, dst_blocks, dev, seed=1))
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    cfg = dict(threads=args.threads, unroll=args.unroll, grid=args.grid, cache=args.cache,
               order=args.order)
    stream = torch.cuda.current_stream()
    stager = fk.PlanStager(dev, capacity=max(1, n))

    def single_request_steps(policy):
        """(make_plan, after_launch, receiver_list) of the 13k request for a
        receiver policy.  The segment allocator runs inside every step on the
        30%-occupied pool: the request's blocks are taken and released again,
        and releasing merges them back, so every step sees the same state.  A
        free list hands out other blocks after every release, so for it the
        receiver's table is the one the seeded free list gave at setup (the
        recipe's), planned and moved every step."""
        if policy == "segment":
            alloc = fk.Allocator(dst_blocks, POLICIES[policy], SEED_DST_TABLE)
            alloc.mark_used(occupied_blocks(dst_blocks, args.dst_occupied, SEED_OCCUPANCY))

            def plan_seg():
                D = alloc.alloc(n)
                return fk.flowkv_plan(S_all, D, src_blocks, dst_blocks), D

            def release(D):
                alloc.free(D)

            def table():
                D = alloc.alloc(n)
                alloc.free(D)
                return D
            return plan_seg, release, table
        D_fixed = D_all if policy == args.dst_policy else recipes.llama8b_13k(
            make_alloc, policy, dst_pool_blocks=dst_blocks, occupied=args.dst_occupied).tables[0][1]

        def plan_fixed():
            return fk.flowkv_plan(S_all, D_fixed, src_blocks, dst_blocks), None
        return plan_fixed, (lambda _: None), (lambda: D_fixed)

    if single:
        make_plan, after_launch, receiver_list = single_request_steps(args.dst_policy)
    else:
        def make_plan():
            return fk.flowkv_plan_batch(offsets, S_all, D_all, src_blocks, dst_blocks), None

        def after_launch(_):
            pass

        def receiver_list():
            return D_all

    def step(events=None, fns=None):
        plan_fn, release_fn = fns or (make_plan, after_launch)
        segs, token = plan_fn()
        # small plans ride in the kernel arguments; longer ones are staged
        inline = (len(segs) <= fk.inline_capacity(src, dst) and not args.layerwise
                  and not args.staged_plan)
        segs_dev = None if inline else stager.stage(segs, stream)
        if events is not None:
            events[0].record(stream)
        if inline:
            fk.flowkv_transfer_inline(src, dst, segs, n, stream=stream, **cfg)
        elif args.layerwise:
            for layer in range(geom.num_layers):
                fk.flowkv_transfer_layers(src, dst, segs_dev, len(segs), n, layer, 1,
                                          stream=stream, **cfg)
        else:
            fk.flowkv_transfer_ex(src, dst, segs_dev, len(segs), n, stream=stream, **cfg)
        if events is not None:
            events[1].record(stream)
        if not inline:
            stager.release(stream)
        release_fn(token)
        return segs

    def spot_check(D_chk):
        """A few moved blocks byte-equal (first, middle, last)."""
        for i in sorted({0, n // 2, n - 1}):
            if layout == fk.LAYOUT_BLOCK_MAJOR:
                ok = torch.equal(src.tensors[0][int(S_all[i])], dst.tensors[0][int(D_chk[i])])
            else:
                ok = all(torch.equal(t_s[:, int(S_all[i])], t_d[:, int(D_chk[i])])
                         for t_s, t_d in zip(src.tensors, dst.tensors))
            assert ok, f"block {i} not moved"

    segs = step()
    torch.cuda.synchronize()
    n_runs = len(segs)
    spot_check(receiver_list())

    # Python's cyclic garbage collector is run before the warmup and kept off
    # through the timed steps (as timeit does): a full collection of the
    # interpreter's heap can stall the host for tens of milliseconds, and run
    # between the warmup and the timed steps it would leave the GPU idle
    # right before them
    evs = timing_pairs(args.steps)
    gc.collect()
    gc.disable()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # ---- timed region -----------------------------------------------------------
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.enable()
    kern_ms = [a.elapsed_time(b) for a, b in evs]
    kern_avg_ms = statistics.fmean(kern_ms)
    ms_per_step = elapsed * 1e3 / args.steps
    value = payload * args.steps / elapsed / 1e9
    algo_bytes = 2 * payload + 16 * n_runs
    achieved = algo_bytes / (kern_avg_ms * 1e-3) / 1e9

    # ---- latency: one plan end to end, synchronised --------------------------------
    lat = []
    for _ in range(20):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        step()
        torch.cuda.synchronize()
        lat.append((time.perf_counter() - t1) * 1e3)
    ms_latency = statistics.median(lat)

    context = {}
    if not args.no_context:
        # kernel time with the 256 MB last-level cache flushed before each launch
        flushed = []
        if not args.calibration_only:
            scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
            for _ in range(10):
                scratch.fill_(1)
                e = timing_pairs(1)[0]
                step(e)
                torch.cuda.synchronize()
                flushed.append(e[0].elapsed_time(e[1]))
            del scratch
        # plain contiguous device-to-device copy: the practical copy ceiling
        # (also the HBM counter calibration kernel)
        nbytes = int(args.calibrate_copy_gib * (1 << 30))
        a = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            b.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        copy_ms = e0.elapsed_time(e1) / 10
        del a, b
        context = {
            "kernel_ms_cache_flushed_median": round(statistics.median(flushed), 4) if flushed else None,
            "contiguous_copy_gbps": round(2 * nbytes / (copy_ms * 1e-3) / 1e9, 1),
            "contiguous_copy_bytes": nbytes,
        }
        # the paper's block-wise pattern: one copy call per (block, layer, K/V)
        # chunk, here as device-to-device copies of the same request
        if single and not args.calibration_only:
            D = receiver_list()
            t_chunks = time.perf_counter()
            calls = 0
            if layout == fk.LAYOUT_BLOCK_MAJOR:
                sv = src.tensors[0].view(src_blocks, 2 * geom.num_layers, -1)
                dv = dst.tensors[0].view(dst_blocks, 2 * geom.num_layers, -1)
                for i in range(n):
                    for r in range(2 * geom.num_layers):
                        dv[int(D[i]), r].copy_(sv[int(S_all[i]), r])
                        calls += 1
                del sv, dv
            else:
                for ts, td in zip(src.tensors, dst.tensors):
                    for kv in range(2):
                        for i in range(n):
                            td[kv, int(D[i])].copy_(ts[kv, int(S_all[i])])
                            calls += 1
                del ts, td
            torch.cuda.synchronize()
            context["per_chunk_copy_calls"] = calls
            context["per_chunk_copy_ms"] = round((time.perf_counter() - t_chunks) * 1e3, 2)
            # one copy per aligned run (per run, layer and K/V in the layer-major
            # layout): the call pattern of a per-run transfer API
            segs_h = fk.flowkv_plan(S_all, D, src_blocks, dst_blocks)
            torch.cuda.synchronize()
            t_runs = time.perf_counter()
            calls = 0
            if layout == fk.LAYOUT_BLOCK_MAJOR:
                for sg in segs_h:
                    s0, d0, m = int(sg["src_block"]), int(sg["dst_block"]), int(sg["n_blocks"])
                    dst.tensors[0][d0:d0 + m].copy_(src.tensors[0][s0:s0 + m])
                    calls += 1
            else:
                for ts, td in zip(src.tensors, dst.tensors):
                    for kv in range(2):
                        for sg in segs_h:
                            s0, d0 = int(sg["src_block"]), int(sg["dst_block"])
                            m = int(sg["n_blocks"])
                            td[kv, d0:d0 + m].copy_(ts[kv, s0:s0 + m])
                            calls += 1
                del ts, td
            torch.cuda.synchronize()
            context["per_run_copy_calls"] = calls
            context["per_run_copy_ms"] = round((time.perf_counter() - t_runs) * 1e3, 3)
        # the other receiver policy, timed the same way in the same run (the
        # segment allocator beside the seeded free list, or the reverse)
        if single and not args.calibration_only and not args.layerwise:
            alt = "segment" if args.dst_policy != "segment" else "fifo_sorted"
            plan_alt, release_alt, table_alt = single_request_steps(alt)
            fns = (plan_alt, release_alt)
            segs_alt = step(fns=fns)
            torch.cuda.synchronize()
            spot_check(table_alt())
            evs_alt = timing_pairs(args.steps)
            gc.collect()
            gc.disable()
            for _ in range(args.warmup):
                step(fns=fns)
            torch.cuda.synchronize()
            t_alt = time.perf_counter()
            for e in evs_alt:
                step(e, fns=fns)
            torch.cuda.synchronize()
            el_alt = time.perf_counter() - t_alt
            gc.enable()
            k_alt = statistics.fmean(a.elapsed_time(b) for a, b in evs_alt)
            context[f"receiver_{alt}"] = {
                "runs": len(segs_alt),
                "plan_in": ("kernel-arguments" if len(segs_alt) <= fk.inline_capacity(src, dst)
                            and not args.staged_plan else "device-memory"),
                "kernel_ms_avg": round(k_alt, 4),
                "roofline_frac": round((2 * payload + 16 * len(segs_alt)) / (k_alt * 1e-3) / 1e9
                                       / HBM_PEAK_GBPS, 4),
                "ms_per_step": round(el_alt * 1e3 / args.steps, 4)}
        # the headline's own plan read from device memory (uploaded once,
        # outside the timing) instead of the kernel arguments: the kernel
        # time the argument form costs, against the plan copy it saves
        if (single and not args.calibration_only and not args.layerwise
                and not args.staged_plan and n_runs <= fk.inline_capacity(src, dst)):
            segs_d = fk.segments_to_device(segs, dev)
            for _ in range(args.warmup):
                fk.flowkv_transfer_ex(src, dst, segs_d, n_runs, n, stream=stream, **cfg)
            evs_dp = timing_pairs(args.steps)
            torch.cuda.synchronize()
            for e in evs_dp:
                e[0].record(stream)
                fk.flowkv_transfer_ex(src, dst, segs_d, n_runs, n, stream=stream, **cfg)
                e[1].record(stream)
            torch.cuda.synchronize()
            k_dp = statistics.fmean(a.elapsed_time(b) for a, b in evs_dp)
            context["plan_in_device_memory"] = {
                "runs": n_runs, "kernel_ms_avg": round(k_dp, 4),
                "roofline_frac": round((2 * payload + 16 * n_runs) / (k_dp * 1e-3) / 1e9
                                       / HBM_PEAK_GBPS, 4),
                "note": "the same plan and launch shape, the plan uploaded to device memory "
                        "once before the timing"}
            del segs_d
        # the same kernel on a plan of one run of the same bytes (sender
        # blocks [0, n) to receiver blocks [0, n)): the copy's own ceiling
        # for these pools, against which the plan's run structure is judged
        if single and not args.calibration_only and not args.layerwise:
            one = np.array([(0, 0, n, 0)], dtype=fk.SEGMENT_DTYPE)
            for _ in range(args.warmup):
                fk.flowkv_transfer_inline(src, dst, one, n, stream=stream, **cfg)
            evs_one = timing_pairs(args.steps)
            torch.cuda.synchronize()
            for e in evs_one:
                e[0].record(stream)
                fk.flowkv_transfer_inline(src, dst, one, n, stream=stream, **cfg)
                e[1].record(stream)
            torch.cuda.synchronize()
            k_one = statistics.fmean(a.elapsed_time(b) for a, b in evs_one)
            context["single_run_plan"] = {
                "runs": 1, "kernel_ms_avg": round(k_one, 4),
                "roofline_frac": round((2 * payload + 16) / (k_one * 1e-3) / 1e9
                                       / HBM_PEAK_GBPS, 4),
                "note": "the same kernel, sender blocks [0, n) to receiver blocks [0, n)"}

    # ---- CPU baseline: the oracle on the host ----------------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        import oracle

        # a bounded sample: at most 813 blocks (one 13k-token request's worth)
        k = min(n, 813)
        pick = np.linspace(0, n - 1, k).round().astype(np.int64) if n > k else np.arange(n)
        idx = torch.as_tensor(S_all[pick].astype(np.int64), device=dev)
        slot = geom.slot_bytes
        h_src = oracle.HostPool.zeros(layout, geom.num_layers, k, geom.block_size, slot)
        if layout == fk.LAYOUT_BLOCK_MAJOR:
            h_src.buffers[0][:] = src.tensors[0].index_select(0, idx).view(torch.uint8) \
                .reshape(-1).cpu().numpy()
        else:
            for l, t in enumerate(src.tensors):
                h_src.buffers[l][:] = t.index_select(1, idx).contiguous().view(torch.uint8) \
                    .reshape(-1).cpu().numpy()
        h_dst = oracle.HostPool.zeros(layout, geom.num_layers, k, geom.block_size, slot)
        reps, t_cpu = 0, 0.0
        while t_cpu < 10.0 and reps < 100:
            t1 = time.perf_counter()
            oracle.transfer_fast(h_src, h_dst, np.arange(k), np.arange(k))
            t_cpu += time.perf_counter() - t1
            reps += 1
        sample_bytes = k * geom.block_bytes
        # the same oracle call per layer on a thread pool (numpy's copies
        # release the interpreter lock): the host's cores together
        from concurrent.futures import ThreadPoolExecutor
        threads = min(16, os.cpu_count() or 1, geom.num_layers)
        ids = np.arange(k)
        with ThreadPoolExecutor(threads) as ex:
            reps_m, t_m = 0, 0.0
            while t_m < 5.0 and reps_m < 200:
                t1 = time.perf_counter()
                list(ex.map(lambda l: oracle.transfer_fast(h_src, h_dst, ids, ids, layers=[l]),
                            range(geom.num_layers)))
                t_m += time.perf_counter() - t1
                reps_m += 1
        cpu = {"value": round(sample_bytes * reps / t_cpu / 1e9, 3), "unit": "GB/s", "cores": 1,
               "kind": "oracle",
               "sample": f"{k} of the workload's {n} blocks ({sample_bytes} B), repeated {reps}x, "
                         f"compact host pools of those blocks, numpy one thread; "
                         f"{os.cpu_count()} host cores visible",
               "multi_thread": {"value": round(sample_bytes * reps_m / t_m / 1e9, 3),
                                "cores": threads,
                                "sample": f"the same, one oracle call per layer on {threads} "
                                          f"threads, repeated {reps_m}x"}}
        del h_src, h_dst

    summary = PMC_SUMMARIES.get((args.workload, args.layout))
    traffic = traffic_from_profile(summary, runs=n_runs) if summary and not args.layerwise \
        else None
    kv_dtype = {"bfloat16": "bf16", "float16": "fp16"}[geom.dtype]
    config = {"workload": wl_desc, "layers": geom.num_layers, "kv_heads": geom.kv_heads,
              "head_dim": geom.head_dim, "block_size": geom.block_size, "kv_dtype": kv_dtype,
              "requests": len(wl.tables), "blocks": n, "payload_bytes": payload,
              "pool_blocks": [src_blocks, dst_blocks], "layout": f"{args.layout}-major",
              "runs": n_runs}
    if single:
        config.update(receiver_policy=args.dst_policy, receiver_occupied=args.dst_occupied)
        if shrunk:
            config["receiver_pool_shrunk"] = shrunk
    if args.layerwise:
        config.update(launches_per_step=geom.num_layers, mode="layer-wise")
    config["plan_in"] = ("kernel-arguments" if n_runs <= fk.inline_capacity(src, dst)
                         and not args.layerwise and not args.staged_plan else "device-memory")
    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic",
        "config": config,
        "value_is": "payload bytes (each K/V byte moved counted once) per second of the "
                    "timed back-to-back steps",
        ("ms_per_request" if single else "ms_per_plan_latency"): round(ms_latency, 4),
        "hbm_gbps": round(achieved, 1),
        "pct_of_hbm_peak": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "hbm_is": "bytes read plus bytes written by the kernel per second of its own "
                  "launches (HIP events)",
        "kernel_ms_avg": round(kern_avg_ms, 4),
        "kernel_ms_p10_p50_p90": [round(float(x), 4) for x in
                                  np.percentile(np.asarray(kern_ms), [10, 50, 90])],
        "timing_events": TIMING["events"],
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "context": context,
        "setup_s": round(setup_s, 2),
    }
    # the decode attention that reads the receiver pool, timed in the same
    # run (the default line only): the transfer pools are freed first
    if (single and not args.no_context and not args.calibration_only and not args.layerwise
            and args.workload == "8b" and args.layout == "block"):
        del src, dst, stager
        gc.collect()
        torch.cuda.empty_cache()
        context["decode_attention"] = attention_context(args.steps)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
