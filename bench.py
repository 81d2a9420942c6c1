"""Throughput of the whole integrity path on one MI355X, as one JSON line.

A step is one pass of the path over the resident weight set: SHA-256 of every
chunk, RFC 6962 roots per tensor, the manifest root over them, and the on-GPU
comparison of that root with the expected one (synchronous).  Default
workload: the 70B-shaped bf16 weight set (723 tensors, 141.1 GB, 64 KiB
chunks), generated on the GPU before timing; the bytes are already in HBM
when the timed region starts.

    python bench.py [--steps K] [--warmup W] [--config 1..5] [--alg sha256|sha384] [--no-cpu-baseline]

Also reported: the roofline of the dominant kernel (the leaf kernel, timed
with HIP events on its own stream) against the integer-VALU peak, and the CPU
oracle timed on a bounded sample of the same bytes on this host.  With
--alg sha384 every digest and node is SHA-384 (48 bytes, 128-byte blocks).
"""
import argparse
import gc
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GB/s hashed+Merkle-verified on 1 MI355X; % of integer-VALU/HBM roofline"
# Integer VALU peak: 256 CUs x 4 SIMD x 16 lanes x 2.4 GHz, one 32-bit op per lane per cycle.
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# 32-bit VALU ops per SHA-256 block on gfx950 at the ISA minimum: 64 rounds x 14,
# 48 schedule words x 10, 8 feed-forward adds, 16 byte swaps.
OPS_PER_BLOCK = 64 * 14 + 48 * 10 + 8 + 16
# The same for a SHA-384 block (128 bytes) with 64-bit words as 32-bit halves:
# 80 rounds x (Sigma0, Sigma1: 6 alignbit + 2 bitop3 each; Ch, Maj: 2 bitop3
# each; 7 64-bit adds as one v_lshl_add_u64 each), 64 schedule words x
# (sigma0, sigma1: 8 each; 3 adds), 8 feed-forward adds, 32 byte swaps.
OPS_PER_BLOCK_384 = 80 * 27 + 64 * 19 + 8 + 32
# Issue cycles per wave-block if every double-rate instruction (v_bitop3, v_add_u32,
# v_lshrrev: two per quad-cycle when two waves offer them together) paired up and
# the others (v_alignbit, v_add3, v_perm, v_lshl_add_u64) took a quad-cycle each:
# SHA-256 832 x 4 + 568 x 2, SHA-384 2392 x 4 + 1024 x 2.  The bound on the mix
# that this dual issue allows, beside the one-op-per-lane-cycle peak.
DUAL_ISSUE_CYCLES = {"sha256": 832 * 4 + 568 * 2, "sha384": 2392 * 4 + 1024 * 2}
CSRC = "paper_2510_23938_amd/csrc/"
# per hash: block bytes, length-field bytes, ops per block, leaf kernel, traffic summary, kernel sources
ALGS = {
    "sha256": (64, 8, OPS_PER_BLOCK, "sha256_leaves_kernel", "sha256_leaves_traffic.json",
               [CSRC + "sha256_leaves.hip", CSRC + "sha256_device.h"]),
    "sha384": (128, 16, OPS_PER_BLOCK_384, "sha384_leaves_kernel", "sha384_leaves_traffic.json",
               [CSRC + "sha384_leaves.hip", CSRC + "sha384_device.h"]),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(alg="sha256"):
    h = hashlib.sha256()
    for p in ALGS[alg][5]:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def sha_blocks(lens, C, alg="sha256"):
    """Blocks the leaf kernel compresses (data + padding: 0x80 and the length
    field), from the message lengths and the chunk size."""
    B, lf = ALGS[alg][0], ALGS[alg][1]
    lens = np.asarray(lens, dtype=np.uint64).astype(object)
    total = 0
    for L in lens:
        L = int(L)
        if C == 0:
            total += (L + lf + B) // B
            continue
        full, tail = divmod(L, C)
        total += full * ((C + lf + B) // B)
        if tail:
            total += (tail + lf + B) // B
    return total


def traffic_for_current_kernel(alg="sha256", config=5):
    """HBM bytes per leaf-kernel launch from the committed rocprofv3 counter
    summary, or None when it is missing, covers another workload or was taken
    on different kernel code."""
    try:
        with open(os.path.join(ROOT, "profiles", ALGS[alg][4])) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash(alg) or rec.get("config", 5) != config:
        return None
    return rec.get("hbm_bytes_per_launch")


def host_cpu_info():
    """The host CPU as lscpu reports it (model, sockets, cores, SMT), else /proc/cpuinfo's model name."""
    info = {"host_cpu": "", "host_cpus_visible": os.cpu_count()}
    fields = {"Model name": "host_cpu", "Socket(s)": "host_sockets", "Core(s) per socket": "host_cores_per_socket",
              "Thread(s) per core": "host_threads_per_core"}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10, check=True).stdout
        for ln in out.splitlines():
            key, _, val = ln.partition(":")
            if key.strip() in fields:
                val = val.strip()
                info[fields[key.strip()]] = int(val) if val.isdigit() else val
    except (OSError, subprocess.SubprocessError):
        pass
    if not info["host_cpu"]:
        try:
            with open("/proc/cpuinfo") as f:
                info["host_cpu"] = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), "")
        except OSError:
            pass
    return info


def cpu_baseline(wl, pipe, sample_bytes, alg="sha256"):
    """The oracle (plain C, threaded over chunks) on the first whole chunks of
    the first messages, about sample_bytes in all, one message at a time so
    that host memory stays bounded; only the oracle's work is timed.  Also
    checks those digests against the GPU's, and the root of every message
    sampled whole against the GPU's root of that message."""
    from oracle import oracle

    C = wl.chunk_bytes
    views = wl.msgs.views
    threads = min(16, len(os.sched_getaffinity(0)))
    gpu = pipe.leaves
    left, nbytes, n_leaves, n_msgs, dt, ok = sample_bytes, 0, 0, 0, 0.0, True
    roots_checked = roots_ok = 0
    if views is None and C == 0 and len(wl.msgs) > 1:
        # many whole messages packed in one buffer: copy the sampled range once
        # and hash it with the oracle's packed driver (one message at a time
        # would time per-message copies and calls instead of hashing)
        lens = np.asarray(wl.msgs.lens, dtype=np.uint64)
        offs = np.asarray(wl.msgs.offsets, dtype=np.uint64)
        k = max(1, int(np.searchsorted(np.cumsum(lens), sample_bytes, side="left")) + 1)
        k = min(k, len(lens))
        end = int(offs[k - 1] + lens[k - 1])
        host = wl.msgs.buffer[:end].cpu().numpy()
        t0 = time.perf_counter()
        leaves = oracle.leaf_digests_mt_packed(host, offs[:k], lens[:k], 0, threads, alg)
        oracle.mth(leaves, alg)
        dt = time.perf_counter() - t0
        ok = bool(np.array_equal(gpu[:k].cpu().numpy(), leaves))
        if k == len(lens):  # every message sampled: the single tree's root too
            roots_checked, roots_ok = 1, int(bytes(pipe.root.cpu().numpy().reshape(-1)) == oracle.mth(leaves, alg))
        nbytes, n_leaves, n_msgs, left = int(lens[:k].sum()), k, k, 0
        del host
    for m in range(len(wl.msgs)):
        if left <= 0:
            break
        L = int(wl.msgs.lens[m])
        n = L if C == 0 else min(L, -(-left // C) * C)  # whole messages / whole chunks
        if views is not None:
            src = views[m][:n]
        else:
            o = int(wl.msgs.offsets[m])
            src = wl.msgs.buffer[o:o + n]
        host = src.cpu().numpy()
        t0 = time.perf_counter()
        leaves = oracle.leaf_digests_mt([host], C, threads, alg)
        root = oracle.mth(leaves, alg)
        dt += time.perf_counter() - t0
        first = int(pipe.seg[m])
        ok &= bool(np.array_equal(gpu[first:first + len(leaves)].cpu().numpy(), leaves))
        if n == L and (wl.manifest or len(wl.msgs) == 1):  # the whole message was sampled: its root too
            roots_checked += 1
            gpu_root = pipe.roots[m] if wl.manifest else pipe.root.reshape(-1)
            roots_ok += int(bytes(gpu_root.cpu().numpy()) == root)
        nbytes += n
        n_leaves += len(leaves)
        n_msgs += 1
        left -= n
        del host
    # one thread on the first 1 GiB: the oracle's rate per core
    first = views[0][: min(1 << 30, int(wl.msgs.lens[0]))] if views is not None else \
        wl.msgs.buffer[: min(1 << 30, int(wl.msgs.offsets[-1] + wl.msgs.lens[-1]))]
    host = first.cpu().numpy()
    t0 = time.perf_counter()
    oracle.leaf_digests_mt([host], C, 1, alg)
    per_core = host.size / (time.perf_counter() - t0) / 1e9
    del host
    return {
        "value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": threads, "kind": "oracle",
        "single_thread_GBps": round(per_core, 4), **host_cpu_info(),
        "sample": f"first {nbytes} bytes ({n_leaves} whole chunks of {n_msgs} message(s)) of this workload, one "
                  f"message at a time; oracle chunk digests on {threads} threads + the Merkle root over them; "
                  f"device-to-host copies not timed",
        "seconds": round(dt, 3), "matches_gpu_digests": ok,
        # messages sampled whole: their roots (the oracle's recursive tree) against the GPU's
        "roots_compared": roots_checked, "matches_gpu_roots": roots_ok == roots_checked,
    }


def stream_bench(args, dev):
    """Host-resident weights: Algorithm 1's load / hash / free loop, then the same roots and verify."""
    import torch
    import workloads as W
    from paper_2510_23938_amd import hv

    limit = int(args.stream * (1 << 30))
    names, lens, total = [], [], 0
    for name, shape in W.tensors_70b():
        n = W.numel(shape) * 2
        if total + n > limit:
            break
        names.append(name)
        lens.append(n)
        total += n
    host = torch.empty(total, dtype=torch.uint8, pin_memory=True)
    offs = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    order = {n: i for i, (n, _) in enumerate(W.tensors_70b())}
    shapes = dict(W.tensors_70b())
    for name, o, n in zip(names, offs, lens):
        host[o:o + n].copy_(W.as_bytes(W.bf16_weights(shapes[name], W.tensor_seed(5, order[name]), dev)).cpu())
    msgs = [host[o:o + n] for o, n in zip(offs, lens)]
    C = W.CHUNK_BYTES[5]
    batch = args.batch_mib << 20
    log(f"stream: {len(msgs)} tensors, {total} bytes in pinned host memory, batch {batch} bytes")
    # plain host-to-device copy bandwidth of the same bytes (the PCIe roofline)
    dst = torch.empty(min(total, 4 << 30), dtype=torch.uint8, device=dev)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for lo in range(0, total, dst.numel()):
        hi = min(lo + dst.numel(), total)
        dst[: hi - lo].copy_(host[lo:hi], non_blocking=True)
    b.record()
    b.synchronize()
    h2d = total / (a.elapsed_time(b) / 1e3) / 1e9
    del dst
    ws = hv.Workspace(dev)
    copy_stream = torch.cuda.Stream(dev)

    def step():
        leaves, seg = hv.hv_hash_host_chunks(msgs, C, batch, dev, ws, copy_stream, alg=args.alg)
        roots = hv.hv_merkle_reduce(leaves, seg, alg=args.alg)
        return hv.hv_merkle_reduce(roots, np.array([0, len(msgs)], dtype=np.uint64), alg=args.alg)

    expected = bytes(step().cpu().numpy().reshape(-1))
    for _ in range(args.warmup):
        assert hv.hv_verify_root(step(), expected, alg=args.alg)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        assert hv.hv_verify_root(step(), expected, alg=args.alg)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / args.steps
    value = total / dt / 1e9
    log(f"stream: {dt * 1e3:.1f} ms/step, {value:.2f} GB/s; plain host-to-device copy {h2d:.2f} GB/s")
    print(json.dumps({
        "metric": "GB/s hashed+Merkle-verified from pinned host memory (streamed) on 1 MI355X",
        "value": round(value, 3), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(dt * 1e3, 3), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u32", "data": "synthetic",
        "config": {"workload": f"first {len(msgs)} tensors of the 70B-shaped bf16 weight set in pinned host memory",
                   "hash": args.alg,
                   "bytes": total, "chunk_bytes": C, "batch_bytes": batch},
        "roofline": {"bound": "pcie", "achieved": round(value, 3), "peak": round(h2d, 3), "unit": "GB/s",
                     "frac": round(value / h2d, 4), "traffic": None,
                     "peak_is": "measured pinned host-to-device copy of the same bytes"},
    }), flush=True)


def incremental_bench(args, dev):
    """Re-verification after K chunks change: rehash K chunks, update their branches, manifest, verify."""
    import torch
    import workloads as W
    from paper_2510_23938_amd import hv

    wl = W.workload(args.config, dev)
    C = wl.chunk_bytes
    msgs = wl.msgs
    leaves, seg = hv.hv_hash_chunks(msgs, C, dev, alg=args.alg)
    tree = hv.Tree(leaves, seg, alg=args.alg)
    n_seg = len(seg) - 1
    top_seg = np.array([0, n_seg], dtype=np.uint64)
    rng = np.random.default_rng(W.seed_of(args.config) + 7)
    n_leaves = int(seg[-1])
    k = min(args.incremental, n_leaves)
    pipe = hv.Pipeline(msgs, C, "manifest", dev, alg=args.alg)  # full re-verification, time and expected root
    rehash_ws, top_ws = hv.Workspace(dev), hv.Workspace(dev)
    inc_ms, full_ms = [], []
    for rep in range(args.warmup + args.steps):
        dirty = np.sort(rng.choice(n_leaves, size=k, replace=False)).astype(np.uint64)
        owners = np.searchsorted(seg, dirty, side="right") - 1
        for leaf, m in zip(dirty, owners):     # flip one byte inside each chosen chunk
            off = (int(leaf) - int(seg[m])) * C if C else 0
            v = msgs.views[m] if msgs.views is not None else None
            if v is not None:
                v[off] ^= 0x01
            else:
                o = int(msgs.offsets[m]) + off
                msgs.buffer[o] ^= 0x01
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        hv.hv_rehash_chunks(msgs, C, dirty, leaves, rehash_ws, alg=args.alg)
        roots = tree.update(leaves, dirty)
        top = hv.hv_merkle_reduce(roots, top_seg, top_ws, alg=args.alg)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        expected = bytes(pipe.compute().cpu().numpy().reshape(-1))
        t2 = time.perf_counter()
        assert hv.hv_verify_root(top, expected, alg=args.alg), "incremental root differs from the full recompute"
        if rep >= args.warmup:
            inc_ms.append((t1 - t0) * 1e3)
            full_ms.append((t2 - t1) * 1e3)
    inc, full = float(np.median(inc_ms)), float(np.median(full_ms))
    log(f"incremental: {k} changed chunks of {n_leaves}: {inc:.3f} ms vs full {full:.2f} ms ({full / inc:.1f}x)")
    print(json.dumps({
        "metric": "ms to re-verify after K changed chunks (rehash K + branch update + manifest), 1 MI355X",
        "value": round(inc, 4), "unit": "ms", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(inc, 4), "higher_is_better": False, "scaling": "weak", "vs_baseline": None,
        "dtype": "u32", "data": "synthetic",
        "config": {"workload": wl.description, "hash": args.alg, "changed_chunks": k, "leaves": n_leaves,
                   "chunk_bytes": C,
                   "full_reverify_ms": round(full, 3), "speedup": round(full / inc, 2),
                   "matches_full_recompute": True},
    }), flush=True)


def monitor_bench(args, dev):
    """Continuous runtime monitoring beside inference-shaped work on the same
    weights: the slowdown of that work against the monitor's verification
    rate, per slice length (the monitor's budget)."""
    import torch
    import torch.nn.functional as F
    import workloads as W
    from paper_2510_23938_amd import hv

    wl = W.workload(5, dev)
    C, alg = wl.chunk_bytes, args.alg
    pipe = hv.Pipeline(wl.msgs, C, "manifest", dev, alg=alg)
    expected = bytes(pipe.compute().cpu().numpy().reshape(-1))
    assert pipe.run(expected)  # the initial verification; its leaf digests are the monitor's references
    ref = pipe.leaves
    named = dict(zip(wl.msgs.names, wl.msgs.owners))
    proj = ("self_attn.q_proj", "self_attn.k_proj", "self_attn.v_proj", "self_attn.o_proj", "mlp.gate_proj",
            "mlp.up_proj", "mlp.down_proj")
    layers = [[named[f"model.layers.{l}.{p}.weight"] for p in proj] for l in range(80)]
    # two streams, made once and reused: streams beyond the device's hardware
    # queues share queues, and a monitor stream sharing the inference stream's
    # queue would run after it instead of beside it
    inf = torch.cuda.Stream(dev)
    mon_stream = torch.cuda.Stream(dev)

    def workload_of(tokens, mats):
        with torch.cuda.stream(inf):
            xs = {d: torch.randn(tokens, d, device=dev, dtype=torch.bfloat16) for d in {w.shape[1] for w in mats}}

        def step():
            for w in mats:
                F.linear(xs[w.shape[1]], w)
        return step, sum(w.numel() * 2 for w in mats), sum(2 * tokens * w.numel() for w in mats)

    kinds = {
        "decode": workload_of(args.decode_batch, [w for L in layers for w in L] + [named["lm_head.weight"]]),
        "prefill": workload_of(2048, [w for L in layers[:8] for w in L]),
    }

    def timed(step, n, stream=None):
        stream = stream or inf
        with torch.cuda.stream(stream):
            step()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(n):
                step()
            b.record(stream)
        b.synchronize()
        return a, b

    seg = pipe.seg
    lens = wl.msgs.lens.astype(np.int64)

    def leaf_bytes(first, count):
        # bytes of leaves [first, first + count): full chunks except each message's last
        m0 = int(np.searchsorted(seg, first, side="right")) - 1
        m1 = int(np.searchsorted(seg, first + count - 1, side="right")) - 1
        total = 0
        for m in range(m0, m1 + 1):
            lo, hi = max(first, int(seg[m])), min(first + count, int(seg[m + 1]))
            if hi <= lo:
                continue
            last = int(seg[m + 1]) - 1
            total += (hi - lo) * C
            if lo <= last < hi:
                total -= C - (int(lens[m]) - (last - int(seg[m])) * C)
        return total

    def run_monitor(slice_leaves, ring, stream=None):
        """Queue ring - 1 scans back to back; returns (monitor, t0 event, [(end event, bytes)]).
        ``stream``: a torch stream or a CuMaskedStream (whose close() then closes the monitor)."""
        mon = hv.Monitor(wl.msgs, C, ref, alg, slice_leaves, dev, stream=stream or mon_stream, ring=ring)
        t0 = torch.cuda.Event(enable_timing=True)
        t0.record(mon.stream)
        ends = []
        for _ in range(ring - 1):
            first, count = mon.step()
            e = torch.cuda.Event(enable_timing=True)
            e.record(mon.stream)
            ends.append((e, leaf_bytes(first, count)))
        return mon, t0, ends

    # each kind alone
    alone = {}
    for kind, (step, wbytes, flops) in kinds.items():
        a, b = timed(step, args.steps)
        alone[kind] = a.elapsed_time(b) / args.steps
        log(f"{kind} alone: {alone[kind]:.2f} ms/step ({wbytes / alone[kind] / 1e6:.0f} GB/s of weights, "
            f"{flops / alone[kind] / 1e9:.0f} TFLOP/s)")
    rows = []
    for S in args.monitor_slices:
        # the monitor alone at this slice length
        probe = max(8, min(400, int(2 ** 30 * 4 / (S * C)) + 8))
        mon, t0, ends = run_monitor(S, probe)
        ends[-1][0].synchronize()
        ms = t0.elapsed_time(ends[-1][0])
        solo = sum(nb for _, nb in ends) / (ms / 1e3) / 1e9
        mon.poll(wait=True)
        assert mon.mismatches == []
        row = {"slice_leaves": S, "slice_bytes": S * C, "monitor_alone_GBps": round(solo, 1)}
        for kind, (step, wbytes, flops) in kinds.items():
            window = args.steps * alone[kind] / 1e3
            n_scans = int(2.0 * window * solo * 1e9 / (S * C)) + 8
            mon, t0, ends = run_monitor(S, n_scans + 1)
            a, b = timed(step, args.steps)
            ends[-1][0].synchronize()
            ta, tb = t0.elapsed_time(a), t0.elapsed_time(b)
            inside = [nb for e, nb in ends if ta < t0.elapsed_time(e) <= tb]
            last_end = t0.elapsed_time(ends[-1][0])
            co = a.elapsed_time(b) / args.steps
            rate = sum(inside) / ((tb - ta) / 1e3) / 1e9
            mon.poll(wait=True)
            assert mon.mismatches == [], "the monitor reported a change in untouched weights"
            slow = (co / alone[kind] - 1) * 100
            sweep = pipe.total_bytes / (rate * 1e9) if rate > 0 else None
            row[kind] = {"alone_ms": round(alone[kind], 3), "with_monitor_ms": round(co, 3),
                         "slowdown_pct": round(slow, 2), "monitor_GBps": round(rate, 1),
                         "monitor_busy_whole_window": last_end > tb,
                         "sweep_s": round(sweep, 3) if sweep else None,
                         # one sweep per interval, at this slice length: the average cost over the interval
                         f"avg_slowdown_pct_at_{args.monitor_interval:g}s_interval":
                             round(slow * min(1.0, sweep / args.monitor_interval), 3) if sweep else None}
            log(f"slice {S}: {kind} {alone[kind]:.2f} -> {co:.2f} ms/step ({slow:+.1f}%), monitor {rate:.0f} GB/s "
                f"(alone {solo:.0f}), sweep {row[kind]['sweep_s']} s")
        rows.append(row)
    # spatial partitioning: the monitor on K CUs of its own, the inference work
    # on a stream masked to the other CUs; slowdowns against the unmasked run.
    # Each masked stream holds a hardware queue of its own and a process gets
    # few, so one K per run.
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count

    def partitioned(K, inf_p, mon_p):
        mon_cus = list(range(K))
        rest = [c for c in range(n_cu) if c not in set(mon_cus)]
        S = len(mon_cus) * 4 * 64 * 2  # two waves per SIMD of the monitor's CUs
        probe = 24
        mon, t0, ends = run_monitor(S, probe, mon_p)
        ends[-1][0].synchronize()
        solo = sum(nb for _, nb in ends) / (t0.elapsed_time(ends[-1][0]) / 1e3) / 1e9
        mon.poll(wait=True)
        assert mon.mismatches == []
        part = {"monitor_cus": len(mon_cus), "slice_leaves": S, "monitor_alone_GBps": round(solo, 1)}
        for kind, (step, wbytes, flops) in kinds.items():
            a, b = timed(step, args.steps, inf_p.stream)
            rest_ms = a.elapsed_time(b) / args.steps
            window = args.steps * rest_ms / 1e3
            n_scans = int(2.0 * window * solo * 1e9 / (S * C)) + 8
            mon, t0, ends = run_monitor(S, n_scans + 1, mon_p)
            a, b = timed(step, args.steps, inf_p.stream)
            ends[-1][0].synchronize()
            ta, tb = t0.elapsed_time(a), t0.elapsed_time(b)
            inside = [nb for e, nb in ends if ta < t0.elapsed_time(e) <= tb]
            co = a.elapsed_time(b) / args.steps
            rate = sum(inside) / ((tb - ta) / 1e3) / 1e9
            mon.poll(wait=True)
            assert mon.mismatches == []
            slow = (co / alone[kind] - 1) * 100
            sweep = pipe.total_bytes / (rate * 1e9) if rate > 0 else None
            part[kind] = {"alone_ms": round(alone[kind], 3), "on_other_cus_alone_ms": round(rest_ms, 3),
                          "with_monitor_ms": round(co, 3), "slowdown_pct": round(slow, 2),
                          "monitor_GBps": round(rate, 1),
                          "monitor_busy_whole_window": t0.elapsed_time(ends[-1][0]) > tb,
                          "sweep_s": round(sweep, 3) if sweep else None,
                          f"avg_slowdown_pct_at_{args.monitor_interval:g}s_interval":
                              round(slow * min(1.0, sweep / args.monitor_interval), 3) if sweep else None}
            log(f"{len(mon_cus)} monitor CUs: {kind} {alone[kind]:.2f} -> {rest_ms:.2f} on {len(rest)} CUs alone -> "
                f"{co:.2f} ms/step with the monitor ({slow:+.1f}%), monitor {rate:.0f} GB/s (alone {solo:.0f})")
        return part

    parts = []
    for K in [args.monitor_partition] if args.monitor_partition else []:
        # low CU numbers, which the runtime spreads over the XCDs
        inf_p, mon_p = hv.CuMaskedStream(range(K, n_cu), dev), hv.CuMaskedStream(range(K), dev)
        parts.append(partitioned(K, inf_p, mon_p))
        # the events and monitors made on the masked streams died with partitioned()'s
        # frame; the streams are destroyed now, before the process's exit handlers run
        gc.collect()
        inf_p.close()
        mon_p.close()
    # a changed byte is found, at its leaf, by one sweep
    rng = np.random.default_rng(W.seed_of(5) + 11)
    m = int(rng.integers(0, len(wl.msgs)))
    off = int(rng.integers(0, int(lens[m])))
    view = wl.msgs.views[m]
    old = int(view[off].item())
    view[off] = old ^ 0x80
    torch.cuda.synchronize()
    mon = hv.Monitor(wl.msgs, C, ref, alg, 16384, dev, stream=mon_stream, ring=256)
    mon.sweep()
    mon.poll(wait=True)
    view[off] = old
    torch.cuda.synchronize()
    detected = [(fb, cnt) for fb, cnt, _, _ in mon.mismatches] == [(int(seg[m]) + off // C, 1)]
    pick = min(rows, key=lambda r: abs(r["slice_leaves"] - args.monitor_slice))
    line = {
        "metric": "decode slowdown (%) with continuous monitoring of the resident weights beside it, 1 MI355X",
        "value": pick["decode"]["slowdown_pct"], "unit": "%", "n_gpus": 1, "steps": args.steps, "warmup": 1,
        "ms_per_step": pick["decode"]["with_monitor_ms"], "higher_is_better": False, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {"workload": "70B-shaped bf16 weight set (723 tensors, 64 KiB chunks) monitored while "
                               f"decode-shaped (batch {args.decode_batch}, all 560 projections + lm_head) or "
                               "prefill-shaped (2048 tokens, 8 layers) bf16 GEMMs run on the same weights",
                   "hash": alg, "monitor_slice_leaves": pick["slice_leaves"], "monitor_duty": "100% (back to back)",
                   "changed_byte_detected_at_its_leaf": detected, "slices": rows, "partitioned": parts},
    }
    print(json.dumps(line), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=5)
    ap.add_argument("--alg", choices=sorted(ALGS), default="sha256", help="hash of chunks and tree nodes")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-mib", type=int, default=48 << 10,
                    help="bytes of the workload the oracle hashes for cpu_baseline (about 10 s on 16 threads)")
    ap.add_argument("--no-peaks", action="store_true", help="skip the VALU / HBM peak microbenchmarks")
    ap.add_argument("--stream", type=float, default=0.0, metavar="GIB",
                    help="instead: stream this many GiB of the 70B-shaped tensors from pinned host memory "
                         "(host-to-device copy + hash + roots + verify per step)")
    ap.add_argument("--batch-mib", type=int, default=1024, help="staging batch for --stream")
    ap.add_argument("--incremental", type=int, default=0, metavar="K",
                    help="instead: change K random chunks of the workload and time re-verification that rehashes "
                         "only them and updates only their tree branches, against a full re-verification")
    ap.add_argument("--monitor", action="store_true",
                    help="instead: continuous monitoring of the 70B-shaped set beside decode- and prefill-shaped "
                         "GEMMs on the same weights; slowdown vs monitor rate per slice length")
    ap.add_argument("--monitor-slices", type=int, nargs="+", default=[1024, 4096, 16384, 65536])
    ap.add_argument("--monitor-slice", type=int, default=4096, help="slice length of the reported value")
    ap.add_argument("--decode-batch", type=int, default=8)
    ap.add_argument("--monitor-partition", type=int, default=8,
                    help="monitor CU count for the partitioned run (CU-masked streams; 0: none)")
    ap.add_argument("--monitor-interval", type=float, default=30.0,
                    help="seconds between sweeps for the averaged cost (the paper's runtime-monitoring example)")
    ap.add_argument("--leaf-kernel", choices=["auto", "one-wave", "two-wave", "two-wave-compact"], default="auto",
                    help="SHA-256 leaf kernel (auto: the two-wave kernel for at most 128 leaves per CU)")
    ap.add_argument("--graph", action="store_true",
                    help="time HIP-graph replays of the prepared pass (kernel timing from the eager passes)")
    ap.add_argument("--op-rates", action="store_true",
                    help="instead: issue rate of each VALU instruction of the SHA mixes (per-op microbenchmark)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run one 4 GiB device copy first (reference point for HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "the multi-GPU design is described, not run", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1 or args.warmup < 0 or args.config not in (1, 2, 3, 4, 5):
        ap.error("--steps must be at least 1, --warmup at least 0 and --config one of 1-5")

    import torch
    import workloads as W
    from paper_2510_23938_amd import hv

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    hv.set_leaf_kernel(args.leaf_kernel)
    if args.stream > 0:
        stream_bench(args, dev)
        return
    if args.incremental > 0:
        incremental_bench(args, dev)
        return
    if args.monitor:
        monitor_bench(args, dev)
        return
    if args.op_rates:
        rates = hv.measure_op_rates(dev)
        lane_cycles = VALU_PEAK_TOPS  # T lane-cycles/s at 2.4 GHz
        for name, r in rates.items():
            log(f"{name:16s} {r:7.2f} T lane-ops/s = {r / lane_cycles:.2f} per lane per cycle at 2.4 GHz")
        print(json.dumps({"metric": "VALU issue rate per instruction (8 independent chains, full occupancy), 1 MI355X",
                          "unit": "T lane-ops/s", "rates": {k: round(v, 2) for k, v in rates.items()},
                          "per_lane_cycle_at_2.4GHz": {k: round(v / lane_cycles, 3) for k, v in rates.items()}}),
              flush=True)
        return
    if args.copy_calibration:
        a = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
    t0 = time.perf_counter()
    wl = W.workload(args.config, dev)
    torch.cuda.synchronize()
    log(f"workload {args.config}: {wl.description}; generated in {time.perf_counter() - t0:.1f} s")
    mode = "manifest" if wl.manifest else "single"
    alg = args.alg
    block_bytes, _, ops_per_block, leaf_kernel, _, _ = ALGS[alg]
    pipe = hv.Pipeline(wl.msgs, wl.chunk_bytes, mode, dev, alg=alg)

    # the first pass fixes the expected root the timed steps verify against
    root = pipe.compute()
    expected = bytes(root.cpu().numpy().reshape(-1))

    # The timed step: the one-shot calls (hv_hash_chunks, hv_merkle_reduce for the
    # per-tensor roots and again for the manifest, hv_verify_root).  Every step
    # uploads the message descriptors, schedules the leaves, hashes them, reduces
    # both tree levels and compares the root on the GPU: every row of the path.
    ver = hv.Verifier(dev, alg)
    one_root = ver.manifest_root if wl.manifest else ver.single_tree_root

    def oneshot_step():
        return ver.verify_root(one_root(wl.msgs, wl.chunk_bytes), expected)

    for _ in range(args.warmup):
        assert oneshot_step()
    hv.set_kernel_timing(True)
    kernel_ms, step_ms = [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        ts = time.perf_counter()
        ok = oneshot_step()  # synchronous: it ends with the verdict on the host
        step_ms.append((time.perf_counter() - ts) * 1e3)
        kernel_ms.append(hv.leaf_kernel_ms())
        assert ok
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    hv.set_kernel_timing(False)
    del ver
    # The same pass prepared once (hv_plan.h): descriptors uploaded and leaves
    # scheduled when the plan is made, so a pass only queues the hash, tree and
    # compare kernels.  Reported beside the step, not as it.
    for _ in range(args.warmup):
        assert pipe.run(expected)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        assert pipe.run(expected)
    torch.cuda.synchronize()
    prepared_ms = (time.perf_counter() - t0) / args.steps * 1e3
    graph_ms = None
    if args.graph:
        # the prepared pass captured once in a HIP graph, then replayed
        pipe.capture(expected)
        for _ in range(args.warmup):
            assert pipe.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            assert pipe.replay()
        torch.cuda.synchronize()
        graph_ms = (time.perf_counter() - t0) / args.steps * 1e3
        log(f"graph replay of the prepared pass: {graph_ms:.2f} ms/step (eager {prepared_ms:.2f})")
    # a flipped expected byte must fail, a matching one pass
    bad = bytearray(expected)
    bad[int(np.random.default_rng(W.seed_of(args.config) + 1).integers(0, len(bad)))] ^= 0x01
    negative_ok = not pipe.run(bytes(bad))

    ms_step = dt / args.steps * 1e3
    total = pipe.total_bytes
    value = total / (ms_step / 1e3) / 1e9
    k_ms = float(np.mean(kernel_ms))
    med = float(np.median(step_ms))
    step_stats = {"median": round(med, 3), "min": round(min(step_ms), 3), "max": round(max(step_ms), 3),
                  "spread_pct": round((max(step_ms) - min(step_ms)) / med * 100, 2),
                  "median_GBps": round(total / (med / 1e3) / 1e9, 2),
                  "leaf_kernel_median_ms": round(float(np.median(kernel_ms)), 3)}
    blocks = sha_blocks(wl.msgs.lens, wl.chunk_bytes, alg)
    achieved = blocks * ops_per_block / (k_ms / 1e3) / 1e12
    ran = hv.leaf_kernel_for(pipe.n_leaves)  # the leaf kernel the timed passes ran
    if ran != "one-wave":
        leaf_kernel = f"{alg}_split_kernel"
    log(f"{args.steps} steps: {ms_step:.2f} ms/step, {value:.1f} GB/s (median step {med:.2f} ms, spread "
        f"{step_stats['spread_pct']:.2f}%); leaf kernel {k_ms:.2f} ms avg ({total / k_ms / 1e6:.1f} GB/s, "
        f"{achieved:.2f} TOP/s); prepared pass {prepared_ms:.2f} ms/step")

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u32", "data": "synthetic",
        "config": {
            "workload": wl.description, "config_index": args.config, "bytes": total, "messages": len(wl.msgs),
            "leaves": pipe.n_leaves, "chunk_bytes": wl.chunk_bytes, "hash": alg, f"{alg}_blocks": blocks,
            "verified": True, "mismatch_detected": negative_ok,
            "step": "one-shot calls: descriptor upload, leaf scheduling, leaf hashes, per-tensor roots, manifest, "
                    "root compare" if wl.manifest else
                    "one-shot calls: descriptor upload, leaf scheduling, leaf hashes, one tree, root compare",
            "step_ms": step_stats,
            "leaf_kernel": args.leaf_kernel, "leaf_kernel_ran": ran,
            "prepared_ms_per_step": round(prepared_ms, 3),
            "prepared_GBps": round(pipe.total_bytes / (prepared_ms / 1e3) / 1e9, 2),
            **({"graph_ms_per_step": round(graph_ms, 3)} if graph_ms is not None else {}),
        },
        "roofline": {
            "kernel": leaf_kernel, "bound": "alu", "achieved": round(achieved, 3), "peak": round(VALU_PEAK_TOPS, 3),
            "unit": "TOP/s", "frac": round(achieved / VALU_PEAK_TOPS, 4),
            "traffic": traffic_for_current_kernel(alg, args.config) if ran == "one-wave" else None,
            "kernel_ms": round(k_ms, 3), "ops_per_block": ops_per_block,
            "hashed_GBps": round(total / k_ms / 1e6, 2),
            "roof_GBps": round(VALU_PEAK_TOPS * 1e12 / ops_per_block * block_bytes / 1e9, 1),
            "dual_issue_bound_GBps": round(1024 * 64 * 2.4e9 / DUAL_ISSUE_CYCLES[alg] * block_bytes / 1e9, 1),
            "frac_of_dual_issue_bound": round(total / k_ms / 1e6 / (1024 * 64 * 2.4e9 / DUAL_ISSUE_CYCLES[alg]
                                                                    * block_bytes / 1e9), 4),
        },
    }
    if not args.no_peaks:
        valu = hv.measure_valu_peak(dev, mix=alg)
        sha = hv.measure_sha256_ceiling(dev, alg=alg)
        hbm = hv.measure_hbm_read(16 << 30, dev)
        kernel_blocks_per_s = blocks / (k_ms / 1e3)
        log(f"measured peaks: {alg} VALU mix {valu['tops']:.2f} TOP/s, register-only {alg} "
            f"{sha['GBps_equiv']:.0f} GB/s-equiv, HBM read {hbm['GBps']:.0f} GB/s")
        line["roofline"]["measured_valu_peak"] = round(valu["tops"], 3)
        line["roofline"]["frac_of_measured_valu_peak"] = round(achieved / valu["tops"], 4)
        line["roofline"][f"register_{alg}_GBps"] = round(sha["GBps_equiv"], 1)
        line["roofline"][f"frac_of_register_{alg}"] = round(kernel_blocks_per_s / sha["blocks_per_s"], 4)
        line["roofline"]["measured_hbm_read_GBps"] = round(hbm["GBps"], 1)
    if not args.no_cpu_baseline:
        log("cpu baseline ...")
        line["cpu_baseline"] = cpu_baseline(wl, pipe, args.cpu_sample_mib << 20, alg)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
