"""Seeded random cases through the streaming, incremental, prepared and
monitoring paths, each against the resident one-shot path and the CPU oracle.

Every case draws its own message set (lengths clustered around block and
chunk boundaries, empty messages, 16-byte-aligned or not), chunk size and
hash; then
* streaming: a random batch size (a multiple of 256, at least one chunk),
  pinned or pageable sources -- digests equal the resident ones and the oracle;
* incremental: three rounds of random changed chunks (one byte flipped in
  each), rehash and branch update -- roots equal a full recompute;
* prepared pass: one tree and manifest forms -- the root equals the one-shot
  calls and the oracle, a flipped expected byte fails;
* monitoring: references from the clean set, random flipped chunks, a sweep
  in random slice lengths -- every scan reports exactly the flipped leaves of
  its range (count and lowest leaf).
Expected values come only from ``oracle`` or from the resident path, which
the parity tests pin to the oracle.
"""
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
CASES = 8


def threads():
    return max(1, min(16, len(os.sched_getaffinity(0))))


def draw(rng, alg, n_max=60, allow_whole=True):
    B = 64 if alg == "sha256" else 128
    C = int(rng.choice(([0] if allow_whole else []) + [B, 3 * B, 4096, 65536]))
    n = int(rng.integers(1, n_max))
    unit = C if C else 4096
    kind = rng.integers(0, 4, n)
    lens = np.where(kind == 0, rng.integers(0, 3 * B, n),
            np.where(kind == 1, rng.integers(1, 6, n) * unit + rng.integers(-3, 4, n),
            np.where(kind == 2, rng.integers(0, 300_000, n), 0)))
    return np.maximum(lens, 0).astype(np.uint64), C


def device_set(rng, lens, seed):
    """(buffer, host copy, ptrs, starts) of the messages in one device buffer, half off 16-byte alignment."""
    offs = rng.integers(0, 16, len(lens)) * (rng.random(len(lens)) < 0.5)
    starts = np.zeros(len(lens), dtype=np.uint64)
    pos = 0
    for i, L in enumerate(lens):
        starts[i] = pos + int(offs[i])
        pos += (int(L) + int(offs[i]) + 16 + 15) // 16 * 16
    buf = W.random_bytes(max(pos, 1), seed, DEV)
    ptrs = np.uint64(buf.data_ptr()) + starts
    ptrs[lens == 0] = 0
    return buf, buf.cpu().numpy(), ptrs, starts


def host_msgs(host, starts, lens):
    return [host[int(s):int(s) + int(L)] for s, L in zip(starts, lens)]


@pytest.mark.parametrize("case", range(CASES))
def test_streaming(case):
    rng = np.random.default_rng(7100 + case)
    alg = ("sha256", "sha384")[case % 2]
    lens, C = draw(rng, alg)
    D = 32 if alg == "sha256" else 48
    # at least one chunk: with C = 0 a chunk is a whole message
    unit = C if C else max(int(lens.max()) if len(lens) else 0, 256)
    batch = int(unit * int(rng.integers(1, 6)) + 256 * int(rng.integers(0, 3)))
    batch = -(-batch // 256) * 256
    pinned = bool(case % 3)
    msgs = []
    for i, L in enumerate(lens):
        d = W.random_bytes(int(L), 7200 + 50 * case + i, DEV).cpu()
        if pinned:
            p = torch.empty(int(L), dtype=torch.uint8, pin_memory=True)
            p.copy_(d)
            d = p
        msgs.append(d)
    tag = f"case {case}: {alg}, C={C}, batch={batch}, pinned={pinned}, {len(lens)} messages"
    got, seg = hv.hv_hash_host_chunks(msgs, C, batch, alg=alg)
    resident, seg2 = hv.hv_hash_chunks([m.to(DEV) for m in msgs], C, alg=alg)
    torch.cuda.synchronize()
    assert np.array_equal(seg, seg2), tag
    assert got.shape[1] == D and torch.equal(got, resident), tag
    want = oracle.leaf_digests_mt([m.numpy() for m in msgs], C, threads(), alg)
    assert np.array_equal(got.cpu().numpy(), want), tag


@pytest.mark.parametrize("case", range(CASES))
def test_incremental(case):
    rng = np.random.default_rng(7300 + case)
    alg = ("sha256", "sha384")[case % 2]
    lens, C = draw(rng, alg)
    buf, host, ptrs, starts = device_set(rng, lens, 7400 + case)
    msgs = (ptrs, lens)
    leaves, seg = hv.hv_hash_chunks(msgs, C, alg=alg)
    tree = hv.Tree(leaves, seg, alg=alg)
    n_leaves = int(seg[-1])
    for rnd in range(3):
        if n_leaves == 0:
            break
        k = int(rng.integers(1, min(n_leaves, 40) + 1))
        dirty = np.sort(rng.choice(n_leaves, size=k, replace=False)).astype(np.uint64)
        for leaf in dirty:  # flip one byte inside each chosen chunk
            m = int(np.searchsorted(seg, leaf, side="right") - 1)
            if int(lens[m]) == 0:
                continue
            off = (int(leaf) - int(seg[m])) * C if C else 0
            span = min(C, int(lens[m]) - off) if C else int(lens[m])
            at = int(starts[m]) + off + int(rng.integers(0, span))
            buf[at] ^= 0xFF
        hv.hv_rehash_chunks(msgs, C, dirty, leaves, alg=alg)
        roots = tree.update(leaves, dirty)
        full_leaves, _ = hv.hv_hash_chunks(msgs, C, alg=alg)
        full_roots = hv.hv_merkle_reduce(full_leaves, seg, alg=alg)
        torch.cuda.synchronize()
        tag = f"case {case} round {rnd}: {alg}, C={C}, {k} changed chunks of {n_leaves}"
        assert torch.equal(leaves, full_leaves), tag
        assert torch.equal(roots, full_roots), tag
    host = buf.cpu().numpy()
    want = oracle.seg_roots_from_leaves(oracle.leaf_digests_mt(host_msgs(host, starts, lens), C, threads(), alg),
                                        np.diff(seg), alg)
    assert [bytes(r) for r in tree.roots.cpu().numpy()] == want, f"case {case}: final roots differ from the oracle"


@pytest.mark.parametrize("case", range(CASES))
def test_prepared_pass(case):
    rng = np.random.default_rng(7500 + case)
    alg = ("sha256", "sha384")[case % 2]
    lens, C = draw(rng, alg)
    buf, host, ptrs, starts = device_set(rng, lens, 7600 + case)
    mode = ("manifest", "single")[(case // 2) % 2]
    pipe = hv.Pipeline((ptrs, lens), C, mode, DEV, alg=alg)
    root = bytes(pipe.compute().cpu().numpy().reshape(-1))
    v = hv.Verifier(DEV, alg)
    one = v.manifest_root((ptrs, lens), C) if mode == "manifest" else v.single_tree_root((ptrs, lens), C)
    want_leaves = oracle.leaf_digests_mt(host_msgs(host, starts, lens), C, threads(), alg)
    if mode == "manifest":
        want = oracle.mth(oracle.seg_roots_from_leaves(want_leaves, np.diff(pipe.seg), alg), alg)
    else:
        want = oracle.mth(want_leaves, alg)
    tag = f"case {case}: {alg}, {mode}, C={C}, {len(lens)} messages"
    assert root == bytes(one.cpu().numpy().reshape(-1)) == want, tag
    assert pipe.run(want), tag
    bad = bytearray(want)
    bad[int(rng.integers(0, len(bad)))] ^= 1 << int(rng.integers(0, 8))
    assert not pipe.run(bytes(bad)), tag


@pytest.mark.parametrize("case", range(CASES))
def test_monitor_sweep(case):
    rng = np.random.default_rng(7700 + case)
    alg = ("sha256", "sha384")[case % 2]
    lens, C = draw(rng, alg, allow_whole=False)
    buf, host, ptrs, starts = device_set(rng, lens, 7800 + case)
    msgs = (ptrs, lens)
    ref, seg = hv.hv_hash_chunks(msgs, C, alg=alg)
    n_leaves = int(seg[-1])
    if n_leaves == 0:
        pytest.skip("no leaves drawn")
    flipped = np.sort(rng.choice(n_leaves, size=int(rng.integers(0, min(n_leaves, 12) + 1)), replace=False))
    really = []
    for leaf in flipped:
        m = int(np.searchsorted(seg, leaf, side="right") - 1)
        off = (int(leaf) - int(seg[m])) * C
        span = min(C, int(lens[m]) - off)
        if span <= 0:
            continue
        buf[int(starts[m]) + off + int(rng.integers(0, span))] ^= 0x5A
        really.append(int(leaf))
    torch.cuda.synchronize()
    slice_leaves = int(rng.choice([1, 3, 64, 65, 1000, n_leaves]))
    slice_leaves = max(slice_leaves, -(-n_leaves // 400))  # at most about 400 scans
    mon = hv.Monitor(msgs, C, ref, alg=alg, slice_leaves=slice_leaves, device=DEV)
    mon.sweep()
    mon.poll(wait=True)
    got = sorted(mon.mismatches, key=lambda r: r[2])
    want = []
    for first in range(0, n_leaves, slice_leaves):
        hit = [x for x in really if first <= x < first + slice_leaves]
        if hit:
            want.append((min(hit), len(hit), first, min(slice_leaves, n_leaves - first)))
    assert got == want, f"case {case}: {alg}, C={C}, slice {slice_leaves}, flipped {really}"
