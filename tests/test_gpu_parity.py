"""GPU path vs the CPU oracle, bit for bit, at sizes the oracle finishes in seconds.

Every call goes through the C ABI (libhv.so) via the ctypes binding.  Inputs
come from the seeded generators in ``workloads``; expected values come only
from ``oracle``.
"""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")


def place(lens, align_off, seed, gap=16):
    """One device buffer holding the messages at 16-byte slots + align_off.

    Returns (buf, host bytes, ptrs, lens, starts)."""
    lens = np.asarray(lens, dtype=np.uint64)
    starts = np.zeros(len(lens), dtype=np.uint64)
    pos = 0
    for i, n in enumerate(lens):
        starts[i] = pos + align_off
        pos += (int(n) + align_off + gap + 15) // 16 * 16
    buf = W.random_bytes(max(pos, 1), seed, DEV)
    host = buf.cpu().numpy()
    ptrs = np.uint64(buf.data_ptr()) + starts
    ptrs[lens == 0] = 0  # empty messages may carry a NULL pointer
    return buf, host, ptrs, lens, starts


def host_msgs(host, starts, lens):
    return [host[int(s):int(s) + int(n)] for s, n in zip(starts, lens)]


def check_all(buf, host, ptrs, lens, starts, C, tag=""):
    v = hv.Verifier(DEV)
    leaves, seg = v.leaf_digests((ptrs, lens), C)
    roots = hv.hv_merkle_reduce(leaves, seg, v.ws_tree)
    manifest = hv.hv_merkle_reduce(roots, np.array([0, len(lens)], dtype=np.uint64), v.ws_manifest)
    torch.cuda.synchronize()
    msgs = host_msgs(host, starts, lens)
    want_leaves = oracle.leaf_digests_mt(msgs, C, 8)
    got_leaves = leaves.cpu().numpy()
    if not np.array_equal(got_leaves, want_leaves):
        bad = np.nonzero((got_leaves != want_leaves).any(axis=1))[0]
        owner = np.searchsorted(seg, bad[0], side="right") - 1
        raise AssertionError(f"{tag}: {len(bad)} leaf digests differ; first leaf {bad[0]} "
                             f"(message {owner}, length {int(lens[owner])}, C={C})")
    counts = np.diff(seg)
    want_roots = oracle.seg_roots_from_leaves(want_leaves, counts)
    got_roots = [bytes(r) for r in roots.cpu().numpy()]
    assert got_roots == want_roots, f"{tag}: segment roots differ"
    assert bytes(manifest.cpu().numpy().reshape(-1)) == oracle.mth(want_roots), f"{tag}: manifest differs"
    return want_roots


@pytest.mark.parametrize("align_off", [0, 1, 3, 15])
@pytest.mark.parametrize("C", [64, 128, 4096, 0])
def test_every_length_up_to_4160(C, align_off):
    lens = np.arange(0, 4161)
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=100 + align_off)
    check_all(buf, host, ptrs, lens, starts, C, f"C={C} off={align_off}")


@pytest.mark.parametrize("C", [64, 4096, 65536, 1 << 20, 0])
def test_mixed_batch(C):
    rng = np.random.default_rng(7)
    lens = np.concatenate([
        rng.integers(0, 300, 200), rng.integers(1, 70000, 200), [0, 0, 1, 64, 65536, 65537, 3 * (1 << 20) + 11],
        rng.integers(1 << 20, 3 << 20, 4),
    ])
    rng.shuffle(lens)
    buf, host, ptrs, lens, starts = place(lens, 0, seed=8)
    check_all(buf, host, ptrs, lens, starts, C, f"mixed C={C}")


def test_bf16_tensors_as_messages():
    named = [(f"t{i}", W.bf16_weights(s, 50 + i, DEV)) for i, s in enumerate([(3, 7), (1000, 33), (2048,), (64, 1024)])]
    C = 4096
    v = hv.Verifier(DEV)
    roots, leaves, seg = v.roots([t for _, t in named], C)
    torch.cuda.synchronize()
    host = [W.as_bytes(t).cpu().numpy().tobytes() for _, t in named]
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.seg_root(m, C) for m in host]
    assert hv.manifest_root(dict(named), C) == oracle.manifest_root([host[i] for i in (0, 1, 2, 3)], C)


def test_empty_cases():
    v = hv.Verifier(DEV)
    # no messages at all
    leaves, seg = v.leaf_digests((np.zeros(0, np.uint64), np.zeros(0, np.uint64)), 64)
    assert leaves.shape == (0, 32) and list(seg) == [0]
    # empty messages: no leaves with C > 0, one leaf each with C = 0
    ptrs, lens = np.zeros(3, np.uint64), np.zeros(3, np.uint64)
    leaves, seg = v.leaf_digests((ptrs, lens), 64)
    assert leaves.shape == (0, 32)
    roots = hv.hv_merkle_reduce(leaves, seg, v.ws_tree)
    assert [bytes(r) for r in roots.cpu().numpy()] == [oracle.mth([])] * 3
    leaves, seg = v.leaf_digests((ptrs, lens), 0)
    assert [bytes(r) for r in leaves.cpu().numpy()] == [oracle.sha256(b"")] * 3


@pytest.mark.parametrize("sizes", [
    [0], [1], [2], [3], [5], [511, 512, 513], [0, 1, 0, 2, 0], [1023, 1024, 1025, 4097],
    [300_000], [262_145, 3, 0, 70_000],
])
def test_merkle_segments(sizes):
    n = int(sum(sizes))
    entries = W.random_bytes(max(n, 1) * 32, 200 + n, DEV)[: n * 32].view(n, 32)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    roots = hv.hv_merkle_reduce(entries, seg)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[s]):int(seg[s + 1])]) for s in range(len(sizes))]
    assert [bytes(r) for r in roots.cpu().numpy()] == want


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_merkle_every_segment_size_up_to_600(alg):
    # every node count a tile can start from, around the 64-node point where the
    # kernel moves from LDS levels to wavefront shuffles, and second tiles with
    # ragged tails; one call over 601 segments of 0..600 entries
    D = 32 if alg == "sha256" else 48
    sizes = list(range(601))
    n = sum(sizes)
    entries = W.random_bytes(n * D, 250 + D, DEV).view(n, D)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    roots = hv.hv_merkle_reduce(entries, seg, alg=alg)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[k]):int(seg[k + 1])], alg) for k in range(len(sizes))]
    got = [bytes(r) for r in roots.cpu().numpy()]
    bad = [k for k in range(len(sizes)) if got[k] != want[k]]
    assert not bad, f"{alg}: roots differ for segment sizes {bad[:10]}"


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
@pytest.mark.parametrize("big_first", [False, True])
def test_merkle_group_launch_every_segment_size(alg, big_first):
    # 2^18 entries or more start with a group launch (8 entries per lane,
    # three levels in registers): every segment size 0..600 (every short last
    # group, empty segments) in one call made large by a segment of 100,003
    # entries, placed last or first; each root against the oracle and against
    # the same segments reduced by the tile launches alone (a call under 2^18)
    D = 32 if alg == "sha256" else 48
    small = list(range(601))
    sizes = [100_003] + small if big_first else small + [100_003]
    n = sum(sizes)
    assert n >= 1 << 18 and sum(small) < 1 << 18
    entries = W.random_bytes(n * D, 260 + D + big_first, DEV).view(n, D)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    roots = hv.hv_merkle_reduce(entries, seg, alg=alg)
    lo = 1 if big_first else 0
    part = entries[int(seg[lo]):int(seg[lo + len(small)])]
    part_roots = hv.hv_merkle_reduce(part.contiguous(), np.concatenate([[0], np.cumsum(small)]).astype(np.uint64),
                                     alg=alg)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[k]):int(seg[k + 1])], alg) for k in range(len(sizes))]
    got = [bytes(r) for r in roots.cpu().numpy()]
    bad = [sizes[k] for k in range(len(sizes)) if got[k] != want[k]]
    assert not bad, f"{alg}: roots differ for segment sizes {bad[:10]}"
    assert [bytes(r) for r in part_roots.cpu().numpy()] == want[lo:lo + len(small)]


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_merkle_two_group_launches_every_segment_size(alg):
    # a level of 2^18 nodes or more also runs as a group launch: here the
    # level-3 nodes (about 285,000) too, so the second group launch meets every
    # short last group of the segments of sizes 0..600 reduced once already
    D = 32 if alg == "sha256" else 48
    sizes = list(range(601)) + [2_100_007]
    n = sum(sizes)
    groups = sum(max(1, -(-c // 8)) for c in sizes)
    assert groups >= 1 << 18
    entries = W.random_bytes(n * D, 280 + D, DEV).view(n, D)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    roots = hv.hv_merkle_reduce(entries, seg, alg=alg)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[k]):int(seg[k + 1])], alg) for k in range(len(sizes))]
    got = [bytes(r) for r in roots.cpu().numpy()]
    bad = [sizes[k] for k in range(len(sizes)) if got[k] != want[k]]
    assert not bad, f"{alg}: roots differ for segment sizes {bad[:10]}"


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_merkle_four_lane_groups_every_segment_size(alg):
    # A group launch gives its last groups four lanes each once the rest fill
    # whole rounds of one wave per SIMD (256 groups per compute unit).  A first
    # segment of exactly 64 such rounds' entries makes the one-lane part of
    # both group launches end where the segments of sizes 0..600 begin, so the
    # four-lane form meets every short group, in leaf mode (launch 1) and on
    # level-3 nodes (launch 2); every root against the oracle.
    D = 32 if alg == "sha256" else 48
    cus = torch.cuda.get_device_properties(DEV).multi_processor_count
    rnd = 256 * cus
    small = list(range(601))
    sizes = [64 * rnd] + small
    n = sum(sizes)
    seg = np.concatenate([[0], np.cumsum(sizes)]).astype(np.uint64)
    plan = hv.merkle_launches(seg, alg)
    groups1 = sum(max(1, -(-c // 8)) for c in sizes)
    groups2 = sum(max(1, -(-max(1, -(-c // 8)) // 8)) for c in sizes)
    assert plan[0] == ("group", groups1, 8 * rnd), plan
    assert plan[1] == ("group", groups2, rnd), plan
    entries = W.random_bytes(n * D, 290 + D, DEV).view(n, D)
    roots = hv.hv_merkle_reduce(entries, seg, alg=alg)
    torch.cuda.synchronize()
    host = entries.cpu().numpy()
    want = [oracle.mth(host[int(seg[k]):int(seg[k + 1])], alg) for k in range(len(sizes))]
    got = [bytes(r) for r in roots.cpu().numpy()]
    bad = [sizes[k] for k in range(len(sizes)) if got[k] != want[k]]
    assert not bad, f"{alg}: roots differ for segment sizes {bad[:10]}"


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_merkle_single_trees_of_500_to_1100_entries(alg):
    # one segment around the 512-node tile: one launch up to 512 entries, a
    # second over the first launch's two or three tile nodes after it
    D = 32 if alg == "sha256" else 48
    entries = W.random_bytes(1100 * D, 295 + D, DEV).view(1100, D)
    host = entries.cpu().numpy()
    ws = hv.Workspace(DEV)
    bad = []
    for n in range(500, 1101):
        seg = np.array([0, n], dtype=np.uint64)
        kinds = [p[0] for p in hv.merkle_launches(seg, alg)]
        assert kinds == (["tile"] if n <= 512 else ["tile", "tile"]), (n, kinds)
        root = hv.hv_merkle_reduce(entries[:n], seg, ws, alg=alg)
        if bytes(root.cpu().numpy().reshape(-1)) != oracle.mth(host[:n], alg):
            bad.append(n)
    assert not bad, f"{alg}: roots differ for tree sizes {bad[:10]}"


def test_merkle_launch_plan_of_the_70b_set():
    # the 723 per-tensor trees of the 70B-shaped set: two group launches (the
    # first with its last groups on four lanes when the rest fill whole
    # rounds), then tiles
    lens = W.workload_lengths(5)
    leaves = [-(-int(L) // 65536) for L in lens]
    seg = np.concatenate([[0], np.cumsum(leaves)]).astype(np.uint64)
    rnd = 256 * torch.cuda.get_device_properties(DEV).multi_processor_count
    plan = hv.merkle_launches(seg)
    assert [p[0] for p in plan] == ["group", "group", "tile"], plan
    kind, units, one = plan[0]
    assert units == sum(-(-c // 8) for c in leaves)
    assert one == units or (one % rnd == 0 and units - one < rnd), plan
    assert plan[1][2] == plan[1][1]  # under one round: every group on one lane
    # the manifest over the 723 roots: a 512-node tile and a tile of two
    assert hv.merkle_launches(np.array([0, len(leaves)], dtype=np.uint64)) == [("tile", 2, 0), ("tile", 1, 0)]


@pytest.mark.parametrize("n", [(1 << 18) - 1, 1 << 18, (1 << 18) + 1, (1 << 18) + 7, 3 * (1 << 18) + 5,
                               (1 << 21) - 8, (1 << 21) - 7, (1 << 21) + 1])
def test_merkle_single_tree_around_the_group_threshold(n):
    entries = W.random_bytes(n * 32, 270 + n % 97, DEV).view(n, 32)
    root = hv.hv_merkle_reduce(entries, np.array([0, n], dtype=np.uint64))
    torch.cuda.synchronize()
    assert bytes(root.cpu().numpy().reshape(-1)) == oracle.mth(entries.cpu().numpy())


def test_verify_and_compare():
    entries = W.random_bytes(5 * 32, 300, DEV).view(5, 32)
    root = hv.hv_merkle_reduce(entries, np.array([0, 5], dtype=np.uint64))
    want = oracle.mth(entries.cpu().numpy())
    assert hv.hv_verify_root(root, want)
    for byte in (0, 13, 31):
        for bit in (0, 7):
            bad = bytearray(want)
            bad[byte] ^= 1 << bit
            assert not hv.hv_verify_root(root, bytes(bad))
    a = W.random_bytes(10 * 32, 301, DEV).view(10, 32)
    b = a.clone()
    b[3, 0] ^= 1
    b[9, 31] ^= 128
    mism = hv.hv_compare_roots(a, b).cpu().numpy()
    assert list(np.nonzero(mism)[0]) == [3, 9]


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
@pytest.mark.parametrize("align_off", [0, 5])
def test_single_long_chunk(alg, align_off):
    # one 48 MiB + 17 byte message as one chunk: one lane runs ~786K dependent
    # blocks (the long-loop and tail paths of both load paths)
    n = (48 << 20) + 17
    buf, host, ptrs, lens, starts = place([n], align_off, seed=77)
    leaves, _ = hv.hv_hash_chunks((ptrs, lens), 0, DEV, alg=alg)
    torch.cuda.synchronize()
    assert bytes(leaves.cpu().numpy()[0]) == oracle.digest(host[int(starts[0]):int(starts[0]) + n].tobytes(), alg)


@pytest.fixture
def leaf_kernel():
    yield hv.set_leaf_kernel
    hv.set_leaf_kernel("auto")


def test_automatic_leaf_kernel_choice_by_leaf_count(leaf_kernel):
    # the two-wave kernel while every CU holds at most one workgroup (one pair
    # up to 64 leaves per CU, two up to 128), the one-wave kernel beyond
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    leaf_kernel("auto")
    assert [hv.leaf_kernel_for(n) for n in (1, 64 * cus, 64 * cus + 1, 128 * cus, 128 * cus + 1)] == \
        ["two-wave", "two-wave", "two-wave-compact", "two-wave-compact", "one-wave"]
    leaf_kernel("one-wave")
    assert hv.leaf_kernel_for(10) == "one-wave"


@pytest.mark.parametrize("choice", ["one-wave", "two-wave", "two-wave-compact"])
@pytest.mark.parametrize("align_off", [0, 3])
@pytest.mark.parametrize("C", [64, 4096, 0])
def test_both_sha256_leaf_kernels(C, align_off, choice, leaf_kernel):
    # the one-wave kernel and the two-wave kernel (message schedule on a second
    # wave) forced on the same inputs, every length 0..1100
    leaf_kernel(choice)
    lens = np.arange(0, 1101)
    buf, host, ptrs, lens, starts = place(lens, align_off, seed=150 + align_off)
    check_all(buf, host, ptrs, lens, starts, C, f"{choice} C={C} off={align_off}")


@pytest.mark.parametrize("choice", ["one-wave", "two-wave", "two-wave-compact"])
@pytest.mark.parametrize("C", [64, 0])
def test_both_kernels_mixed_alignment(C, choice, leaf_kernel):
    # every message at its own offset 0..15 from a 16-byte boundary, so waves
    # mix aligned and unaligned chunks (the kernels choose a load path per wave)
    leaf_kernel(choice)
    rng = np.random.default_rng(152)
    lens = np.concatenate([np.arange(0, 300), rng.integers(300, 5000, 200)]).astype(np.uint64)
    offs = (np.arange(len(lens)) * 7) % 16
    starts = np.zeros(len(lens), dtype=np.uint64)
    pos = 0
    for i, n in enumerate(lens):
        starts[i] = pos + offs[i]
        pos += (int(n) + int(offs[i]) + 16 + 15) // 16 * 16
    buf = W.random_bytes(pos, 153, DEV)
    host = buf.cpu().numpy()
    ptrs = np.uint64(buf.data_ptr()) + starts
    ptrs[lens == 0] = 0
    check_all(buf, host, ptrs, lens, starts, C, f"{choice} mixed C={C}")


@pytest.mark.parametrize("choice", ["auto", "two-wave"])
def test_two_wave_kernel_two_pairs(choice, leaf_kernel):
    # more than 64 chunks per CU: the two-wave kernel runs two producer/consumer
    # pairs per workgroup; random lengths and offsets give the pairs of a
    # workgroup different block counts and load paths
    leaf_kernel(choice)
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 100 * cus
    rng = np.random.default_rng(154)
    lens = rng.integers(0, 1500, n).astype(np.uint64)
    lens[rng.integers(0, n, 40)] = rng.integers(20000, 70000, 40).astype(np.uint64)
    offs = rng.integers(0, 16, n) * (rng.random(n) < 0.1)
    starts = np.zeros(n, dtype=np.uint64)
    pos = 0
    for i, L in enumerate(lens):
        starts[i] = pos + offs[i]
        pos += (int(L) + int(offs[i]) + 16 + 15) // 16 * 16
    buf = W.random_bytes(pos, 155, DEV)
    host = buf.cpu().numpy()
    ptrs = np.uint64(buf.data_ptr()) + starts
    ptrs[lens == 0] = 0
    check_all(buf, host, ptrs, lens, starts, 0, f"{choice} two pairs n={n}")


@pytest.mark.parametrize("choice", ["one-wave", "two-wave"])
def test_both_kernels_long_chunks(choice, leaf_kernel):
    leaf_kernel(choice)
    lens = [(8 << 20) + 55, (8 << 20) + 56, 3 << 20, 1, 0]
    buf, host, ptrs, lens, starts = place(lens, 0, seed=151)
    check_all(buf, host, ptrs, lens, starts, 0, f"{choice} long")
