"""hv_hash_chunks_noalloc (the allocation-free form of hv_hash_chunks_alg, its
scratch in a static device array of the library) gives bit for bit the chunk
digests of the workspace entry point, on consecutive calls that reuse the
array, the second with a smaller input, and on a message set that fills the
array exactly.  Called through the C ABI by way of the binding."""
import numpy as np
import pytest
import torch

import workloads as W
from oracle import oracle

from paper_2510_23938_amd import hv  # noqa: E402  (a missing library fails the run, never skips it)

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda")
SCRATCH = hv.HV_NOALLOC_SCRATCH_BYTES


def packed(lens, seed):
    """Messages at unaligned offsets inside one buffer (ragged tails, empty messages)."""
    starts, pos = [], 3
    for n in lens:
        starts.append(pos)
        pos += n + 5
    buf = W.random_bytes(pos + 16, seed, DEV)
    return [buf[s:s + n] for s, n in zip(starts, lens)], buf


def both_ways(msgs, C, alg):
    want, seg = hv.hv_hash_chunks(msgs, C, DEV, alg=alg)
    got, seg2 = hv.hv_hash_chunks_noalloc(msgs, C, DEV, alg=alg)
    torch.cuda.synchronize()
    assert np.array_equal(seg, seg2)
    return got, want, seg


@pytest.mark.parametrize("alg", ["sha256", "sha384"])
def test_two_calls_in_a_row_the_second_smaller(alg):
    rng = np.random.default_rng(77 if alg == "sha256" else 78)
    big = [0, 1, 55, 56, 64, 127, 128, 1000, 4096, 70000, 3 * 65536 + 17] + \
        [int(x) for x in rng.integers(0, 200000, 300)]
    small = [129, 0, 5000, 65536]
    for lens, C, seed in ((big, 4096, 900), (small, 1024, 901)):
        msgs, _ = packed(lens, seed)
        got, want, seg = both_ways(msgs, C, alg)
        assert torch.equal(got, want), (alg, len(lens))
        # and the oracle on the same bytes
        host = [m.cpu().numpy() for m in msgs]
        assert np.array_equal(got.cpu().numpy(), oracle.leaf_digests_mt(host, C, 8, alg)), (alg, len(lens))


@pytest.mark.parametrize("C", [0, 128])
def test_whole_messages_and_empty_sets(C):
    msgs, _ = packed([0, 7, 300, 4097, 0, 128], 902)
    got, want, _ = both_ways(msgs, C, "sha256")
    assert torch.equal(got, want)
    out, seg = hv.hv_hash_chunks_noalloc([], C, DEV)
    assert out.shape == (0, 32) and list(seg) == [0]


def test_message_set_that_fills_the_scratch_exactly():
    # one message of n 64-byte chunks needs 4 x 256 B + 32 KiB + 24 n bytes (rounded up to 256)
    n = 2_794_794
    assert hv.lib.hv_hash_workspace_bytes(1, n) == SCRATCH
    buf = W.random_bytes(n * 64, 903, DEV)
    got, want, _ = both_ways([buf], 64, "sha256")
    assert torch.equal(got, want)
    # sampled leaves against the oracle
    idx = np.random.default_rng(904).choice(n, 64, replace=False)
    host = buf.cpu().numpy()
    for j in idx:
        assert bytes(got[int(j)].cpu().numpy()) == oracle.sha256(host[64 * int(j):64 * int(j) + 64]), int(j)
    # a smaller call right after it reuses the array
    msgs, _ = packed([100, 64 * 1000 + 3, 1], 905)
    got, want, _ = both_ways(msgs, 64, "sha256")
    assert torch.equal(got, want)

