"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module only produces bytes and their layout: no hashing, chunking or
tree arithmetic lives here, so that the oracle and the HIP path can both take
their inputs from it without sharing any of the method.

The paper measures nothing on a public dataset; its workloads are "multi-GB
model shards" and ">100 GB models" (Introduction; Discussion).  These
generators stand in for real checkpoints with the tensor shapes of
Llama-style decoders, weights drawn N(0, 0.02) and rounded to bfloat16
(round-to-nearest-even, torch's cast), stored little-endian as on the GPU.

Workloads (index k, seed 251023938 + k):
  1  64 MiB of uniform random bytes, one message, 1 MiB chunks
  2  1B-shaped decoder (16 layers, d 2048, FFN 8192, vocab 32000, untied
     lm_head): 147 tensors, each its own message, 1 MiB chunks, manifest
  3  7B-shaped decoder (32 layers, d 4096, FFN 11008, vocab 32000): 291
     tensors packed into 32 shard files by layer, 4 MiB chunks, manifest
  4  1,000,000 messages, lengths uniform in [4096, 65536] with multiples of
     64 redrawn, packed at 64-byte aligned offsets, whole-message chunks,
     one tree over all message digests
  5  70B-shaped decoder (80 layers, d 8192, FFN 28672, 64 heads / 8 KV
     heads, vocab 128256): 723 tensors, 64 KiB chunks, manifest
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

SEED_BASE = 251023938
MiB = 1 << 20
KiB = 1 << 10


def seed_of(k: int) -> int:
    return SEED_BASE + k


def tensor_seed(k: int, i: int) -> int:
    """Seed of tensor i (in name order) of workload k."""
    return (seed_of(k) * 1000003 + i) % (1 << 63)


# --------------------------------------------------------------------------
# tensor lists

def decoder_tensors(layers, d, ffn, vocab, kv_dim=None):
    """[(name, shape)] of a Llama-style decoder in byte-wise name order."""
    kv_dim = d if kv_dim is None else kv_dim
    out = [("model.embed_tokens.weight", (vocab, d)), ("model.norm.weight", (d,)), ("lm_head.weight", (vocab, d))]
    for l in range(layers):
        p = f"model.layers.{l}."
        out += [
            (p + "self_attn.q_proj.weight", (d, d)),
            (p + "self_attn.k_proj.weight", (kv_dim, d)),
            (p + "self_attn.v_proj.weight", (kv_dim, d)),
            (p + "self_attn.o_proj.weight", (d, d)),
            (p + "mlp.gate_proj.weight", (ffn, d)),
            (p + "mlp.up_proj.weight", (ffn, d)),
            (p + "mlp.down_proj.weight", (d, ffn)),
            (p + "input_layernorm.weight", (d,)),
            (p + "post_attention_layernorm.weight", (d,)),
        ]
    return sorted(out, key=lambda t: t[0].encode("utf-8"))


def tensors_1b():
    return decoder_tensors(16, 2048, 8192, 32000)


def tensors_7b():
    return decoder_tensors(32, 4096, 11008, 32000)


def tensors_70b():
    return decoder_tensors(80, 8192, 28672, 128256, kv_dim=1024)


def shard_files_7b():
    """[(file name, [tensor names in name order])]: layer k's tensors in file k,
    embed_tokens in file 0, lm_head and the final norm in file 31."""
    files = [[] for _ in range(32)]
    for name, _ in tensors_7b():
        if name.startswith("model.layers."):
            files[int(name.split(".")[2])].append(name)
        elif name == "model.embed_tokens.weight":
            files[0].append(name)
        else:
            files[31].append(name)
    return [(f"model-{k + 1:05d}-of-00032", sorted(v, key=lambda s: s.encode("utf-8"))) for k, v in enumerate(files)]


def numel(shape) -> int:
    n = 1
    for s in shape:
        n *= s
    return n


# --------------------------------------------------------------------------
# generators (device-side; any torch device works)

def bf16_weights(shape, seed: int, device) -> torch.Tensor:
    """N(0, 0.02) fp32 rounded to bf16, as a tensor of the given shape."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = torch.empty(shape, dtype=torch.bfloat16, device=device)
    flat = out.view(-1)
    step = 1 << 28  # bound the fp32 temporary to 1 GiB
    for lo in range(0, flat.numel(), step):
        hi = min(lo + step, flat.numel())
        tmp = torch.randn(hi - lo, generator=g, dtype=torch.float32, device=device)
        flat[lo:hi] = (tmp * 0.02).to(torch.bfloat16)
    return out


def random_bytes(n: int, seed: int, device) -> torch.Tensor:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randint(0, 256, (n,), generator=g, dtype=torch.uint8, device=device)


def as_bytes(t: torch.Tensor) -> torch.Tensor:
    """A flat uint8 view of a contiguous tensor's storage bytes."""
    return t.contiguous().view(-1).view(torch.uint8)


@dataclass
class MessageSet:
    """Messages to hash: names, device byte tensors and/or raw (ptr, len) arrays.

    ``ptrs`` / ``lens`` describe every message (device addresses); ``owners``
    keeps the storage alive.  ``views`` holds per-message uint8 tensors when
    the set is small enough to keep them as Python objects.
    """
    names: list
    ptrs: np.ndarray
    lens: np.ndarray
    owners: list = field(default_factory=list)
    views: list | None = None
    buffer: torch.Tensor | None = None    # one packed buffer holding every message, if any
    offsets: np.ndarray | None = None     # byte offsets of the messages in ``buffer``

    def __post_init__(self):
        # the message table is fixed once made: read-only arrays let a caller
        # (the binding's Verifier) keep the descriptor table built from them
        self.ptrs = np.asarray(self.ptrs, dtype=np.uint64)
        self.lens = np.asarray(self.lens, dtype=np.uint64)
        self.ptrs.flags.writeable = False
        self.lens.flags.writeable = False

    @property
    def total_bytes(self) -> int:
        return int(self.lens.sum()) if len(self.lens) else 0

    def __len__(self):
        return len(self.lens)


def message_set(named) -> MessageSet:
    """From [(name, tensor)]: each tensor's bytes are one message."""
    views = [as_bytes(t) for _, t in named]
    ptrs = np.array([v.data_ptr() for v in views], dtype=np.uint64)
    lens = np.array([v.numel() for v in views], dtype=np.uint64)
    return MessageSet([n for n, _ in named], ptrs, lens, owners=[t for _, t in named], views=views)


@dataclass
class Workload:
    k: int
    chunk_bytes: int
    msgs: MessageSet
    manifest: bool          # roots per message, then one root over them
    description: str


def workload(k: int, device) -> Workload:
    """Build workload k on ``device`` (see the module docstring)."""
    if k == 1:
        buf = random_bytes(64 * MiB, seed_of(1), device)
        return Workload(1, MiB, message_set([("blob", buf)]), False,
                        "64 MiB uniform random bytes, 1 MiB chunks, single root")
    if k == 2:
        named = [(n, bf16_weights(s, tensor_seed(2, i), device)) for i, (n, s) in enumerate(tensors_1b())]
        return Workload(2, MiB, message_set(named), True,
                        "1B-shaped bf16 decoder, 147 tensors, 1 MiB chunks, per-tensor roots + manifest")
    if k == 3:
        shapes = dict(tensors_7b())
        order = {n: i for i, (n, _) in enumerate(tensors_7b())}
        named = []
        for fname, tnames in shard_files_7b():
            size = sum(numel(shapes[t]) * 2 for t in tnames)
            buf = torch.empty(size, dtype=torch.uint8, device=device)
            off = 0
            for t in tnames:
                nb = numel(shapes[t]) * 2
                buf[off:off + nb] = as_bytes(bf16_weights(shapes[t], tensor_seed(3, order[t]), device))
                off += nb
            named.append((fname, buf))
        return Workload(3, 4 * MiB, message_set(named), True,
                        "7B-shaped bf16 decoder in 32 shard files, 4 MiB chunks, per-file roots + manifest")
    if k == 4:
        return _small_messages(device)
    if k == 5:
        named = [(n, bf16_weights(s, tensor_seed(5, i), device)) for i, (n, s) in enumerate(tensors_70b())]
        return Workload(5, 64 * KiB, message_set(named), True,
                        "70B-shaped bf16 decoder, 723 tensors, 64 KiB chunks, per-tensor roots + manifest")
    raise ValueError(f"no workload {k}")


def small_message_lengths(n: int = 1_000_000, seed: int | None = None) -> np.ndarray:
    """Lengths uniform over [4096, 65536], multiples of 64 redrawn."""
    rng = np.random.default_rng(seed_of(4) if seed is None else seed)
    out = rng.integers(4096, 65536, n, endpoint=True, dtype=np.int64)
    bad = out % 64 == 0
    while bad.any():
        out[bad] = rng.integers(4096, 65536, int(bad.sum()), endpoint=True, dtype=np.int64)
        bad = out % 64 == 0
    return out.astype(np.uint64)


def packed_offsets(lens: np.ndarray, align: int = 64) -> np.ndarray:
    """Start offsets of messages packed back to back at ``align``-byte boundaries."""
    padded = (lens + np.uint64(align - 1)) // np.uint64(align) * np.uint64(align)
    offs = np.zeros(len(lens), dtype=np.uint64)
    if len(lens) > 1:
        offs[1:] = np.cumsum(padded[:-1])
    return offs


def _small_messages(device, n: int = 1_000_000) -> Workload:
    lens = small_message_lengths(n)
    offs = packed_offsets(lens)
    total = int(offs[-1] + lens[-1]) if n else 0
    buf = random_bytes(total, seed_of(4), device)
    ptrs = np.uint64(buf.data_ptr()) + offs
    ms = MessageSet([], ptrs, lens, owners=[buf], buffer=buf, offsets=offs)
    return Workload(4, 0, ms, False,
                    "1,000,000 messages of 4-64 KiB (random bytes), whole-message digests, one root")


def workload_bytes(k: int) -> int:
    """Total message bytes of workload k, from the shapes alone."""
    if k == 1:
        return 64 * MiB
    if k == 2:
        return sum(numel(s) * 2 for _, s in tensors_1b())
    if k == 3:
        return sum(numel(s) * 2 for _, s in tensors_7b())
    if k == 4:
        return int(small_message_lengths().sum())
    if k == 5:
        return sum(numel(s) * 2 for _, s in tensors_70b())
    raise ValueError(k)


def workload_lengths(k: int) -> list:
    """Per-message byte lengths of workload k (cheap; no data generated)."""
    if k == 1:
        return [64 * MiB]
    if k == 2:
        return [numel(s) * 2 for _, s in tensors_1b()]
    if k == 3:
        shapes = dict(tensors_7b())
        return [sum(numel(shapes[t]) * 2 for t in ts) for _, ts in shard_files_7b()]
    if k == 4:
        return [int(x) for x in small_message_lengths()]
    if k == 5:
        return [numel(s) * 2 for _, s in tensors_70b()]
    raise ValueError(k)


CHUNK_BYTES = {1: MiB, 2: MiB, 3: 4 * MiB, 4: 0, 5: 64 * KiB}
