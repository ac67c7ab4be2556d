"""Seeded synthetic workloads: shapes, chunk layouts and input tensors.

This module holds no attention arithmetic.  It only describes the workloads
(the Wan2.1-shaped teacher-forcing attention problems) and draws their inputs,
so that the HIP path and the CPU oracle can be fed the very same values.

Workload shapes follow the paper's video setting (Sec. 4 setup: Wan2.1 T2V at
832x480, 21 latent frames of 1560 tokens each; chunk-wise = 3 latent frames
per chunk, frame-wise = 1 latent frame per chunk; the teacher-forcing sequence
packs [clean | noisy] copies of all chunks).  Inputs are i.i.d. normal, drawn
in fp32 in the order Q, K, V, dQ, dK, dV with a seeded torch generator, the
tangents scaled by ``tangent_std``, then rounded to the workload dtype
(round-to-nearest-even).  These random inputs stand in for real activations,
which need model weights that are not available.
"""
from dataclasses import dataclass, field

import torch

MASK_FULL = "full"
MASK_BLOCK_CAUSAL = "block_causal"
MASK_TEACHER_FORCING = "teacher_forcing"
MASK_RANGES = "ranges"

TOKENS_PER_LATENT_FRAME = 1560


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    D: int
    dtype: str                 # "f32" or "bf16"
    kind: str                  # MASK_* above
    # chunk prefix offsets (TF / block-causal), or query groups ((q0, q1, ((k0, k1), ...)), ...)
    # tiling [0, L) (ranges)
    offsets: tuple = field(default=())
    L_full: int = 0            # sequence length for the full mask
    tangent_std: float = 1.0

    @property
    def L(self) -> int:
        if self.kind == MASK_FULL:
            return self.L_full
        if self.kind == MASK_RANGES:
            return self.offsets[-1][1]
        half = self.offsets[-1]
        return 2 * half if self.kind == MASK_TEACHER_FORCING else half

    @property
    def num_chunks(self) -> int:
        return len(self.offsets) if self.kind == MASK_RANGES else max(0, len(self.offsets) - 1)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def describe(self) -> dict:
        d = {"workload": self.name, "B": self.B, "H": self.H, "L": self.L, "D": self.D,
             "dtype": self.dtype, "mask": self.kind}
        if self.kind == MASK_RANGES:
            d["groups"] = len(self.offsets)
        elif self.kind != MASK_FULL:
            sizes = sorted(set(self.offsets[i + 1] - self.offsets[i] for i in range(self.num_chunks)))
            d["chunks"] = self.num_chunks
            d["chunk_tokens"] = sizes[0] if len(sizes) == 1 else sizes
        return d


def uniform_offsets(num_chunks: int, chunk: int) -> tuple:
    return tuple(i * chunk for i in range(num_chunks + 1))


WORKLOADS = {
    # 4 chunks x 16 tokens, [clean | noisy] = 128 tokens, fp32, unit-variance tangents, seed 0
    "tiny_tf": Workload("tiny_tf", 1, 2, 64, "f32", MASK_TEACHER_FORCING, uniform_offsets(4, 16)),
    # Wan2.1-1.3B chunk-wise: 7 chunks x 3 latent frames x 1560 tokens, TF length 65520
    "wan1.3b_chunkwise_tf": Workload("wan1.3b_chunkwise_tf", 1, 12, 128, "bf16", MASK_TEACHER_FORCING,
                                     uniform_offsets(7, 3 * TOKENS_PER_LATENT_FRAME), tangent_std=0.5),
    # Wan2.1-1.3B frame-wise: 21 chunks x 1 latent frame, TF length 65520
    "wan1.3b_framewise_tf": Workload("wan1.3b_framewise_tf", 1, 12, 128, "bf16", MASK_TEACHER_FORCING,
                                     uniform_offsets(21, TOKENS_PER_LATENT_FRAME), tangent_std=0.5),
    # bidirectional teacher: 21 latent frames, full attention, 32760 tokens
    "wan1.3b_bidirectional": Workload("wan1.3b_bidirectional", 1, 12, 128, "bf16", MASK_FULL,
                                      L_full=21 * TOKENS_PER_LATENT_FRAME, tangent_std=0.5),
    # Wan2.1-14B-shaped chunk-wise TF: B=2, 40 heads
    "wan14b_chunkwise_tf": Workload("wan14b_chunkwise_tf", 2, 40, 128, "bf16", MASK_TEACHER_FORCING,
                                    uniform_offsets(7, 3 * TOKENS_PER_LATENT_FRAME), tangent_std=0.5),
}

# workload whose throughput is the headline number (Wan2.1-1.3B chunk-wise TF, one GPU)
HEADLINE = "wan1.3b_chunkwise_tf"


def make_inputs(w: Workload, device="cpu", seed: int = 0, B=None, H=None):
    """Draw Q, K, V, dQ, dK, dV of shape [B, H, L, D] in the workload dtype.

    ``B``/``H`` may shrink the batch/head count (same per-head shape).
    """
    B = w.B if B is None else B
    H = w.H if H is None else H
    shape = (B, H, w.L, w.D)
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    out = {}
    for name in ("Q", "K", "V", "dQ", "dK", "dV"):
        x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        if name.startswith("d") and w.tangent_std != 1.0:
            x.mul_(w.tangent_std)
        out[name] = x.to(w.torch_dtype)
        del x
    return out


def custom_workload(name, B, H, D, dtype, kind, num_chunks=0, chunk=0, L=0, tangent_std=1.0, offsets=None):
    """A workload of arbitrary shape (tests: ragged tails, C=1, N=1, D=64 ...)."""
    if kind == MASK_FULL:
        return Workload(name, B, H, D, dtype, kind, (), L, tangent_std)
    if kind == MASK_RANGES:
        groups = tuple((int(q0), int(q1), tuple((int(a), int(b)) for a, b in ks)) for q0, q1, ks in offsets)
        return Workload(name, B, H, D, dtype, kind, groups, 0, tangent_std)
    offs = tuple(offsets) if offsets is not None else uniform_offsets(num_chunks, chunk)
    return Workload(name, B, H, D, dtype, kind, offs, 0, tangent_std)
