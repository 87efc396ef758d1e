"""Seeded synthetic workloads for the ACRL scoring / discrepancy path.

This module is the only thing the oracle side and the GPU side share: it
draws random inputs and holds none of the method's arithmetic.  Every
workload is synthetic; the shapes follow the paper's setting (Qwen-shaped LM
heads, G rollouts per prompt as in the training configuration of Appendix A,
ragged right-padded responses with a response mask).

Distributions:
  * hidden states H ~ N(0, 1), rounded to bf16 (post-RMSNorm activations);
  * LM head W ~ N(0, (2.5/sqrt(d))^2), rounded to bf16;
  * response lengths uniform over the integers [lo, hi]; mask = right padding;
  * rewards Bernoulli(0.5) per response, advantages GRPO-normalised per
    prompt (Sec. 2, the advantage definition after Eq. grpo_objective);
  * uniforms in [0, 1) for inverse-CDF sampling of token ids.

Two backends draw the big tensors: numpy PCG64 on the host (small configs,
CPU tests) and torch's device generator (full-size configs on the GPU).  Each
is deterministic for its seed; they do not produce the same numbers.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

# sub-stream ids per tensor
STREAM_H, STREAM_W, STREAM_LEN, STREAM_IDS, STREAM_ADV = 0, 1, 2, 3, 4

PER_TENSOR, PER_ROW, MX32 = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    d: int              # hidden size
    V: int              # vocabulary size
    n_prompts: int      # groups
    G: int              # rollouts per prompt
    L: int              # slots per response (max response length)
    len_lo: int
    len_hi: int
    scaling: int        # mu's FP8 scaling: PER_TENSOR / PER_ROW / MX32
    temperature: float
    seed: int
    chunk_rows: int = 0  # >0: the scorer is called on row chunks of this size

    @property
    def B(self) -> int:
        return self.n_prompts * self.G

    @property
    def slots(self) -> int:
        return self.B * self.L

    @property
    def inv_temperature(self) -> float:
        return 1.0 / self.temperature

    def describe(self) -> str:
        sc = {PER_TENSOR: "fp8 e4m3 per-tensor", PER_ROW: "fp8 e4m3 per-row/per-token",
              MX32: "mxfp8 (e4m3, e8m0 per 32 along d)"}[self.scaling]
        return ("%s: d=%d V=%d, %d prompts x %d rollouts x %d slots, lengths U[%d,%d], mu=%s, tau=%g"
                % (self.name, self.d, self.V, self.n_prompts, self.G, self.L, self.len_lo,
                   self.len_hi, sc, self.temperature))


WORKLOADS: Dict[str, Workload] = {
    # small parity case: 1 prompt x 4 rollouts x 64 slots
    "tiny": Workload("tiny", 256, 2048, 1, 4, 64, 32, 64, PER_ROW, 1.0, 1),
    # Qwen-1.7B-shaped head
    "q17b": Workload("q17b", 2048, 151936, 16, 8, 1024, 256, 1024, PER_ROW, 1.0, 2),
    # Qwen-8B-shaped head (the headline workload)
    "q8b": Workload("q8b", 4096, 151936, 8, 8, 4096, 1024, 4096, PER_TENSOR, 1.0, 3),
    # long responses, scored in token chunks
    "long": Workload("long", 4096, 151936, 4, 16, 16384, 1024, 16384, PER_ROW, 1.0, 4,
                     chunk_rows=65536),
    # MXFP8 variant at temperature 0.7
    "mx": Workload("mx", 5120, 151936, 16, 8, 2048, 512, 2048, MX32, 0.7, 5),
}


def rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def float_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, np.float32).view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return b.astype(np.uint16)


# ------------------------------------------------------------ structure
def lengths(w: Workload) -> np.ndarray:
    return rng(w.seed, STREAM_LEN).integers(w.len_lo, w.len_hi + 1, size=w.B).astype(np.int32)


def mask(w: Workload) -> np.ndarray:
    n = lengths(w)
    m = (np.arange(w.L)[None, :] < n[:, None]).astype(np.uint8)
    return m  # [B, L], right padding


def group_of_seq(w: Workload) -> np.ndarray:
    return (np.arange(w.B) // w.G).astype(np.int32)


def valid_slots(w: Workload) -> np.ndarray:
    """Slot index (i*L + j) of every valid token, sequence-major."""
    return np.flatnonzero(mask(w).reshape(-1)).astype(np.int32)


def n_valid(w: Workload) -> int:
    return int(lengths(w).sum())


def advantages(w: Workload) -> np.ndarray:
    """GRPO advantages from Bernoulli(0.5) rewards, one per response."""
    r = rng(w.seed, STREAM_ADV).integers(0, 2, size=w.B).astype(np.float64)
    r = r.reshape(w.n_prompts, w.G)
    a = (r - r.mean(axis=1, keepdims=True)) / (r.std(axis=1, keepdims=True) + 1e-6)
    return a.reshape(-1).astype(np.float32)


def uniforms(w: Workload, n: int, offset: int = 0) -> np.ndarray:
    u = rng(w.seed, STREAM_IDS).random(offset + n)
    return u[offset:]


# ------------------------------------------------------------ host tensors
def hidden_bf16(w: Workload, n_rows: Optional[int] = None) -> np.ndarray:
    """H for the valid tokens, uint16 bf16 bits [n_rows, d] (numpy backend)."""
    n = n_valid(w) if n_rows is None else n_rows
    x = rng(w.seed, STREAM_H).standard_normal((n, w.d), dtype=np.float32)
    return float_to_bf16_bits(x)


def weights_bf16(w: Workload) -> np.ndarray:
    """W [V, d] bf16 bits (numpy backend)."""
    x = rng(w.seed, STREAM_W).standard_normal((w.V, w.d), dtype=np.float32)
    x *= np.float32(2.5 / np.sqrt(w.d))
    return float_to_bf16_bits(x)


def uniform_ids(w: Workload, n: int) -> np.ndarray:
    return rng(w.seed, STREAM_IDS + 100).integers(0, w.V, size=n).astype(np.int32)


# ------------------------------------------------------------ device tensors
def _torch_gen(seed: int, stream: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000003 + stream)
    return g


def hidden_bf16_torch(w: Workload, n_rows: int, device, row_offset: int = 0):
    """H rows [row_offset, row_offset+n_rows) drawn on `device` (torch backend).

    Rows are drawn in blocks of 8192 with one generator per block, so any row
    range is reproducible without drawing the rows before it."""
    import torch
    out = torch.empty((n_rows, w.d), dtype=torch.bfloat16, device=device)
    blk = 8192
    r = row_offset
    end = row_offset + n_rows
    while r < end:
        b = r // blk
        lo, hi = r - b * blk, min(end - b * blk, blk)
        g = _torch_gen(w.seed, 10_000 + b, device)
        x = torch.randn((blk, w.d), generator=g, dtype=torch.float32, device=device)
        out[r - row_offset: r - row_offset + (hi - lo)] = x[lo:hi].to(torch.bfloat16)
        r += hi - lo
    return out


def weights_bf16_torch(w: Workload, device):
    import torch
    out = torch.empty((w.V, w.d), dtype=torch.bfloat16, device=device)
    blk = 8192
    for b in range(0, w.V, blk):
        g = _torch_gen(w.seed, 20_000 + b // blk, device)
        n = min(blk, w.V - b)
        x = torch.randn((n, w.d), generator=g, dtype=torch.float32, device=device)
        out[b:b + n] = (x * (2.5 / float(np.sqrt(w.d)))).to(torch.bfloat16)
    return out
