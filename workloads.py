"""Seeded synthetic workloads for neighborhood attention (inputs only).

This module holds the problem shapes and the seeded input generator shared by
the tests, the smoke check and the benchmark.  It contains none of the
method's arithmetic: it only draws iid N(0, 1) tensors and rounds them to the
working dtype.

Recipe (the paper benchmarks random tensors of many shapes, Sec. 4; its sweep
sizes are not published, so these five problems, plus a causal-time variant
of the 3-D one, stand in for it):
  * torch.randn on a CPU generator seeded with ``seed`` (0 by default),
    drawn in the order q, k, v, dO, each fp32 with shape [B, H, X_1..X_r, D];
  * then cast to the working dtype with round-to-nearest-even;
  * softmax scale 1/sqrt(D).
"""
import math
from dataclasses import dataclass, field
from typing import Tuple

import torch


@dataclass(frozen=True)
class Problem:
    name: str
    batch: int
    heads: int
    extents: Tuple[int, ...]
    head_dim: int
    kernel_size: Tuple[int, ...]
    dilation: Tuple[int, ...]
    dtype: str  # "fp32" | "fp16" | "bf16"
    backward: bool = False
    scale: float = field(default=None)
    causal: Tuple[bool, ...] = field(default=None)  # per axis; None: no causal axis

    @property
    def rank(self):
        return len(self.extents)

    @property
    def tokens(self):
        return int(math.prod(self.extents))

    @property
    def window(self):
        return int(math.prod(self.kernel_size))

    @property
    def causal_axes(self):
        return tuple(bool(c) for c in self.causal) if self.causal else (False,) * self.rank

    def pairs_per_slice(self):
        """Query-neighbour pairs of one (batch, head): N * ell without causal axes.

        The neighbourhood is a product of per-axis windows, so the count is a
        product of per-axis sums; along a causal axis position p of a group
        has min(k, p + 1) neighbours.
        """
        total = 1
        for L, k, d, c in zip(self.extents, self.kernel_size, self.dilation, self.causal_axes):
            total *= sum(min(k, x // d + 1) for x in range(L)) if c else L * k
        return total

    @property
    def softmax_scale(self):
        return self.scale if self.scale is not None else 1.0 / math.sqrt(self.head_dim)

    @property
    def shape(self):
        return (self.batch, self.heads) + tuple(self.extents) + (self.head_dim,)

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "fp32" else 2

    def fwd_flops(self):
        """Useful forward FLOPs: 4 * D per query-neighbour pair, i.e. 4 * B * H * N * ell * D
        without causal axes (unmasked neighbourhood work only)."""
        return 4 * self.batch * self.heads * self.pairs_per_slice() * self.head_dim

    def bwd_flops(self):
        """Useful backward FLOPs: 10 * D per pair (S, dP, dV, dQ, dK contractions)."""
        return 10 * self.batch * self.heads * self.pairs_per_slice() * self.head_dim

    def fwd_bytes(self):
        """Algorithmic forward HBM bytes: read q, k, v; write out and fp32 logsumexp."""
        rows = self.batch * self.heads * self.tokens
        return rows * (4 * self.head_dim * self.elem_bytes + 4)

    def bwd_bytes(self):
        """Algorithmic backward HBM bytes: read q, k, v, out, dO, lse; write dq, dk, dv; Delta w+r."""
        rows = self.batch * self.heads * self.tokens
        return rows * (8 * self.head_dim * self.elem_bytes + 12)

    def describe(self):
        ext = "x".join(str(e) for e in self.extents)
        ks = "x".join(str(k) for k in self.kernel_size)
        ds = "x".join(str(d) for d in self.dilation)
        cs = "".join("c" if c else "-" for c in self.causal_axes)
        return (f"{self.rank}-D NA {'fwd+bwd' if self.backward else 'fwd'} {self.dtype}: "
                f"B={self.batch} H={self.heads} X={ext} D={self.head_dim} k={ks} d={ds}"
                + (f" causal={cs}" if any(self.causal_axes) else ""))


# The five workloads: shapes, windows and dilations of the paper's 1-D, 2-D and
# 3-D problem families (Sec. 4), one of each kind.
CONFIGS = {
    "1d_fp32_L256_k7": Problem("1d_fp32_L256_k7", 1, 2, (256,), 32, (7,), (1,), "fp32"),
    "2d_fp16_56x56_k7": Problem("2d_fp16_56x56_k7", 4, 4, (56, 56), 32, (7, 7), (1, 1), "fp16"),
    "2d_bf16_128x128_k13_d2": Problem("2d_bf16_128x128_k13_d2", 2, 8, (128, 128), 64, (13, 13),
                                      (2, 2), "bf16", backward=True),
    "1d_fp16_L32768_k1023_d4": Problem("1d_fp16_L32768_k1023_d4", 1, 16, (32768,), 64, (1023,),
                                       (4,), "fp16"),
    "3d_fp16_16x64x64_k7_d122": Problem("3d_fp16_16x64x64_k7_d122", 1, 8, (16, 64, 64), 64,
                                        (7, 7, 7), (1, 2, 2), "fp16", backward=True),
    # the same volume with causal masking along time (T), the spatio-temporal
    # use of causal NA that Sec. 3.4 names
    "3d_fp16_16x64x64_k7_d122_causal_t": Problem(
        "3d_fp16_16x64x64_k7_d122_causal_t", 1, 8, (16, 64, 64), 64, (7, 7, 7), (1, 2, 2), "fp16",
        backward=True, causal=(True, False, False)),
}
CONFIG_ORDER = list(CONFIGS)
# The workload the benchmark times (forward and backward): 2-D 7x7 fp16.
BENCH_WORKLOAD = "2d_fp16_56x56_k7"

TORCH_DTYPE = {"fp32": torch.float32, "fp16": torch.float16, "bf16": torch.bfloat16}


def make_inputs(problem: Problem, seed: int = 0, with_grad: bool = None):
    """Seeded CPU inputs (q, k, v[, dO]) already rounded to the problem's dtype.

    Draw order q, k, v, dO from torch.Generator().manual_seed(seed), fp32 N(0,1),
    then ``.to(dtype)`` (round to nearest even).
    """
    if with_grad is None:
        with_grad = problem.backward
    gen = torch.Generator().manual_seed(seed)
    dt = TORCH_DTYPE[problem.dtype]
    names = ["q", "k", "v"] + (["dout"] if with_grad else [])
    out = {}
    for n in names:
        out[n] = torch.randn(problem.shape, generator=gen, dtype=torch.float32).to(dt)
    return out


def sample_rows(total_rows: int, count: int, seed: int = 1):
    """Seeded sample of flat row indices (always includes the first and last rows)."""
    gen = torch.Generator().manual_seed(seed)
    if count >= total_rows:
        return torch.arange(total_rows, dtype=torch.int64)
    pick = torch.randperm(total_rows, generator=gen)[: max(count - 2, 0)]
    pick = torch.cat([pick, torch.tensor([0, total_rows - 1])])
    return torch.unique(pick)
