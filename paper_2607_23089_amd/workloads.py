"""Seeded synthetic inputs for row softmax.

This module draws and shapes input matrices only; it holds none of the
softmax arithmetic, and it is the one piece shared by the GPU path's tests and
benchmark and by the oracle's tests.

Named workloads (rows x cols, dtypes in -> out, value recipe):

  fp32_64x1000       64 x 1000,     f32 -> f32,  N(0, 1), seed 0
  small_262144x64    262144 x 64,   bf16 -> bf16, N(0, 4^2), seed 0
  causal_32768x4096  32768 x 4096,  bf16 -> bf16, N(0, 8^2), seed 0, then
                     x[r, c] = -inf where c > r mod 4096 (8 heads x 4096
                     queries of causally masked attention scores)
  large_1024x262144  1024 x 262144, f32 -> f32,  N(0, 2^2), seed 0, then one
                     entry per row set to +50 at column randint(0, cols)
                     (generator seeded 1)
  vocab_4096x151936  4096 x 151936, bf16 -> f32, N(0, 3^2), seed 0, then
                     k = round(1e-3 * rows * cols) flat positions drawn with
                     randint (generator seeded 1), de-duplicated, each set to
                     +-1e4 (sign from the same generator); 1e4 is 9984 in bf16

Softmax-backward workloads (y and dy of in dtype, dx of out dtype):

  bwd_small_262144x64    262144 x 64,   bf16 -> bf16, alpha 0.5
  bwd_causal_32768x4096  32768 x 4096,  bf16 -> bf16, alpha 0.1, causal
                         (y[r, c] = 0 for c > r mod 4096)
  bwd_large_1024x262144  1024 x 262144, f32 -> f32,  alpha 0.05

  y: each row an independent Dirichlet(alpha) sample over its kept columns
  (gamma(alpha, 1) draws from torch._standard_gamma with a generator seeded
  2, divided by their row total in fp32; small alpha gives the peaked rows
  of trained attention and output layers), 0 in masked columns; dy: N(0, 1)
  with a generator seeded 3.  Both drawn in fp32 on the chosen device, then
  cast to the input dtype.  This is a probability-vector sampler, not the
  softmax: no exponential and no maximum is involved.

MoE group-score workloads (scores tokens x experts of in dtype; group
scores tokens x experts / 32 written):

  moe_65536x256_f32      65536 x 256, f32 -> f32, groups of 32
  moe_65536x256_bf16     65536 x 256, bf16 -> f32, groups of 32
  moe_1048576x256_f32    1048576 x 256, f32 -> f32, groups of 32

  256 routed experts in 8 groups of 32 is the routing shape the paper's
  operator serves; 65536 tokens is a large prefill batch, 1048576 tokens a
  bandwidth-scale batch.  Scores: N(0, 1) in fp32 from a generator seeded 4,
  cast to the input dtype; in bf16 about one group in a hundred holds a
  tied maximum, the case the paper's rewrite must keep.

Recipe: draw fp32 N(0, 1) with torch.randn from a torch.Generator seeded as
stated on the chosen device, scale by sigma, apply the structure, then cast
to the input dtype (round to nearest even for bf16).  The GPU and the oracle
always read the same cast tensor.  The large workloads are drawn on the GPU
(torch's CPU normal generator needs over a minute for 622M values); the
device is part of the recipe because the two generators give different
streams.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

F32, BF16 = "f32", "bf16"
TORCH_DTYPES = {F32: torch.float32, BF16: torch.bfloat16}


@dataclass(frozen=True)
class Workload:
    name: str
    rows: int
    cols: int
    in_dtype: str
    out_dtype: str
    sigma: float
    structure: str = "none"      # none | causal | spike | outliers
    period: int = 0              # causal: queries per head
    spike: float = 0.0           # spike value
    outlier_frac: float = 0.0    # outliers: fraction of entries
    outlier_value: float = 0.0

    @property
    def in_bytes(self) -> int:
        return 4 if self.in_dtype == F32 else 2

    @property
    def out_bytes(self) -> int:
        return 4 if self.out_dtype == F32 else 2

    @property
    def algorithmic_bytes(self) -> int:
        """x read once plus y written once."""
        return self.rows * self.cols * (self.in_bytes + self.out_bytes)


WORKLOADS = {w.name: w for w in (
    Workload("fp32_64x1000", 64, 1000, F32, F32, 1.0),
    Workload("small_262144x64", 262144, 64, BF16, BF16, 4.0),
    Workload("causal_32768x4096", 32768, 4096, BF16, BF16, 8.0, "causal", period=4096),
    Workload("large_1024x262144", 1024, 262144, F32, F32, 2.0, "spike", spike=50.0),
    Workload("vocab_4096x151936", 4096, 151936, BF16, F32, 3.0, "outliers",
             outlier_frac=1e-3, outlier_value=1e4),
)}

# The four row-length regimes timed together by the benchmark.
REGIMES = ("small_262144x64", "causal_32768x4096", "large_1024x262144",
           "vocab_4096x151936")


@dataclass(frozen=True)
class BackwardWorkload:
    name: str
    rows: int
    cols: int
    in_dtype: str
    out_dtype: str
    alpha: float
    period: int = 0              # causal: queries per head (0: no mask)

    @property
    def in_bytes(self) -> int:
        return 4 if self.in_dtype == F32 else 2

    @property
    def out_bytes(self) -> int:
        return 4 if self.out_dtype == F32 else 2

    @property
    def algorithmic_bytes(self) -> int:
        """y and dy read once plus dx written once."""
        return self.rows * self.cols * (2 * self.in_bytes + self.out_bytes)


BACKWARD_WORKLOADS = {w.name: w for w in (
    BackwardWorkload("bwd_small_262144x64", 262144, 64, BF16, BF16, 0.5),
    BackwardWorkload("bwd_causal_32768x4096", 32768, 4096, BF16, BF16, 0.1, period=4096),
    BackwardWorkload("bwd_large_1024x262144", 1024, 262144, F32, F32, 0.05),
)}


@dataclass(frozen=True)
class MoeWorkload:
    name: str
    tokens: int
    experts: int
    group: int
    in_dtype: str
    out_dtype: str

    @property
    def in_bytes(self) -> int:
        return 4 if self.in_dtype == F32 else 2

    @property
    def out_bytes(self) -> int:
        return 4 if self.out_dtype == F32 else 2

    @property
    def algorithmic_bytes(self) -> int:
        """Scores read once plus group scores written once."""
        return self.tokens * self.experts * self.in_bytes + \
            self.tokens * (self.experts // self.group) * self.out_bytes


MOE_WORKLOADS = {w.name: w for w in (
    MoeWorkload("moe_65536x256_f32", 65536, 256, 32, F32, F32),
    MoeWorkload("moe_65536x256_bf16", 65536, 256, 32, BF16, F32),
    MoeWorkload("moe_1048576x256_f32", 1048576, 256, 32, F32, F32),
)}


def make_moe_scores(w: MoeWorkload, device="cpu", tokens: int | None = None) -> torch.Tensor:
    """Expert scores of a MoE workload on ``device`` in its input dtype."""
    return random_matrix(w.tokens if tokens is None else tokens, w.experts, w.in_dtype,
                         sigma=1.0, seed=4, device=device)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_input(w: Workload, device="cpu", seed: int = 0, structure_seed: int = 1,
               rows: int | None = None) -> torch.Tensor:
    """The workload's input matrix on ``device`` in its input dtype.  ``rows``
    overrides the row count (same recipe, fewer rows) for scaled-down tests."""
    R = w.rows if rows is None else rows
    C = w.cols
    x = torch.randn(R, C, generator=_gen(seed, device), device=device,
                    dtype=torch.float32)
    x.mul_(w.sigma)
    if w.structure == "causal":
        col = torch.arange(C, device=device)
        lim = torch.arange(R, device=device) % w.period
        x.masked_fill_(col[None, :] > lim[:, None], float("-inf"))
    elif w.structure == "spike":
        g1 = _gen(structure_seed, device)
        cols = torch.randint(0, C, (R,), generator=g1, device=device)
        x[torch.arange(R, device=device), cols] = w.spike
    elif w.structure == "outliers":
        g1 = _gen(structure_seed, device)
        k = int(round(w.outlier_frac * R * C))
        pos = torch.unique(torch.randint(0, R * C, (k,), generator=g1, device=device))
        sign = torch.randint(0, 2, (pos.numel(),), generator=g1, device=device)
        vals = (sign.to(torch.float32) * 2.0 - 1.0) * w.outlier_value
        x.view(-1)[pos] = vals
    return x.to(TORCH_DTYPES[w.in_dtype])


def random_matrix(rows: int, cols: int, dtype: str, sigma: float = 1.0, seed: int = 0,
                  device="cpu") -> torch.Tensor:
    """Plain N(0, sigma^2) matrix (no structure) for shape sweeps."""
    x = torch.randn(rows, cols, generator=_gen(seed, device), device=device,
                    dtype=torch.float32)
    x.mul_(sigma)
    return x.to(TORCH_DTYPES[dtype])


def random_probabilities(rows: int, cols: int, dtype: str, alpha: float, seed: int = 2,
                         period: int = 0, device="cpu") -> torch.Tensor:
    """Rows of Dirichlet(alpha) samples (see the module notes); with period > 0,
    row r keeps columns 0 .. r mod period and holds 0 elsewhere."""
    conc = torch.full((rows, cols), float(alpha), device=device, dtype=torch.float32)
    g = torch._standard_gamma(conc, generator=_gen(seed, device))
    del conc
    if period > 0:
        col = torch.arange(cols, device=device)
        lim = torch.arange(rows, device=device) % period
        g.masked_fill_(col[None, :] > lim[:, None], 0.0)
    tot = g.sum(dim=1, keepdim=True)
    g.div_(torch.where(tot > 0, tot, torch.ones_like(tot)))
    return g.to(TORCH_DTYPES[dtype])


def make_backward_inputs(w: BackwardWorkload, device="cpu", rows: int | None = None):
    """(y, dy) of a backward workload on ``device`` in its input dtype."""
    R = w.rows if rows is None else rows
    y = random_probabilities(R, w.cols, w.in_dtype, w.alpha, seed=2, period=w.period,
                             device=device)
    dy = random_matrix(R, w.cols, w.in_dtype, sigma=1.0, seed=3, device=device)
    return y, dy


def to_bits_numpy(t: torch.Tensor):
    """Host numpy view of a tensor's stored values: fp32 values, or bf16 bit
    patterns as uint16 (exact; no arithmetic)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    return t.numpy()


def outlier_count(w: Workload) -> int:
    return int(round(w.outlier_frac * w.rows * w.cols)) if w.structure == "outliers" else 0

