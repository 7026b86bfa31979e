"""Seeded synthetic ICL-attention inputs shaped like the paper's workloads.

This module holds no arithmetic of the method (no scaling, no quantization,
no attention): it only draws random tables, so both the GPU tests and the
CPU oracle can be fed the same inputs.

The paper measures on TabArena / BeyondArena with TabPFN-v3 activations,
which are not available here; these draws stand in for them.  Shapes follow
the paper: head_dim 64 (and 128 in its appendix), H = 8 heads with H_kv = H
(Table 2 caption), up to hundreds of thousands of train rows.  Values are
i.i.d. N(0,1) times a per-(table, tensor, head) multiplier drawn uniformly,
with a few per-head outlier channels inflated to stress the absmax scale.

Draw order (frozen; changing it changes every stored expectation): for each
table b, for X in (Q over all N+M rows, K, V): the H head multipliers, then
(if outliers are on) the outlier channels of each head without replacement,
then the (rows, H, D) float32 normals.  Q_test is the last M rows of Q, so it
shares the train queries' multipliers and outlier channels (same projection).
bf16 workloads are rounded to bf16 (round-to-nearest-even, by torch) and
returned widened to float32, which represents them exactly.
"""
from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    D: int
    N: int
    M: int
    dtype: str                 # "f32" or "bf16": the dtype handed to the library
    mult_lo: float = 0.5
    mult_hi: float = 4.0
    outlier_frac: float = 0.01
    outlier_factor: float = 20.0
    seed: int = 0

    @property
    def alpha(self):
        """Softmax scale 1/sqrt(d) as the fp32 value passed to the library."""
        return float(np.float32(1.0 / np.sqrt(self.D)))

    @property
    def flops(self):
        """QK^T + PV multiply-adds x2 over both ICL calls: 4*B*H*D*N*(N+M)."""
        return 4.0 * self.B * self.H * self.D * self.N * (self.N + self.M)

    def with_(self, **kw):
        return replace(self, **kw)


WORKLOADS = {
    # tiny: fp32 inputs, outlier stress, finishes on the oracle in seconds
    "tiny": Workload("tiny", B=1, H=2, D=64, N=512, M=128, dtype="f32", seed=0),
    # the train-row count at which FP8 attention is switched on
    "threshold": Workload("threshold", B=1, H=6, D=64, N=8192, M=2048, dtype="bf16", seed=1),
    # headline: two independent tables, 64k train rows
    "mid": Workload("mid", B=2, H=6, D=64, N=65536, M=16384, dtype="bf16", seed=2),
    # long K/V streaming and a wide quantization range, head_dim 128
    "large": Workload("large", B=1, H=8, D=128, N=262144, M=32768, dtype="bf16",
                      mult_lo=0.25, mult_hi=8.0, outlier_frac=0.005, outlier_factor=50.0, seed=3),
    # many small tables below the switch-on threshold, no outliers
    "many_tables": Workload("many_tables", B=64, H=6, D=64, N=4096, M=1024, dtype="bf16",
                            outlier_frac=0.0, seed=4),
}


def _to_bf16_values(x):
    import torch
    return torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()


def generate(w):
    """Draw one workload: dict of float32 arrays q_train (B,N,H,D), k, v (B,N,H,D), q_test (B,M,H,D)."""
    rng = np.random.default_rng(w.seed)
    B, H, D, N, M = w.B, w.H, w.D, w.N, w.M
    out = {"q_train": np.empty((B, N, H, D), np.float32), "k": np.empty((B, N, H, D), np.float32),
           "v": np.empty((B, N, H, D), np.float32), "q_test": np.empty((B, M, H, D), np.float32)}
    n_out = max(1, int(round(w.outlier_frac * D))) if w.outlier_frac > 0 else 0
    for b in range(B):
        for name, rows in (("q", N + M), ("k", N), ("v", N)):
            mult = rng.uniform(w.mult_lo, w.mult_hi, size=H).astype(np.float32)
            chans = [rng.choice(D, n_out, replace=False) for _ in range(H)] if n_out else []
            z = rng.standard_normal((rows, H, D), dtype=np.float32)
            z *= mult[None, :, None]
            for h, ch in enumerate(chans):
                z[:, h, ch] *= np.float32(w.outlier_factor)
            if w.dtype == "bf16":
                z = _to_bf16_values(z)
            if name == "q":
                out["q_train"][b] = z[:N]
                out["q_test"][b] = z[N:]
            else:
                out[name][b] = z
    return out
