"""Seeded synthetic inputs for the SSD layer, shared by the oracle-side tests and the HIP path.

This module only draws random numbers and casts them to storage dtypes.  It contains none of
the SSD/SSDi8 arithmetic (no softplus, no cumsum, no quantization): the time step is handed
out raw (pre-softplus) and both implementations apply the ChunkCumsum softplus themselves
(Alg. 2, module 1).

Shapes follow the paper's statement of the SSD problem (Sec. 4.1): x (B,L,H,P), dt (B,L,H),
A (H), B and C (B,L,G,N).  The five presets are Mamba-2-shaped layers; their value
distributions stand in for real activations, which the paper shows to have fixed outlier
channels along the H/P axes of x (Fig. 2, Fig. 7) and per-group outliers in B and C (Fig. 7).

Recipe (one place, so that every consumer draws the same tensors):
  * three independent streams  numpy Generator(PCG64(SeedSequence([seed, s]))):
      s = 0  structure and parameters  (A, D, outlier channel sets)
      s = 1  evaluation activations
      s = 2  calibration activations   (same distributions, fresh draw)
  * structure stream, in this order:  A_log ~ U(a_lo, a_hi) [H],  A = -exp(A_log) rounded once
    to fp32;  D ~ N(1, 0.1) [H] rounded to fp32;  x outlier channels: `x_outliers` distinct
    flat (h, p) indices;  for each group g: `bc_outlier_dims` distinct state dims for B, then
    the same count for C.
  * activation streams, per batch element b in order:  x[b] ~ N(0,1) (L,H,P),
    B[b] ~ N(0,1) (L,G,N),  C[b] ~ N(0,1) (L,G,N),  dt_raw[b] ~ N(dt_mu, dt_sigma) (L,H), all
    drawn in fp64; outlier channels are multiplied by their factor; each tensor is then
    rounded once (round-to-nearest-even) to its storage dtype (fp16, or fp32 for the tiny
    preset; dt_raw is always fp32).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class SSDConfig:
    name: str
    batch: int
    seqlen: int
    nheads: int
    headdim: int
    dstate: int
    ngroups: int
    chunk: int
    dtype: str                      # storage dtype of x, B, C and y: "fp16" | "fp32"
    x_outliers: int                 # number of (h, p) outlier channels in x
    x_outlier_scale: float
    bc_outlier_dims: int            # outlier state dims per group, drawn separately for B and C
    bc_outlier_scale: float
    dt_mu: float
    dt_sigma: float
    a_lo: float                     # A = -exp(U(a_lo, a_hi))
    a_hi: float
    xs_per_head: bool = False       # X_scaled step size per head instead of per (head, channel)
    seed: int = 0

    @property
    def tokens(self) -> int:
        return self.batch * self.seqlen

    @property
    def nchunks(self) -> int:
        return self.seqlen // self.chunk

    def scaled(self, **kw) -> "SSDConfig":
        return dataclasses.replace(self, **kw)


LN16 = float(np.log(16.0))

# The five Mamba-2-shaped workloads the throughput and parity figures are quoted on.
CONFIGS: Dict[str, SSDConfig] = {
    "tiny": SSDConfig("tiny", 1, 512, 24, 64, 128, 1, 256, "fp32",
                      31, 20.0, 3, 20.0, -2.0, 0.5, 0.0, LN16),
    "mamba2-130m": SSDConfig("mamba2-130m", 8, 2048, 24, 64, 128, 1, 256, "fp16",
                             31, 20.0, 3, 20.0, -2.0, 0.5, 0.0, LN16),
    "mamba2-2.7b": SSDConfig("mamba2-2.7b", 4, 4096, 80, 64, 128, 1, 256, "fp16",
                             51, 30.0, 4, 15.0, -2.0, 0.5, 0.0, LN16),
    "mamba2-8b-g8": SSDConfig("mamba2-8b-g8", 2, 8192, 128, 64, 128, 8, 256, "fp16",
                              164, 20.0, 3, 20.0, -3.0, 1.0, 0.0, LN16, xs_per_head=True),
    "long-64k": SSDConfig("long-64k", 1, 65536, 80, 64, 128, 1, 256, "fp16",
                          102, 20.0, 3, 20.0, -2.0, 0.5, -4.0, LN16),
}
CONFIG_ORDER = ["tiny", "mamba2-130m", "mamba2-2.7b", "mamba2-8b-g8", "long-64k"]


def _gen(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


def _np_dtype(name: str):
    return {"fp16": np.float16, "fp32": np.float32}[name]


def structure(cfg: SSDConfig) -> Dict[str, np.ndarray]:
    """Parameters and fixed outlier channel sets (stream s = 0)."""
    g = _gen(cfg.seed, 0)
    H, P, N, G = cfg.nheads, cfg.headdim, cfg.dstate, cfg.ngroups
    a_log = g.uniform(cfg.a_lo, cfg.a_hi, size=H)
    A = (-np.exp(a_log)).astype(np.float32)
    D = g.normal(1.0, 0.1, size=H).astype(np.float32)
    x_out = np.sort(g.choice(H * P, size=cfg.x_outliers, replace=False)) if cfg.x_outliers else \
        np.zeros(0, np.int64)
    b_out = np.zeros((G, cfg.bc_outlier_dims), np.int64)
    c_out = np.zeros((G, cfg.bc_outlier_dims), np.int64)
    for gi in range(G):
        b_out[gi] = np.sort(g.choice(N, size=cfg.bc_outlier_dims, replace=False))
        c_out[gi] = np.sort(g.choice(N, size=cfg.bc_outlier_dims, replace=False))
    return {"A": A, "D": D, "x_outliers": x_out, "B_outliers": b_out, "C_outliers": c_out}


def activations(cfg: SSDConfig, stream: int = 1, batch: Optional[int] = None
                ) -> Dict[str, np.ndarray]:
    """x, B, C (storage dtype) and raw (pre-softplus) dt (fp32) for stream 1 (eval) or 2 (calib).

    `batch` overrides the number of batch elements drawn (the first `batch` elements of the
    same stream), which lets bounded samples of a workload reuse its exact leading inputs.
    """
    st = structure(cfg)
    g = _gen(cfg.seed, stream)
    nb = cfg.batch if batch is None else batch
    L, H, P, N, G = cfg.seqlen, cfg.nheads, cfg.headdim, cfg.dstate, cfg.ngroups
    dt_ = _np_dtype(cfg.dtype)
    xsc = np.ones(H * P)
    xsc[st["x_outliers"]] = cfg.x_outlier_scale
    xsc = xsc.reshape(H, P)
    bsc = np.ones((G, N))
    csc = np.ones((G, N))
    for gi in range(G):
        bsc[gi, st["B_outliers"][gi]] = cfg.bc_outlier_scale
        csc[gi, st["C_outliers"][gi]] = cfg.bc_outlier_scale
    x = np.empty((nb, L, H, P), dt_)
    B = np.empty((nb, L, G, N), dt_)
    C = np.empty((nb, L, G, N), dt_)
    dt = np.empty((nb, L, H), np.float32)
    rows = max(1, (1 << 22) // (H * P))   # tokens per block of x (32 MB of fp64 at a time)
    for b in range(nb):
        # x[b] in consecutive token blocks: the stream yields the same values as one draw of
        # (L, H, P), without the multi-GB fp64 temporaries
        for r0 in range(0, L, rows):
            r1 = min(L, r0 + rows)
            blk = g.standard_normal((r1 - r0, H, P))
            blk *= xsc
            x[b, r0:r1] = blk.astype(dt_)
        B[b] = (g.standard_normal((L, G, N)) * bsc).astype(dt_)
        C[b] = (g.standard_normal((L, G, N)) * csc).astype(dt_)
        dt[b] = g.normal(cfg.dt_mu, cfg.dt_sigma, size=(L, H)).astype(np.float32)
    return {"x": x, "B": B, "C": C, "dt_raw": dt}


def draw(cfg: SSDConfig, stream: int = 1, batch: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Parameters plus one activation draw."""
    out = dict(structure(cfg))
    out.update(activations(cfg, stream, batch))
    return out
