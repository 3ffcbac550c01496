"""Seeded synthetic inputs for the QuantEase hot path.

Shared by the tests, the smoke check and the benchmark, for both the HIP
library and the CPU oracle.  It draws random numbers and shapes them like the
paper's workloads; it contains none of the method's arithmetic (no Gram
matrix, no grid, no quantization).

The paper calibrates on 128 sequences x 2048 tokens of C4 pushed through OPT,
BLOOM and Falcon layers (Sec. 5, experimental set-up); neither the dataset nor
the weights exist here, so these generators stand in for them with layers of
the same shapes: Gaussian weights with a sprinkle of large entries, and
heavy-tailed (Student-t, nu = 4) activations with a few outlier channels.

Seeding: every draw comes from ``numpy.random.Generator(PCG64(SeedSequence(
[1885, cfg, stream, chunk])))``.  Streams: 0 weight values, 1 weight outlier
positions, 2 activation outlier channels, 3 activation values (one chunk =
2048 tokens, so any chunk can be regenerated alone), 4 oracle row sample,
5 Gram entry sample, 6 free-form test inputs, 7 device-drawn activations.
Draws are fp64, cast to fp32.

The Falcon-180B-shaped layer needs 59392 x 262144 activations (62 GB); the
host generator would take the better part of an hour for them, so
``activation_chunk_device`` draws such chunks on the GPU with torch's seeded
Philox generator (same t4 law: Z / sqrt(chi2_4 / 4), chi2_4 the sum of four
squared standard normals).  Tests copy the channels the oracle needs back to
the host, so both sides still see identical numbers.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Optional

import numpy as np

SEED = 1885
CHUNK_TOKENS = 2048


def rng(cfg: int, stream: int, chunk: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED, cfg, stream, chunk])))


@dataclass(frozen=True)
class LayerSpec:
    """One synthetic linear layer: W is q x p, X is p x n."""
    name: str
    cfg: int                 # seed id
    q: int
    p: int
    n: int
    bits: int
    sweeps: int
    w_std: float = 0.02
    w_out_frac: float = 0.0  # fraction of weight entries scaled by w_out_mult
    w_out_mult: float = 10.0
    x_dist: str = "normal"   # "normal" or "t4"
    x_out_count: int = 0     # number of activation outlier channels
    x_out_mult: float = 1.0
    damp: float = 0.01       # relative diagonal damping of Sigma
    s_frac: float = 0.0      # outlier budget s = floor(s_frac * q * p) (outlier-aware variant)
    x_cfg: Optional[int] = None   # seed id of the activations when shared with another layer

    @property
    def s_budget(self) -> int:
        return int(self.s_frac * self.q * self.p)


# Layer shapes of the paper's workloads (OPT / Falcon-sized linear layers,
# 128 x 2048 calibration tokens).
CONFIGS = {
    # small single layer: full oracle runs in seconds
    "c1": LayerSpec("c1_512x512_4bit", 1, 512, 512, 2048, 4, 5, w_std=0.02,
                    x_dist="normal", x_out_count=10, x_out_mult=20.0),
    # attention projection 4096 x 4096, 4-bit: the headline workload
    "c2": LayerSpec("c2_attn_4096x4096_4bit", 2, 4096, 4096, 128 * 2048, 4, 10,
                    w_std=0.02, w_out_frac=0.001, w_out_mult=10.0,
                    x_dist="t4", x_out_count=41, x_out_mult=30.0),
    # MLP up / down projections, 3-bit
    "c3up": LayerSpec("c3_up_11008x4096_3bit", 3, 11008, 4096, 128 * 2048, 3, 10,
                      w_std=0.02, w_out_frac=0.001, w_out_mult=10.0,
                      x_dist="t4", x_out_count=41, x_out_mult=30.0, x_cfg=2),
    "c3down": LayerSpec("c3_down_4096x11008_3bit", 4, 4096, 11008, 128 * 2048, 3, 10,
                        w_std=0.02, w_out_frac=0.001, w_out_mult=10.0,
                        x_dist="t4", x_out_count=110, x_out_mult=30.0),
    # outlier-aware variant on the attention projection, 3-bit, 1% outliers
    "c4": LayerSpec("c4_outlier_4096x4096_3bit_1pct", 2, 4096, 4096, 128 * 2048, 3, 10,
                    w_std=0.02, w_out_frac=0.001, w_out_mult=10.0,
                    x_dist="t4", x_out_count=41, x_out_mult=30.0, s_frac=0.01),
    # Falcon-180B MLP down-projection
    "c5": LayerSpec("c5_falcon180b_down_14848x59392_4bit", 5, 14848, 59392, 128 * 2048, 4, 5,
                    w_std=0.015, x_dist="t4"),
}


def weights(spec: LayerSpec, q: Optional[int] = None, p: Optional[int] = None) -> np.ndarray:
    """W ~ N(0, w_std^2), with round(w_out_frac * q * p) entries (uniform
    positions, without replacement) multiplied by w_out_mult.  fp32."""
    q = spec.q if q is None else q
    p = spec.p if p is None else p
    W = rng(spec.cfg, 0).normal(0.0, spec.w_std, size=(q, p))
    n_out = int(round(spec.w_out_frac * q * p))
    if n_out > 0:
        pos = rng(spec.cfg, 1).choice(q * p, size=n_out, replace=False)
        W.reshape(-1)[pos] *= spec.w_out_mult
    return W.astype(np.float32)


def outlier_channels(spec: LayerSpec, p: Optional[int] = None) -> np.ndarray:
    p = spec.p if p is None else p
    if spec.x_out_count <= 0:
        return np.zeros(0, np.int64)
    cfg = spec.cfg if spec.x_cfg is None else spec.x_cfg
    count = min(spec.x_out_count, p)
    return np.sort(rng(cfg, 2).choice(p, size=count, replace=False)).astype(np.int64)


def activation_chunk(spec: LayerSpec, chunk: int, p: Optional[int] = None,
                     tokens: int = CHUNK_TOKENS) -> np.ndarray:
    """Tokens [chunk*2048, chunk*2048 + tokens) of X (p x tokens, fp32)."""
    p = spec.p if p is None else p
    cfg = spec.cfg if spec.x_cfg is None else spec.x_cfg
    g = rng(cfg, 3, chunk)
    if spec.x_dist == "t4":
        x = g.standard_t(4.0, size=(p, tokens))
    elif spec.x_dist == "normal":
        x = g.standard_normal(size=(p, tokens))
    else:
        raise ValueError(spec.x_dist)
    ch = outlier_channels(spec, p)
    if ch.size:
        x[ch, :] *= spec.x_out_mult
    return x.astype(np.float32)


def activations(spec: LayerSpec, n: Optional[int] = None, p: Optional[int] = None,
                threads: Optional[int] = None, out: Optional[np.ndarray] = None) -> np.ndarray:
    """X (p x n, fp32, channel-major) assembled from 2048-token chunks, drawn
    in parallel threads (numpy releases the GIL while drawing)."""
    p = spec.p if p is None else p
    n = spec.n if n is None else n
    if out is None:
        out = np.empty((p, n), dtype=np.float32)
    nchunks = (n + CHUNK_TOKENS - 1) // CHUNK_TOKENS
    if threads is None:
        threads = min(16, len(os.sched_getaffinity(0)))

    def fill(c):
        t0 = c * CHUNK_TOKENS
        t1 = min(n, t0 + CHUNK_TOKENS)
        out[:, t0:t1] = activation_chunk(spec, c, p, t1 - t0)

    if threads <= 1 or nchunks == 1:
        for c in range(nchunks):
            fill(c)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(fill, range(nchunks)))
    return out


def activation_chunk_device(spec: LayerSpec, chunk: int, tokens: int, device,
                            p: Optional[int] = None):
    """Chunk `chunk` of a device-drawn X stream (p x tokens, fp32, on
    `device`): t4 values (or N(0, 1)), outlier channels scaled as in
    activation_chunk.  Seeded from SeedSequence([1885, cfg, 7, chunk])."""
    import torch
    p = spec.p if p is None else p
    cfg = spec.cfg if spec.x_cfg is None else spec.x_cfg
    seed = int(np.random.SeedSequence([SEED, cfg, 7, chunk]).generate_state(1, np.uint64)[0])
    g = torch.Generator(device=device)
    g.manual_seed(seed & ((1 << 63) - 1))
    x = torch.randn((p, tokens), generator=g, device=device, dtype=torch.float32)
    if spec.x_dist == "t4":
        chi2 = torch.zeros_like(x)
        for _ in range(4):
            z = torch.randn((p, tokens), generator=g, device=device, dtype=torch.float32)
            chi2.addcmul_(z, z)
        x.div_(torch.sqrt(chi2 * 0.25))
    elif spec.x_dist != "normal":
        raise ValueError(spec.x_dist)
    ch = outlier_channels(spec, p)
    if ch.size:
        x[torch.as_tensor(ch, device=device)] *= spec.x_out_mult
    return x


def correlated_activations(p: int, n: int, rho: float, seed: int,
                           out_channels: int = 0, out_mult: float = 1.0) -> np.ndarray:
    """AR(1) across channels: x_0 = e_0, x_a = rho x_{a-1} + sqrt(1 - rho^2) e_a,
    e ~ N(0, 1).  Real activations are strongly correlated across channels; an
    i.i.d. X gives a nearly diagonal Sigma, which barely exercises CD.  fp32."""
    g = rng(100 + seed, 6)
    e = g.standard_normal(size=(p, n))
    x = np.empty_like(e)
    x[0] = e[0]
    c = np.sqrt(1.0 - rho * rho)
    for a in range(1, p):
        x[a] = rho * x[a - 1] + c * e[a]
    if out_channels > 0:
        ch = g.choice(p, size=out_channels, replace=False)
        x[ch, :] *= out_mult
    return x.astype(np.float32)


def gaussian(shape, seed: int, std: float = 1.0) -> np.ndarray:
    """Free-form N(0, std^2) test input, fp32."""
    return (rng(200 + seed, 6).standard_normal(size=shape) * std).astype(np.float32)


def uniform(shape, seed: int, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    """Free-form U(lo, hi) test input, fp32."""
    return rng(300 + seed, 6).uniform(lo, hi, size=shape).astype(np.float32)


def integers(shape, seed: int, lo: int, hi: int) -> np.ndarray:
    """Free-form integers in [lo, hi), int64."""
    return rng(400 + seed, 6).integers(lo, hi, size=shape, dtype=np.int64)


def row_sample(q: int, r: int, cfg: int) -> np.ndarray:
    """Sorted seeded sample of r distinct rows out of q (stream 4)."""
    r = min(r, q)
    return np.sort(rng(cfg, 4).choice(q, size=r, replace=False)).astype(np.int64)


def entry_sample(p: int, m: int, cfg: int, must: Optional[np.ndarray] = None):
    """Seeded m x m index grid of Sigma entries (stream 5); the indices in
    ``must`` (e.g. outlier channels) are always included."""
    g = rng(cfg, 5)
    base = g.choice(p, size=min(m, p), replace=False)
    if must is not None and len(must):
        base = np.unique(np.concatenate([np.asarray(must, np.int64), base]))[:max(m, len(must))]
    idx = np.sort(np.unique(base)).astype(np.int64)
    return idx
