"""Seeded synthetic workloads for the VSA2 routed sparse-attention path.

This module only describes problem shapes and draws inputs.  It holds none of
the method's arithmetic (no pooling, scoring, selection or attention), so both
the HIP path and the CPU oracle may take their inputs from it.

The paper trains on VAE video latents that are not available here; these
seeded tensors stand in for them.  Recipe (per tensor X in {Q, K, V} and per
(batch, head of that tensor, cube)):

    X[token] = mu[cube] + 0.5 * eps[token],   eps ~ N(0, 1) iid per element,
    mu[cube] ~ N(0, I_D)                       (independent per tensor),
    mu[cube] *= exp(xi[cube]), xi ~ N(0, 1)    (log-normal cube norms, "skewed"),

so tokens of one cube share a mean and routing has signal.  dO ~ N(0, 1).
All draws are float32, then rounded to the problem dtype (bf16 with
round-to-nearest-even); the rounded values are the inputs of both sides.
Tensors are produced directly in cube-major order [batch, head, L, D],
L = N * B (every per-element draw is iid, so drawing in cube-major order is
the same distribution as drawing in raster order and permuting).

Streams: every (tensor, batch, head) slab has its own generator,
numpy PCG64 seeded with SeedSequence([base_seed, tensor_id, b, h]), so the
result does not depend on the thread count that draws it.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

F32, BF16 = 0, 1
DTYPE_NAMES = {F32: "f32", BF16: "bf16"}


@dataclasses.dataclass(frozen=True)
class Problem:
    """Shape of one routed sparse-attention call (notation of the paper's
    Table 1: grid T x H x W, cube B = Bt*Bh*Bw, router pool R = Rt*Rh*Rw)."""
    batch: int
    heads_q: int
    heads_kv: int
    head_dim: int
    T: int
    H: int
    W: int
    Bt: int = 4
    Bh: int = 4
    Bw: int = 4
    Rt: int = 2
    Rh: int = 2
    Rw: int = 2
    dtype: int = BF16
    text_len: int = 0          # text tokens joined to the video (MMDiT), 0 = none

    @property
    def L(self) -> int:
        """Video tokens in the cube-major layout, padding included."""
        return self.N * self.B

    @property
    def M(self) -> int:
        """Text blocks of B tokens (the last one padded)."""
        return -(-self.text_len // self.B)

    @property
    def N_joint(self) -> int:
        """Blocks of one (batch, head) sequence: N video cubes, then M text blocks."""
        return self.N + self.M

    @property
    def L_joint(self) -> int:
        """Tokens of one (batch, head) sequence: video, then text, padding included."""
        return self.N_joint * self.B

    @property
    def B(self) -> int:
        return self.Bt * self.Bh * self.Bw

    @property
    def N(self) -> int:
        return self.Nt * self.Nh * self.Nw

    @property
    def Nt(self) -> int:
        return -(-self.T // self.Bt)

    @property
    def Nh(self) -> int:
        return -(-self.H // self.Bh)

    @property
    def Nw(self) -> int:
        return -(-self.W // self.Bw)

    @property
    def padded(self) -> bool:
        return bool(self.T % self.Bt or self.H % self.Bh or self.W % self.Bw)

    def token_real(self) -> np.ndarray:
        """bool [L_joint]: token of the sequence that is not padding: a video
        token inside the real T x H x W grid (a grid not divisible by the cube
        is padded up, Sec. 2.2), or one of the first text_len text tokens."""
        n = np.arange(self.N)[:, None]
        beta = np.arange(self.B)[None, :]
        nt, nh, nw = n // (self.Nh * self.Nw), (n // self.Nw) % self.Nh, n % self.Nw
        bt, bh, bw = beta // (self.Bh * self.Bw), (beta // self.Bw) % self.Bh, beta % self.Bw
        video = ((nt * self.Bt + bt < self.T) & (nh * self.Bh + bh < self.H) &
                 (nw * self.Bw + bw < self.W)).reshape(-1)
        return np.concatenate([video, np.arange(self.M * self.B) < self.text_len])

    @property
    def R(self) -> int:
        return self.Rt * self.Rh * self.Rw

    @property
    def G(self) -> int:
        return (self.Bt // self.Rt) * (self.Bh // self.Rh) * (self.Bw // self.Rw)

    def replace(self, **kw) -> "Problem":
        return dataclasses.replace(self, **kw)


@dataclasses.dataclass(frozen=True)
class Selection:
    """Selection rule: mode 0 = top-k per query block, 1 = smallest prefix
    reaching `mass` of the row's score total, capped at `cap` blocks, 2 =
    the N*k best pairs of each (batch, head)'s whole N x N map."""
    mode: int = 0
    k: int = 8
    mass: float = 0.9
    cap: int = 0


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    problem: Problem
    select: Selection
    seed: int
    skewed: bool = False       # log-normal cube-mean norms
    backward: bool = True


# Workload shapes: tiny, 480p, 720p, 720p with mass selection, long-clip GQA;
# 720p-seq and 720p-vsa reuse the 720p inputs under the per-sequence rule and
# under the coarse (R = B) router.
WORKLOADS = {
    "tiny": Workload(
        "tiny", Problem(1, 2, 2, 64, 8, 16, 16, dtype=F32), Selection(0, 8), 1000,
        backward=False),
    "480p": Workload(
        "480p", Problem(1, 12, 12, 128, 20, 32, 56), Selection(0, 70), 1001),
    "720p": Workload(
        "720p", Problem(1, 40, 40, 128, 20, 48, 80), Selection(0, 120), 1002),
    "720p-mass": Workload(
        "720p-mass", Problem(1, 40, 40, 128, 20, 48, 80), Selection(1, 0, 0.9, 240), 1003,
        skewed=True),
    "gqa-long": Workload(
        "gqa-long", Problem(1, 40, 8, 128, 40, 48, 80), Selection(0, 120), 1004),
    # the paper's own rule, TopK_{N k} per (batch, head), on the 720p inputs
    "720p-seq": Workload(
        "720p-seq", Problem(1, 40, 40, 128, 20, 48, 80), Selection(2, 120), 1002),
    # the coarse cube-level router of VSA (router pool R = B, G = 1) on the 720p inputs
    "720p-vsa": Workload(
        "720p-vsa", Problem(1, 40, 40, 128, 20, 48, 80, Rt=4, Rh=4, Rw=4), Selection(0, 120), 1002),
    # the latent grid of an 81-frame 1280x720 clip itself (21 x 45 x 80: 4x
    # temporal, 16x spatial compression), not a multiple of the cube: padded
    # to 24 x 48 x 80, N = 1440 cubes, top-120
    "720p-latent": Workload(
        "720p-latent", Problem(1, 40, 40, 128, 21, 45, 80), Selection(0, 120), 1005),
    # the 720p grid joined by 512 text tokens (MMDiT joint attention: every
    # video block also attends to the 8 text blocks, text attends to all)
    "720p-text": Workload(
        "720p-text", Problem(1, 40, 40, 128, 20, 48, 80, text_len=512), Selection(0, 120), 1006),
}


def round_bf16_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even), returned as
    float32 holding the rounded values.  Input preparation only."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    # keep NaN/inf patterns untouched (not produced by these generators)
    special = (u & np.uint32(0x7F800000)) == np.uint32(0x7F800000)
    rounded = np.where(special, u & np.uint32(0xFFFF0000), rounded)
    return rounded.view(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16-representable."""
    return (np.ascontiguousarray(x, dtype=np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _slab(seed: int, tensor_id: int, b: int, h: int, N: int, B: int, D: int,
          with_mean: bool, skewed: bool, out: np.ndarray) -> None:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id, b, h])))
    if with_mean:
        mu = rng.standard_normal((N, D), dtype=np.float32)
        if skewed:
            xi = rng.standard_normal((N, 1), dtype=np.float32)
            mu *= np.exp(xi)
        eps = rng.standard_normal((N, B, D), dtype=np.float32)
        eps *= np.float32(0.5)
        eps += mu[:, None, :]
        out[...] = eps.reshape(N * B, D)
    else:
        out[...] = rng.standard_normal((N * B, D), dtype=np.float32)


def make_tensor(p: Problem, seed: int, tensor_id: int, heads: int, with_mean: bool = True,
                skewed: bool = False, threads: int | None = None) -> np.ndarray:
    """One [batch, heads, L_joint, D] float32 tensor of the recipe above,
    rounded to the problem dtype: the video tokens, then (text_len > 0) the
    text tokens, N(0,1) from a stream of their own.  tensor_id: 0 = Q, 1 = K,
    2 = V, 3 = dO."""
    out = np.empty((p.batch, heads, p.L_joint, p.head_dim), dtype=np.float32)
    jobs = [(b, h) for b in range(p.batch) for h in range(heads)]
    nthr = threads or min(16, os.cpu_count() or 1)

    real = p.token_real() if (p.padded or p.text_len % p.B) else None

    def work(bh):
        b, h = bh
        _slab(seed, tensor_id, b, h, p.N, p.B, p.head_dim, with_mean, skewed, out[b, h, :p.L])
        if p.M:
            rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id, b, h, 1])))
            out[b, h, p.L:] = rng.standard_normal((p.M * p.B, p.head_dim), dtype=np.float32)
        if p.dtype == BF16:
            out[b, h] = round_bf16_f32(out[b, h])
        if real is not None:
            out[b, h][~real] = 0.0          # padding tokens hold zeros

    if nthr > 1 and len(jobs) > 1:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(work, jobs))
    else:
        for j in jobs:
            work(j)
    return out


def make_inputs(w: Workload, with_grad: bool | None = None, threads: int | None = None,
                shared_mean: bool = False) -> dict:
    """Q, K, V (and dO when the workload has a backward pass) for workload w.

    shared_mean=True gives Q, K and V of a head the same cube means (one draw,
    the K/V heads of a GQA group take their first query head's means); then
    every query block's own cube is its best match, which makes a cheap router
    sanity check."""
    p = w.problem
    q = make_tensor(p, w.seed, 0, p.heads_q, True, w.skewed, threads)
    if shared_mean:
        if p.heads_q != p.heads_kv or w.skewed:
            raise ValueError("shared_mean needs heads_q == heads_kv and unskewed means")
        k = _with_means_of(q, p, w.seed, 1, threads)
        v = _with_means_of(q, p, w.seed, 2, threads)
    else:
        k = make_tensor(p, w.seed, 1, p.heads_kv, True, w.skewed, threads)
        v = make_tensor(p, w.seed, 2, p.heads_kv, True, w.skewed, threads)
    out = {"q": q, "k": k, "v": v}
    if with_grad if with_grad is not None else w.backward:
        out["do"] = make_tensor(p, w.seed, 3, p.heads_q, False, False, threads)
    return out


def _with_means_of(ref: np.ndarray, p: Problem, seed: int, tensor_id: int, threads) -> np.ndarray:
    """Tensor whose cube means are those of `ref` (up to its noise), fresh
    0.5*N(0,1) token noise.  The cube mean is recovered exactly from ref's
    generator stream, not estimated."""
    out = np.empty_like(ref)
    for b in range(p.batch):
        for h in range(ref.shape[1]):
            rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 0, b, h])))
            mu = rng.standard_normal((p.N, p.head_dim), dtype=np.float32)
            rng2 = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id, b, h])))
            eps = rng2.standard_normal((p.N, p.B, p.head_dim), dtype=np.float32) * np.float32(0.5)
            x = (eps + mu[:, None, :]).reshape(p.L, p.head_dim)
            if p.text_len:
                raise ValueError("shared_mean inputs have no text tokens")
            out[b, h] = round_bf16_f32(x) if p.dtype == BF16 else x
            if p.padded:
                out[b, h][~p.token_real()] = 0.0        # padding tokens hold zeros
    return out


def raster_to_cube_major(x: np.ndarray, p: Problem) -> np.ndarray:
    """[..., T*H*W (raster, w fastest), D] -> [..., N*B (cube-major), D]; a grid
    not divisible by the cube is padded up with zero tokens."""
    lead = x.shape[:-2]
    D = x.shape[-1]
    Nt, Nh, Nw = p.Nt, p.Nh, p.Nw
    g = x.reshape(*lead, p.T, p.H, p.W, D)
    if p.padded:
        pad = [(0, 0)] * len(lead) + [(0, Nt * p.Bt - p.T), (0, Nh * p.Bh - p.H), (0, Nw * p.Bw - p.W), (0, 0)]
        g = np.pad(g, pad)
    y = g.reshape(*lead, Nt, p.Bt, Nh, p.Bh, Nw, p.Bw, D)
    nd = len(lead)
    perm = list(range(nd)) + [nd + 0, nd + 2, nd + 4, nd + 1, nd + 3, nd + 5, nd + 6]
    return np.ascontiguousarray(y.transpose(perm)).reshape(*lead, p.L, D)


def cube_major_to_raster(x: np.ndarray, p: Problem) -> np.ndarray:
    """Inverse of raster_to_cube_major (padding tokens dropped)."""
    lead = x.shape[:-2]
    D = x.shape[-1]
    Nt, Nh, Nw = p.Nt, p.Nh, p.Nw
    y = x.reshape(*lead, Nt, Nh, Nw, p.Bt, p.Bh, p.Bw, D)
    nd = len(lead)
    perm = list(range(nd)) + [nd + 0, nd + 3, nd + 1, nd + 4, nd + 2, nd + 5, nd + 6]
    g = np.ascontiguousarray(y.transpose(perm)).reshape(*lead, Nt * p.Bt, Nh * p.Bh, Nw * p.Bw, D)
    return np.ascontiguousarray(g[..., :p.T, :p.H, :p.W, :]).reshape(*lead, p.T * p.H * p.W, D)
