"""Seeded synthetic Q/K/V workloads for Token Radius Attention.

This module only produces inputs.  It holds none of the method's arithmetic
(no scores, softmax, entropy, budget, radius or mask), so both the CPU oracle
and the GPU library can consume what it makes without sharing any code path.

The paper measures on real Wan2.1 / Wan2.2 / HunyuanVideo self-attention
activations (Sec. 4, "Implementation details"); those are not available, so
the workloads below stand in for them with the same shapes:

* a latent grid F x H x W, raster token index i = (f*H + x)*W + y
  (Sec. 2.1: each token carries a coordinate (f, x, y));
* 64 random Fourier features of the normalised coordinate,
  p_i = sqrt(2) * cos(2*pi * Omega c_i + beta), Omega ~ N(0, 2^2), beta ~ U[0, 2*pi);
* per head: Wq, Wk ~ N(0, 1/64) (d x 64), a per-query scale s_i log-uniform on
  [s_min, s_max], eps_q, eps_k, v ~ N(0, 1);
* q_i = s_i * (Wq p_i + 0.5 eps_q),  k_j = Wk p_j + 0.5 eps_k.

The per-query scale spreads the attention temperature, and therefore the
attention entropy, over several nats, which is what drives the per-query
budgets of Sec. 3.1.  Values are rounded once to the workload dtype (fp32, or
bf16 with round-to-nearest-even); the oracle and the kernels see the identical
rounded values.

Joint text-video workloads (Sec. 3.2) append ``text_tokens`` text tokens after
the N video tokens: their 64 features are i.i.d. N(0, 1) (unit variance like the
Fourier features, no spatial structure), with the same per-head projections,
per-query scale and noise; they are drawn after all of the head's video values,
so the video part of a workload does not depend on the text length.

Each head is drawn from its own stream, SeedSequence([seed, head]), so heads can
be generated in parallel and any subset of heads reproduced on its own.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "workload", "generate", "generate_head",
    "bf16_bits_from_f32", "f32_from_bf16_bits", "to_f64", "drift_step",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic self-attention call (batch, heads, grid, dtype, block)."""
    name: str
    batch: int
    heads: int
    head_dim: int
    dtype: str            # "fp32" or "bf16"
    frames: int
    height: int
    width: int
    block: int
    s_min: float
    s_max: float
    gamma: float          # temporal decay rate of the radius (Sec. 3.2)
    tau: float = 0.9      # target attention mass (Sec. 3.1)
    seed: int = 1000
    tile_h: int = 8
    tile_w: int = 8
    text_tokens: int = 0  # joint text-video attention: text tokens after the video

    @property
    def n_video(self) -> int:
        return self.frames * self.height * self.width

    @property
    def n_tokens(self) -> int:
        return self.n_video + self.text_tokens

    @property
    def n_blocks(self) -> int:
        return -(-self.n_tokens // self.block)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads: a tiny grid the oracle handles densely, three
# model-shaped video self-attention calls, and the warm-up reuse sequence.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 2, 64, "fp32", 4, 8, 8, 64, 0.25, 4.0, 0.6,
                     seed=1000, tile_h=8, tile_w=8),
    "wan13b_480p": Workload("wan13b_480p", 1, 12, 128, "bf16", 21, 30, 52, 128,
                            0.25, 4.0, 0.6, seed=1001, tile_h=8, tile_w=16),
    "wan14b_720p": Workload("wan14b_720p", 1, 40, 128, "bf16", 21, 45, 80, 128,
                            0.25, 4.0, 0.6, seed=1002, tile_h=8, tile_w=16),
    "hunyuan_720p": Workload("hunyuan_720p", 1, 24, 128, "bf16", 33, 45, 80, 128,
                             0.1, 8.0, 0.95, seed=1003, tile_h=8, tile_w=16),
    "reuse_480p": Workload("reuse_480p", 1, 12, 128, "bf16", 21, 30, 52, 128,
                           0.25, 4.0, 0.6, seed=1004, tile_h=8, tile_w=16),
    # joint text-video attention at the HunyuanVideo 720p shape with 256 text
    # tokens (the paper gives no text length; 256 is a text-encoder length)
    "hunyuan_joint_720p": Workload("hunyuan_joint_720p", 1, 24, 128, "bf16", 33, 45, 80, 128,
                                   0.1, 8.0, 0.95, seed=1005, tile_h=8, tile_w=16,
                                   text_tokens=256),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------- dtype helpers
def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); uint16 bits."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of a stored workload array (bf16 bits or fp32)."""
    if dtype == "bf16":
        return f32_from_bf16_bits(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


# ---------------------------------------------------------------- generator
def _features(w: Workload) -> np.ndarray:
    """Random Fourier features p (N x 64) of the normalised coordinates,
    evaluated in fp64 and stored as fp32."""
    rng = np.random.default_rng(np.random.SeedSequence([w.seed]))
    omega = rng.normal(0.0, 2.0, size=(64, 3))
    beta = rng.uniform(0.0, 2.0 * np.pi, size=64)
    f, x, y = np.meshgrid(np.arange(w.frames), np.arange(w.height),
                          np.arange(w.width), indexing="ij")
    c = np.stack([(f.ravel() + 0.5) / w.frames, (x.ravel() + 0.5) / w.height,
                  (y.ravel() + 0.5) / w.width], axis=1)
    return (np.sqrt(2.0) * np.cos(2.0 * np.pi * (c @ omega.T) + beta)).astype(np.float32)


def generate_head(w: Workload, batch_index: int, head: int, feats=None,
                  masters: bool = False):
    """q, k, v of one (batch, head) as stored arrays of shape (N, d).

    With ``masters=True`` the fp32 values before the final dtype rounding are
    returned as well (used by the drifting reuse sequence)."""
    if feats is None:
        feats = _features(w)
    n, d = w.n_video, w.head_dim
    rng = np.random.default_rng(np.random.SeedSequence([w.seed, batch_index, head]))
    wq = rng.normal(0.0, 0.125, size=(d, 64)).astype(np.float32)
    wk = rng.normal(0.0, 0.125, size=(d, 64)).astype(np.float32)
    s = np.exp(rng.uniform(np.log(w.s_min), np.log(w.s_max), size=n)).astype(np.float32)
    q = rng.standard_normal((n, d), dtype=np.float32)     # eps_q
    k = rng.standard_normal((n, d), dtype=np.float32)     # eps_k
    v = rng.standard_normal((n, d), dtype=np.float32)
    q *= 0.5
    q += feats @ wq.T
    q *= s[:, None]
    k *= 0.5
    k += feats @ wk.T
    if w.text_tokens:
        t = w.text_tokens
        pt = rng.standard_normal((t, 64), dtype=np.float32)
        st = np.exp(rng.uniform(np.log(w.s_min), np.log(w.s_max), size=t)).astype(np.float32)
        qt = rng.standard_normal((t, d), dtype=np.float32)
        kt = rng.standard_normal((t, d), dtype=np.float32)
        vt = rng.standard_normal((t, d), dtype=np.float32)
        qt *= 0.5
        qt += pt @ wq.T
        qt *= st[:, None]
        kt *= 0.5
        kt += pt @ wk.T
        q, k, v = (np.concatenate([a, b]) for a, b in ((q, qt), (k, kt), (v, vt)))
    out = tuple(bf16_bits_from_f32(a) if w.dtype == "bf16" else a for a in (q, k, v))
    if masters:
        return out, (q, k)
    return out


def _workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def generate(w: Workload, heads=None, batch=None):
    """Stored q, k, v arrays of shape (B, Ha, N, d) for the listed heads.

    bf16 workloads come back as uint16 bit patterns, fp32 ones as float32."""
    heads = list(range(w.heads)) if heads is None else list(heads)
    batches = list(range(w.batch)) if batch is None else list(batch)
    n, d = w.n_tokens, w.head_dim
    dt = np.uint16 if w.dtype == "bf16" else np.float32
    q = np.empty((len(batches), len(heads), n, d), dtype=dt)
    k = np.empty_like(q)
    v = np.empty_like(q)
    feats = _features(w)

    def one(job):
        bi, hi = job
        qq, kk, vv = generate_head(w, batches[bi], heads[hi], feats)
        q[bi, hi], k[bi, hi], v[bi, hi] = qq, kk, vv

    jobs = [(bi, hi) for bi in range(len(batches)) for hi in range(len(heads))]
    with ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(one, jobs))
    return q, k, v


def drift_step(master: np.ndarray, rng: np.random.Generator, dtype: str, scale=0.02):
    """One denoising-step drift of an fp32 master copy: x <- x + scale*N(0,1).

    Updates ``master`` in place and returns the re-rounded stored array."""
    master += scale * rng.standard_normal(master.shape, dtype=np.float32)
    return bf16_bits_from_f32(master) if dtype == "bf16" else master.copy()
