"""Seeded synthetic inputs for the Ball Sparse Attention hot path.

The workloads stand in for the paper's airflow-pressure task (ShapeNet-Car surfaces of
3586 points, Section 3.1) and for its sequence-length sweep (Fig. 2). No dataset is read:
every tensor is drawn from a numpy ``default_rng`` stream, one independent stream per
tensor, spawned from ``SeedSequence(seed)``.

Everything here is input preparation: point clouds, per-point Q/K/V features, gate logits
(the caller's linear projection), compression-MLP weights and the upstream gradient. None
of the attention method's own arithmetic lives here.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

__all__ = ["Config", "CONFIGS", "make_points", "make_inputs", "make_block_inputs", "round_bf16", "bf16_bits",
           "HeadInputs"]


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    batch: int
    n_real: int          # real points per cloud
    n_pad: int           # tokens per cloud after padding (power of two)
    heads: int
    head_dim: int
    dtype: str           # "f32" or "bf16": storage type of Q/K/V/O
    ball: int            # m
    cmp_block: int       # l (compression block length)
    cmp_stride: int      # compression stride (equal to l)
    slc_block: int       # l' (selection block length)
    topk: int            # k*
    group: int           # g (query group size)
    cloud: str           # point-cloud generator
    passes: str          # "fwd" or "fwdbwd"

    @property
    def channels(self) -> int:
        return self.heads * self.head_dim


CONFIGS = {
    # Tiny fp32 forward: 1024 uniform points.
    1: Config("tiny_fp32", 1, 1024, 1024, 4, 32, "f32", 64, 8, 8, 16, 4, 8, "uniform", "fwd"),
    # Airflow-surface-like: 16 perturbed ellipsoids of 3586 points padded to 4096.
    2: Config("airflow_bf16", 16, 3586, 4096, 8, 32, "bf16", 256, 8, 8, 16, 8, 8, "ellipsoid", "fwd"),
    # Scaling: one 65536-point Gaussian-mixture cloud, forward + backward.
    3: Config("scaling_65536", 1, 65536, 65536, 8, 64, "bf16", 256, 16, 16, 32, 16, 16, "gmm", "fwdbwd"),
    # Large: one 2^20-point anisotropic Gaussian-mixture cloud, forward.
    4: Config("large_1m", 1, 1 << 20, 1 << 20, 16, 64, "bf16", 512, 32, 32, 64, 16, 32, "aniso_gmm", "fwd"),
    # Backward-heavy: the airflow shapes, forward + backward.
    5: Config("airflow_bwd", 16, 3586, 4096, 8, 32, "bf16", 256, 8, 8, 16, 8, 8, "ellipsoid", "fwdbwd"),
}


def round_bf16(x: np.ndarray, chunk: int = 1 << 22) -> np.ndarray:
    """Round finite float32 values to the nearest bfloat16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    src = x.reshape(-1).view(np.uint32)
    dst = out.reshape(-1).view(np.uint32)
    for s in range(0, src.size, chunk):
        u = src[s:s + chunk]
        # finite values stay below 0xFF800000, so the carry cannot wrap 32 bits
        dst[s:s + chunk] = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16)) \
            << np.uint32(16)
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of bf16-representable float32 values (the bf16 storage pattern)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def _streams(seed: int, n: int):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def _real_sph_harm(l: int, m: int, theta: np.ndarray, phi: np.ndarray) -> np.ndarray:
    from scipy.special import sph_harm_y
    if m == 0:
        return np.real(sph_harm_y(l, 0, theta, phi))
    y = sph_harm_y(l, abs(m), theta, phi)
    return math.sqrt(2.0) * (np.real(y) if m > 0 else np.imag(y))


def _ellipsoid_cloud(rng, n: int) -> np.ndarray:
    z = rng.standard_normal((n, 3))
    u = z / np.linalg.norm(z, axis=1, keepdims=True)
    theta = np.arccos(np.clip(u[:, 2], -1.0, 1.0))
    phi = np.arctan2(u[:, 1], u[:, 0])
    f = np.zeros(n)
    for l in range(1, 7):
        for m in range(-l, l + 1):
            f += rng.standard_normal() * _real_sph_harm(l, m, theta, phi)
    r = 1.0 + 0.05 * f / np.max(np.abs(f))
    return np.array([2.0, 0.8, 0.6]) * u * r[:, None]


def _gmm_cloud(rng, n: int, comps: int = 32, sigma: float = 0.05) -> np.ndarray:
    means = rng.uniform(0.0, 1.0, (comps, 3))
    lab = rng.integers(0, comps, n)
    return means[lab] + sigma * rng.standard_normal((n, 3))


def _haar_rotation(rng) -> np.ndarray:
    a = rng.standard_normal((3, 3))
    qm, rm = np.linalg.qr(a)
    return qm * np.sign(np.diag(rm))[None, :]


def _aniso_gmm_cloud(rng, n: int, comps: int = 64) -> np.ndarray:
    means = rng.uniform(0.0, 1.0, (comps, 3))
    rots = np.stack([_haar_rotation(rng) for _ in range(comps)])
    sig = rng.uniform(0.01, 0.1, (comps, 3))
    out = np.empty((0, 3))
    while out.shape[0] < n:
        need = n - out.shape[0]
        lab = rng.integers(0, comps, need)
        z = rng.standard_normal((need, 3)) * sig[lab]
        x = means[lab] + np.einsum("nij,nj->ni", rots[lab], z)
        keep = np.all((x >= 0.0) & (x <= 1.0), axis=1)
        out = np.concatenate([out, x[keep]])
    return out[:n]


def make_points(cfg: Config, seed: int | None = None) -> np.ndarray:
    """Point clouds [batch, n_real, 3] float32."""
    seed = _default_seed(cfg, seed)
    rngs = _streams(seed * 1000 + 1, cfg.batch)
    clouds = []
    for b in range(cfg.batch):
        rng = rngs[b]
        if cfg.cloud == "uniform":
            c = rng.uniform(0.0, 1.0, (cfg.n_real, 3))
        elif cfg.cloud == "ellipsoid":
            c = _ellipsoid_cloud(rng, cfg.n_real)
        elif cfg.cloud == "gmm":
            c = _gmm_cloud(rng, cfg.n_real)
        elif cfg.cloud == "aniso_gmm":
            c = _aniso_gmm_cloud(rng, cfg.n_real)
        else:
            raise ValueError(cfg.cloud)
        clouds.append(c.astype(np.float32))
    return np.stack(clouds)


def _default_seed(cfg: Config, seed):
    if seed is not None:
        return int(seed)
    for k, c in CONFIGS.items():
        if c == cfg:
            return k
    return 0


def _normal(rng, shape, scale=1.0, chunk=1 << 24) -> np.ndarray:
    out = np.empty(shape, np.float32)
    flat = out.reshape(-1)
    for s in range(0, flat.size, chunk):
        e = min(flat.size, s + chunk)
        flat[s:e] = rng.standard_normal(e - s, dtype=np.float32) * np.float32(scale)
    return out


def _mlp_weights(rr, ld: int, d: int, rnd) -> dict:
    """One compression / coarsening MLP ld -> d -> d, entries N(0, 0.02^2)."""
    return {
        "w1": rnd((rr.standard_normal((ld, d)) * 0.02).astype(np.float32)),
        "b1": rnd((rr.standard_normal(d) * 0.02).astype(np.float32)),
        "w2": rnd((rr.standard_normal((d, d)) * 0.02).astype(np.float32)),
        "b2": rnd((rr.standard_normal(d) * 0.02).astype(np.float32)),
    }


def make_inputs(cfg: Config, seed: int | None = None, *, layout: str = "ball",
                with_grad: bool | None = None) -> dict:
    """Seeded layer inputs.

    layout="ball": Q/K/V as [B, H, n_pad, d] over token slots (what the attention layer
    consumes after ordering); gate logits [B, n_pad, 3]. Rows of dummy slots hold random
    values too: the layer must ignore them.
    layout="points": Q/K/V as [B, n_real, H*d] per real point (before ordering); gate
    logits [B, n_real, 3].

    Values are float32; for bf16 configs they are bf16-representable, as are the MLP
    weights, so both sides of a comparison consume identical numbers.
    """
    seed = _default_seed(cfg, seed)
    B, H, d = cfg.batch, cfg.heads, cfg.head_dim
    rows = cfg.n_pad if layout == "ball" else cfg.n_real
    if with_grad is None:
        with_grad = cfg.passes == "fwdbwd"
    r = _streams(seed * 1000 + 2, 16)
    rnd = round_bf16 if cfg.dtype == "bf16" else (lambda a: a)
    if layout == "ball":
        shape = (B, H, rows, d)
    else:
        shape = (B, rows, H * d)
    out = {
        "q": rnd(_normal(r[0], shape)),
        "k": rnd(_normal(r[1], shape)),
        "v": rnd(_normal(r[2], shape)),
    }
    # Gate logits: the caller's linear layer X W_g with X ~ N(0,1) [rows, C] and
    # W_g ~ N(0, 1/C) [C, 3], formed in float64 and stored as float32.
    C = H * d
    gate = np.empty((B, rows, 3), np.float32)
    wg = r[3].standard_normal((C, 3)) / math.sqrt(C)
    for b in range(B):
        for s in range(0, rows, 1 << 16):
            e = min(rows, s + (1 << 16))
            x = r[4].standard_normal((e - s, C))
            gate[b, s:e] = (x @ wg).astype(np.float32)
    out["gate"] = gate
    ld = cfg.cmp_block * d
    # phi_q: the query-coarsening MLP of Eq. 13 (own stream; the other tensors are unchanged)
    for name, rr in (("phi_k", r[5]), ("phi_v", r[6]), ("phi_q", r[8])):
        out[name] = _mlp_weights(rr, ld, d, rnd)
    if with_grad:
        out["do"] = rnd(_normal(r[7], (B, H, cfg.n_pad, d)))
    return out


def _gate_logits_chunked(seq, rows: int, C: int, threads: int = 8) -> np.ndarray:
    """Gate logits [1, rows, 3] = X W_g with W_g ~ N(0, 1/C) [C, 3] (drawn in float64, stored
    as float32) and X ~ N(0,1) [rows, C] drawn in float32 in chunks of 2^16 rows, one stream
    per chunk; the product is formed in float32. Chunks run in a thread pool."""
    from concurrent.futures import ThreadPoolExecutor
    nch = (rows + (1 << 16) - 1) >> 16
    seqs = seq.spawn(nch + 1)
    wg = (np.random.default_rng(seqs[0]).standard_normal((C, 3)) / math.sqrt(C)).astype(np.float32)
    gate = np.empty((1, rows, 3), np.float32)

    def chunk(i):
        s0, e = i << 16, min(rows, (i + 1) << 16)
        x = np.empty((e - s0, C), np.float32)
        np.random.default_rng(seqs[i + 1]).standard_normal(out=x, dtype=np.float32)
        gate[0, s0:e] = x @ wg

    with ThreadPoolExecutor(threads) as ex:
        list(ex.map(chunk, range(nch)))
    return gate


class HeadInputs:
    """Seeded layer inputs drawn one head at a time, for workloads whose Q/K/V do not fit
    comfortably in host memory at once (2^20 points x 16 heads): each (tensor, head) pair has
    its own stream spawned from SeedSequence(seed * 1000 + 5), so any head can be drawn alone.
    Same distributions as make_inputs (N(0,1) Q/K/V/dO rounded to bf16 for bf16 workloads,
    gate logits X W_g, MLP weights N(0, 0.02^2)); cfg.batch must be 1."""

    def __init__(self, cfg: Config, seed: int | None = None):
        if cfg.batch != 1:
            raise ValueError("HeadInputs draws one cloud")
        self.cfg = cfg
        self.seed = _default_seed(cfg, seed)
        self._rnd = round_bf16 if cfg.dtype == "bf16" else (lambda a: a)
        self._seqs = np.random.SeedSequence(self.seed * 1000 + 5).spawn(4 * cfg.heads + 4)
        r = [np.random.default_rng(s) for s in self._seqs[4 * cfg.heads + 1:]]
        ld = cfg.cmp_block * cfg.head_dim
        self.gate = _gate_logits_chunked(self._seqs[4 * cfg.heads], cfg.n_pad, cfg.heads * cfg.head_dim)
        self.phi_k = _mlp_weights(r[0], ld, cfg.head_dim, self._rnd)
        self.phi_v = _mlp_weights(r[1], ld, cfg.head_dim, self._rnd)
        self.phi_q = _mlp_weights(r[2], ld, cfg.head_dim, self._rnd)

    def head(self, h: int, names=("q", "k", "v")) -> dict:
        """{name: float32 [n_pad, d]} of head h (names among q, k, v, do)."""
        out = {}
        for i, n in enumerate(("q", "k", "v", "do")):
            if n in names:
                x = np.empty((self.cfg.n_pad, self.cfg.head_dim), np.float32)
                np.random.default_rng(self._seqs[4 * h + i]).standard_normal(out=x, dtype=np.float32)
                out[n] = self._rnd(x)
        return out

    def heads(self, fn, names=("q", "k", "v"), threads: int = 8):
        """Calls fn(h, head(h, names)) for every head, drawing up to `threads` heads at once
        (fn runs on the calling thread, in head order)."""
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(threads) as ex:
            futs = [ex.submit(self.head, h, names) for h in range(self.cfg.heads)]
            for h, f in enumerate(futs):
                fn(h, f.result())
                futs[h] = None


def make_block_inputs(cfg: Config, valid: np.ndarray, ffn: int | None = None, seed: int | None = None) -> dict:
    """Seeded inputs of one transformer block around the layer: tokens x [B, n_pad, C]
    (N(0,1) on real slots, zero on padding slots), the block's float32 weights (norm gains
    1 + N(0, 0.01), matrices N(0, 1/fan_in)), the layer's MLPs (as in make_inputs) and the
    upstream gradient dy [B, n_pad, C] (N(0,1) on real slots, zero on padding slots).
    C = heads * head_dim, F = ffn (default 4C)."""
    seed = _default_seed(cfg, seed)
    B, C = cfg.batch, cfg.heads * cfg.head_dim
    F = ffn or 4 * C
    r = _streams(seed * 1000 + 3, 12)
    mask = np.asarray(valid, bool)[..., None]
    x = _normal(r[0], (B, cfg.n_pad, C)) * mask
    dy = _normal(r[1], (B, cfg.n_pad, C)) * mask
    W = {
        "g1": (1.0 + 0.1 * r[2].standard_normal(C)).astype(np.float32),
        "wqkv": _normal(r[3], (3 * C, C), 1.0 / math.sqrt(C)),
        "wg": _normal(r[4], (3, C), 1.0 / math.sqrt(C)),
        "wo": _normal(r[5], (C, C), 1.0 / math.sqrt(C)),
        "g2": (1.0 + 0.1 * r[6].standard_normal(C)).astype(np.float32),
        "w1": _normal(r[7], (F, C), 1.0 / math.sqrt(C)),
        "w3": _normal(r[8], (F, C), 1.0 / math.sqrt(C)),
        "w2": _normal(r[9], (C, F), 1.0 / math.sqrt(F)),
    }
    ld = cfg.cmp_block * cfg.head_dim
    rnd = round_bf16 if cfg.dtype == "bf16" else (lambda a: a)
    return {"x": x.astype(np.float32), "dy": dy.astype(np.float32), "W": W, "ffn": F,
            "phi_k": _mlp_weights(r[10], ld, cfg.head_dim, rnd), "phi_v": _mlp_weights(r[11], ld, cfg.head_dim, rnd),
            "phi_q": _mlp_weights(_streams(seed * 1000 + 4, 1)[0], ld, cfg.head_dim, rnd)}
