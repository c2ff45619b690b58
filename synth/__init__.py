"""Seeded synthetic inputs for the routing path.

This module only draws random inputs. It holds none of the method's
arithmetic: no distances, no neighbour search, no averaging, no scores and
no assignment. Both the HIP path and the CPU oracle consume what it returns.

What the inputs stand for (RouteBalance, Sec. 4.2 and Tab. cluster):
  * a labelled reference bank of prompt embeddings, each row carrying a
    per-model quality label in [0, 1] and a per-model output length;
  * a batch of request embeddings with prompt lengths;
  * a table of serving instances, each serving one model, with dead-reckoned
    queue state, token rates and per-token prices.

The paper's own bank (MiniLM embeddings of its training prompts, judge
labels) is not available, so every array is drawn from the distributions
below, seeded. Each array gets its own child of ``SeedSequence(seed)`` so that
resizing one array never shifts another.

Embeddings: K unit-norm cluster centres; a row picks a uniform centre u and is
``c_u + sigma * z`` with ``z ~ N(0, I_d)``, then L2-normalised and cast to the
bank dtype (bf16 by round-to-nearest-even). ``sigma_mode="radius"`` (default)
uses per-coordinate sigma = 0.3/sqrt(d), i.e. a noise radius of 0.3;
``"literal"`` uses per-coordinate 0.3.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence

import numpy as np
import torch

__all__ = ["Config", "CONFIGS", "tiny_config", "Instances", "make_centres", "make_embeddings",
           "make_bank", "make_labels", "make_prompt_lens", "make_instances", "make_queries",
           "make_budgets", "make_availability", "simplex_lattice", "Stream"]


@dataclasses.dataclass(frozen=True)
class Config:
    """One synthetic workload. ``dtype`` is the bank/query storage type."""
    name: str
    B: int
    N: int
    d: int
    dtype: str                     # "f32" or "bf16"
    clusters: int
    M: int
    inst_per_model: tuple          # instance counts per model, contiguous blocks
    k: int = 10
    weights: tuple = (0.4, 0.3, 0.3)   # (w_qual, w_lat, w_cost), Alg. 1 order
    qual_alpha0: float = 2.0       # quality ~ Beta(qual_alpha0 + qual_alpha_step*m, 3)
    qual_alpha_step: float = 1.0
    len_mu0: float = 5.0           # out len ~ round(LogNormal(len_mu0 + len_mu_step*m, len_sigma))
    len_mu_step: float = -0.2
    len_sigma: float = 0.6
    prompt_mu: float = 6.0         # prompt len ~ round(LogNormal(prompt_mu, prompt_sigma))
    prompt_sigma: float = 0.8
    batches: int = 1
    seed: int = 0
    sigma_mode: str = "radius"

    @property
    def I(self) -> int:
        return int(sum(self.inst_per_model))

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def bank_bytes(self) -> int:
        return self.N * self.d * self.elem_bytes


# The five workloads: a tiny one the oracle finishes in seconds, the paper-scale
# online batch, a high-load batch (carried over 100 batches), a compute-bound
# large batch and a wide cluster; and stream64, the online batch of 64 requests
# over the high-load bank, an HBM-scale stream of a small batch.
CONFIGS = {
    "tiny": Config("tiny", B=16, N=2048, d=384, dtype="f32", clusters=32, M=4,
                   inst_per_model=(5, 4, 2, 2), weights=(0.4, 0.3, 0.3)),
    "online": Config("online", B=64, N=100_000, d=768, dtype="bf16", clusters=256, M=4,
                     inst_per_model=(5, 4, 2, 2), weights=(0.4, 0.3, 0.3)),
    "highload": Config("highload", B=256, N=1_000_000, d=768, dtype="bf16", clusters=1024, M=4,
                       inst_per_model=(5, 4, 2, 2), weights=(1 / 3, 1 / 3, 1 / 3), batches=100),
    "largebatch": Config("largebatch", B=1024, N=1_000_000, d=1024, dtype="bf16", clusters=1024,
                         M=8, inst_per_model=(8,) * 8, weights=(0.5, 0.25, 0.25),
                         qual_alpha0=1.5, qual_alpha_step=0.5),
    "stream64": Config("stream64", B=64, N=1_000_000, d=768, dtype="bf16", clusters=1024, M=4,
                       inst_per_model=(5, 4, 2, 2), weights=(0.4, 0.3, 0.3)),
    "wide": Config("wide", B=512, N=4_000_000, d=384, dtype="bf16", clusters=4096, M=16,
                   inst_per_model=(32,) * 16, weights=(0.1, 0.2, 0.7),
                   len_mu0=5.5, len_mu_step=0.0, len_sigma=1.0, prompt_mu=7.0, prompt_sigma=1.0),
}


def tiny_config(**kw) -> Config:
    """A variant of the tiny workload with fields overridden (test shapes)."""
    base = dataclasses.asdict(CONFIGS["tiny"])
    base.update(kw)
    base["inst_per_model"] = tuple(base["inst_per_model"])
    base["weights"] = tuple(base["weights"])
    return Config(**base)


class Stream:
    """Independent child seeds by role: ``Stream(seed).child(role_id)``."""
    ROLES = {"centres": 0, "bank": 1, "labels": 2, "instances": 3, "queries": 4, "prompts": 5,
             "budgets": 6, "availability": 7}

    def __init__(self, seed: int):
        self.seq = np.random.SeedSequence(seed)
        self.kids = self.seq.spawn(len(self.ROLES))

    def numpy(self, role: str, sub: int = 0) -> np.random.Generator:
        ss = self.kids[self.ROLES[role]]
        if sub:
            ss = np.random.SeedSequence(ss.entropy, spawn_key=ss.spawn_key + (sub,))
        return np.random.default_rng(ss)

    def torch_seed(self, role: str, sub: int = 0) -> int:
        return int(self.numpy(role, sub).integers(0, 2**62))


def _torch_gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def make_centres(cfg: Config, device="cpu") -> torch.Tensor:
    """K unit-norm cluster centres, fp32 ``[K][d]``."""
    g = _torch_gen(device, Stream(cfg.seed).torch_seed("centres"))
    c = torch.randn(cfg.clusters, cfg.d, generator=g, device=device, dtype=torch.float32)
    return c / c.norm(dim=1, keepdim=True)


def _sigma(cfg: Config) -> float:
    if cfg.sigma_mode == "radius":
        return 0.3 / math.sqrt(cfg.d)
    if cfg.sigma_mode == "literal":
        return 0.3
    raise ValueError(cfg.sigma_mode)


def make_embeddings(cfg: Config, rows: int, role: str, sub: int = 0, device="cpu",
                    centres: Optional[torch.Tensor] = None, chunk: int = 1 << 18) -> torch.Tensor:
    """``rows`` mixture draws, L2-normalised, stored in the config's dtype."""
    if centres is None:
        centres = make_centres(cfg, device)
    g = _torch_gen(device, Stream(cfg.seed).torch_seed(role, sub))
    out = torch.empty(rows, cfg.d, dtype=cfg.torch_dtype, device=device)
    sig = _sigma(cfg)
    for r0 in range(0, rows, chunk):
        r1 = min(rows, r0 + chunk)
        u = torch.randint(0, cfg.clusters, (r1 - r0,), generator=g, device=device)
        z = torch.randn(r1 - r0, cfg.d, generator=g, device=device, dtype=torch.float32)
        x = centres[u] + sig * z
        x = x / x.norm(dim=1, keepdim=True)
        out[r0:r1] = x.to(cfg.torch_dtype)
        del u, z, x
    return out


def make_bank(cfg: Config, device="cpu", centres=None) -> torch.Tensor:
    """Reference-bank embeddings ``[N][d]``."""
    return make_embeddings(cfg, cfg.N, "bank", 0, device, centres)


def make_queries(cfg: Config, batch: int = 0, device="cpu", centres=None) -> torch.Tensor:
    """Request embeddings ``[B][d]`` of batch ``batch`` (independent draws, same mixture)."""
    return make_embeddings(cfg, cfg.B, "queries", batch + 1, device, centres)


def make_labels(cfg: Config):
    """Per-row, per-model labels ``qual[N][M]``, ``len[N][M]`` as fp32 numpy arrays.

    quality ~ Beta(qual_alpha0 + qual_alpha_step*m, 3); length ~ max(1, round(LogNormal(
    len_mu0 + len_mu_step*m, len_sigma))). Labels are independent of the embedding.
    """
    rng = Stream(cfg.seed).numpy("labels")
    m = np.arange(cfg.M, dtype=np.float64)
    alpha = cfg.qual_alpha0 + cfg.qual_alpha_step * m
    qual = rng.beta(alpha[None, :], 3.0, size=(cfg.N, cfg.M)).astype(np.float32)
    mu = cfg.len_mu0 + cfg.len_mu_step * m
    ln = rng.lognormal(mu[None, :], cfg.len_sigma, size=(cfg.N, cfg.M))
    ln = np.maximum(1.0, np.rint(ln)).astype(np.float32)
    return qual, ln


def make_prompt_lens(cfg: Config, batch: int = 0) -> np.ndarray:
    """Prompt lengths ``[B]`` int32, max(1, round(LogNormal(prompt_mu, prompt_sigma)))."""
    rng = Stream(cfg.seed).numpy("prompts", batch + 1)
    x = rng.lognormal(cfg.prompt_mu, cfg.prompt_sigma, size=cfg.B)
    return np.maximum(1, np.rint(x)).astype(np.int32)


@dataclasses.dataclass
class Instances:
    """Instance table, struct of arrays, each of length I (numpy)."""
    model: np.ndarray          # int32, m(i)
    prefill_q: np.ndarray      # fp32, queued prefill tokens
    decode_q: np.ndarray       # fp32, active decode tokens
    prefill_rate: np.ndarray   # fp32, tokens/s
    decode_rate: np.ndarray    # fp32, tokens/s
    price_in: np.ndarray       # fp32, per input token
    price_out: np.ndarray      # fp32, per output token

    FIELDS = ("model", "prefill_q", "decode_q", "prefill_rate", "decode_rate", "price_in",
              "price_out")

    def copy(self) -> "Instances":
        return Instances(*[getattr(self, f).copy() for f in self.FIELDS])

    @property
    def I(self) -> int:
        return int(self.model.shape[0])


def _log_uniform_band(rng, lo, hi, band, nbands, size):
    """Log-uniform draw inside sub-band ``band`` of ``nbands`` equal log-width bands."""
    a, b = math.log(lo), math.log(hi)
    w = (b - a) / nbands
    return np.exp(rng.uniform(a + band * w, a + (band + 1) * w, size=size))


def make_instances(cfg: Config) -> Instances:
    """Instances in contiguous model blocks (``inst_per_model``).

    queued prefill ~ U[0, 8000], active decode ~ U[0, 20000]; prefill rate in
    [5k, 40k] and decode rate in [200, 3000] tok/s, log-uniform in a sub-band that
    falls as m grows (larger models are slower); price in [0.1, 2.0] per 1k tokens,
    log-uniform in a sub-band that rises with m; input and output price both set
    to that per-token price.
    """
    rng = Stream(cfg.seed).numpy("instances")
    model = np.concatenate([np.full(c, m, dtype=np.int32) for m, c in enumerate(cfg.inst_per_model)])
    I = model.shape[0]
    p = rng.uniform(0.0, 8000.0, size=I)
    a = rng.uniform(0.0, 20000.0, size=I)
    P = np.empty(I)
    D = np.empty(I)
    price = np.empty(I)
    for i in range(I):
        m = int(model[i])
        P[i] = _log_uniform_band(rng, 5000.0, 40000.0, cfg.M - 1 - m, cfg.M, None)
        D[i] = _log_uniform_band(rng, 200.0, 3000.0, cfg.M - 1 - m, cfg.M, None)
        price[i] = _log_uniform_band(rng, 0.1, 2.0, m, cfg.M, None) / 1000.0
    f = np.float32
    return Instances(model, p.astype(f), a.astype(f), P.astype(f), D.astype(f),
                     price.astype(f), price.astype(f))


def make_budgets(cfg: Config, batch: int = 0, fraction: float = 0.45, lo: float = 0.03,
                 hi: float = 1.5) -> np.ndarray:
    """Per-request cost budgets ``[B]`` fp32 (Alg. 1's optional b_r).

    A ``fraction`` of the requests, chosen at random, carry a budget drawn
    log-uniform in [lo, hi] (the currency of the per-token prices; with the
    instance prices and the length distributions above, expected request costs
    run from about 0.04 to 2.2 between their 1st and 99th percentiles); the others carry +inf, i.e. no budget. The paper's
    budget study constrains 75, 45 or 30 % of the prompts.
    """
    rng = Stream(cfg.seed).numpy("budgets", batch + 1)
    has = rng.uniform(size=cfg.B) < fraction
    val = np.exp(rng.uniform(math.log(lo), math.log(hi), size=cfg.B))
    return np.where(has, val, np.inf).astype(np.float32)


def make_availability(cfg: Config, lost_models: Sequence[int] = (), down_fraction: float = 0.0
                      ) -> np.ndarray:
    """Instance availability ``[I]`` uint8 (1 = available).

    Every instance of a model in ``lost_models`` is unavailable (a lost tier, as
    in the paper's tier-loss study); of the rest, each is down independently
    with probability ``down_fraction``.
    """
    rng = Stream(cfg.seed).numpy("availability")
    model = np.concatenate([np.full(c, m, dtype=np.int32) for m, c in enumerate(cfg.inst_per_model)])
    up = ~np.isin(model, np.asarray(list(lost_models), dtype=np.int32))
    up &= rng.uniform(size=model.shape[0]) >= down_fraction
    return up.astype(np.uint8)


def simplex_lattice(step: float) -> list:
    """All (w_qual, w_lat, w_cost) on the 3-simplex lattice with the given step."""
    n = int(round(1.0 / step))
    pts = []
    for i in range(n + 1):
        for j in range(n + 1 - i):
            pts.append((i / n, j / n, (n - i - j) / n))
    return pts
