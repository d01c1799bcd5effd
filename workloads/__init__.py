"""Seeded synthetic workloads for the dual-sparse SpMSpV y = W x.

This module only *draws inputs*: weights, pruning masks, activation vectors
and the activation threshold that reaches a target zero fraction.  It holds
none of the method's arithmetic (no encoding, no selection, no product), so
both the CPU oracle and the GPU library can be fed from it without sharing
any code with each other.

Recipe (all draws from numpy ``default_rng`` / PCG64):

* one generator per (config, seed, layer, projection) via
  ``SeedSequence([config, seed, layer, projection])``; draw order W, mask, x;
* W = fp16(N(0,1) * 0.02), float32 draw then a round-to-nearest-even cast;
* uniform unstructured mask: keep iff U[0,1) >= s (float32 draw);
* per-row magnitude pruning: keep the K - (s*K)//100 largest |w| of each row,
  ties to the lower column index (stable argsort);
* x = fp16 of N(0,1), Laplace(0,1) or Student-t(nu=4);
* tau: the n0-th smallest |x| (as its exact fp16 value), n0 = (p*K)//100, so
  that at least p% of x is not strictly above tau; p = 0 gives tau = -1.

The shapes are those of the LLaMA-2-7B / LLaMA-2-13B / LLaMA-2-70B-class
projections the paper evaluates on (Section 5, Workloads).  No trained weights
or datasets are used: N(0, 0.02) weights and heavy-tailed activations stand
in for them.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

# projection ids used in the seed sequence
PROJ_IDS = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6, "w": 7}


def rng_for(config: int, seed: int, layer: int = 0, proj: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([config, seed, layer, proj]))


def draw_weight(rng: np.random.Generator, M: int, K: int, scale: float = 0.02) -> np.ndarray:
    """fp16 W of shape (M, K) (out x in), values N(0, scale^2)."""
    w = rng.standard_normal((M, K), dtype=np.float32)
    w *= np.float32(scale)
    return w.astype(np.float16)


def draw_mask_uniform(rng: np.random.Generator, M: int, K: int, sparsity_pct: float) -> np.ndarray:
    """Bernoulli keep-mask (uint8 0/1): an entry is kept iff U >= s."""
    u = rng.random((M, K), dtype=np.float32)
    return (u >= np.float32(sparsity_pct / 100.0)).astype(np.uint8)


def mask_row_magnitude(W: np.ndarray, sparsity_pct: int) -> np.ndarray:
    """Per-row magnitude pruning: keep the K - (p*K)//100 largest |w| per row,
    ties broken toward the lower column index."""
    M, K = W.shape
    n_keep = K - (sparsity_pct * K) // 100
    mag = np.abs(W.astype(np.float32))
    order = np.argsort(-mag, axis=1, kind="stable")
    mask = np.zeros((M, K), dtype=np.uint8)
    rows = np.arange(M)[:, None]
    mask[rows, order[:, :n_keep]] = 1
    return mask


def draw_x(rng: np.random.Generator, K: int, dist: str) -> np.ndarray:
    if dist == "normal":
        v = rng.standard_normal(K)
    elif dist == "laplace":
        v = rng.laplace(0.0, 1.0, K)
    elif dist == "student_t4":
        v = rng.standard_t(4.0, K)
    else:
        raise ValueError(f"unknown activation distribution {dist!r}")
    return v.astype(np.float16)


def tau_for_sparsity(x: np.ndarray, sparsity_pct: float) -> float:
    """Threshold reaching at least ``sparsity_pct`` % zeros under |x| > tau."""
    K = x.shape[0]
    n0 = int((int(round(sparsity_pct * 100)) * K) // 10000)
    if n0 <= 0:
        return -1.0
    a = np.sort(np.abs(x.astype(np.float32)))
    return float(a[n0 - 1])


# --------------------------------------------------------------------------
# The five benchmark configurations (shapes are W = out x in = M x K)
# --------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Projection:
    name: str
    M: int
    K: int
    x_group: str      # projections with the same x_group share one x


LLAMA7B = [Projection("q", 4096, 4096, "attn_in"), Projection("k", 4096, 4096, "attn_in"),
           Projection("v", 4096, 4096, "attn_in"), Projection("o", 4096, 4096, "attn_out"),
           Projection("gate", 11008, 4096, "mlp_in"), Projection("up", 11008, 4096, "mlp_in"),
           Projection("down", 4096, 11008, "mlp_mid")]
LLAMA13B = [Projection("q", 5120, 5120, "attn_in"), Projection("k", 5120, 5120, "attn_in"),
            Projection("v", 5120, 5120, "attn_in"), Projection("o", 5120, 5120, "attn_out"),
            Projection("gate", 13824, 5120, "mlp_in"), Projection("up", 13824, 5120, "mlp_in"),
            Projection("down", 5120, 13824, "mlp_mid")]
LLAMA70B = [Projection("q", 8192, 8192, "attn_in"), Projection("k", 1024, 8192, "attn_in"),
            Projection("v", 1024, 8192, "attn_in"), Projection("o", 8192, 8192, "attn_out"),
            Projection("gate", 28672, 8192, "mlp_in"), Projection("up", 28672, 8192, "mlp_in"),
            Projection("down", 8192, 28672, "mlp_mid")]

CONFIGS: Dict[int, dict] = {
    1: dict(name="4096x4096 ws50 as50 normal-x", layers=LLAMA7B[:1], ws=50, as_=50,
            mask="uniform", xdist="normal", seeds=[0], n_layers=1),
    2: dict(name="4096x4096 sweep ws{30,50,70} x as{30,50,70} laplace-x", layers=LLAMA7B[:1],
            ws=(30, 50, 70), as_=(30, 50, 70), mask="uniform", xdist="laplace",
            seeds=[0, 1, 2, 3, 4], n_layers=1),
    3: dict(name="llama-7b-shaped layer, 7 projections, ws50 row-magnitude, as50 t4-x",
            layers=LLAMA7B, ws=50, as_=50, mask="row_magnitude", xdist="student_t4",
            seeds=[0], n_layers=1),
    4: dict(name="llama-13b-shaped step, 40 layers x 7, ws60 as60 t4-x", layers=LLAMA13B,
            ws=60, as_=60, mask="uniform", xdist="student_t4", seeds=[0], n_layers=40),
    5: dict(name="llama-70b-shaped step, 80 layers x 7, ws50 as{40,60,80} laplace-x",
            layers=LLAMA70B, ws=50, as_=(40, 60, 80), mask="uniform", xdist="laplace",
            seeds=[0], n_layers=80),
}

# The headline point: 4096 x 4096 at 70 % weight + 70 % activation sparsity.
HEADLINE = dict(config=2, M=4096, K=4096, ws=70, as_=70, xdist="laplace", seed=0)


@dataclasses.dataclass
class Problem:
    W: np.ndarray        # fp16 (M, K)
    mask: np.ndarray     # uint8 (M, K)
    x: np.ndarray        # fp16 (K,)
    tau: float
    meta: dict


def make_problem(config: int, M: int, K: int, ws: float, as_: float, xdist: str,
                 seed: int = 0, layer: int = 0, proj: int = 0, mask_kind: str = "uniform",
                 x: Optional[np.ndarray] = None) -> Problem:
    """Draw W, then the mask, then x (unless a shared x is passed in)."""
    rng = rng_for(config, seed, layer, proj)
    W = draw_weight(rng, M, K)
    if mask_kind == "uniform":
        mask = draw_mask_uniform(rng, M, K, ws)
    elif mask_kind == "row_magnitude":
        mask = mask_row_magnitude(W, int(ws))
    else:
        raise ValueError(mask_kind)
    if x is None:
        x = draw_x(rng, K, xdist)
    tau = tau_for_sparsity(x, as_)
    meta = dict(config=config, M=M, K=K, ws=ws, as_=as_, xdist=xdist, seed=seed,
                layer=layer, proj=proj, mask=mask_kind)
    return Problem(W=W, mask=mask, x=x, tau=tau, meta=meta)


def outlier_feature_problem(M: int, K: int, ws: int, as_: float, sigma: float = 1.0,
                            seed: int = 0) -> Problem:
    """A layer with outlier input features: every input feature k gets a scale
    c_k = exp(sigma * N(0, 1)) shared by column k of W and by x_k, so large-scale
    columns keep more weights under per-row magnitude pruning and are also the
    ones whose activations pass the threshold (column densities from about 0
    to 95 % at sigma = 1).  Draw order: c, then W (N(0, 0.02) * c_k), then x
    (Laplace(0, 1) * c_k); mask by per-row magnitude; tau as for make_problem.
    Generator id: config 6."""
    rng = rng_for(6, seed, 0, PROJ_IDS["w"])
    c = np.exp(sigma * rng.standard_normal(K)).astype(np.float32)
    w = rng.standard_normal((M, K), dtype=np.float32)
    w *= np.float32(0.02)
    w *= c[None, :]
    W = w.astype(np.float16)
    mask = mask_row_magnitude(W, int(ws))
    x = (rng.laplace(0.0, 1.0, K) * c).astype(np.float16)
    tau = tau_for_sparsity(x, as_)
    meta = dict(config=6, M=M, K=K, ws=ws, as_=as_, xdist="laplace*c", sigma=sigma, seed=seed,
                mask="row_magnitude")
    return Problem(W=W, mask=mask, x=x, tau=tau, meta=meta)


def shared_x(config: int, seed: int, layer: int, group: str, K: int, xdist: str) -> np.ndarray:
    """The activation vector shared by projections of one x-group in a layer."""
    gid = {"attn_in": 100, "attn_out": 101, "mlp_in": 102, "mlp_mid": 103}[group]
    return draw_x(rng_for(config, seed, layer, gid), K, xdist)


def layer_problems(config: int, seed: int, layer: int, as_: Optional[float] = None) -> List[Problem]:
    """The 7 projections of one decoder layer of config 3, 4 or 5."""
    c = CONFIGS[config]
    a = c["as_"] if as_ is None else as_
    out = []
    xs: Dict[str, np.ndarray] = {}
    for p in c["layers"]:
        if p.x_group not in xs:
            xs[p.x_group] = shared_x(config, seed, layer, p.x_group, p.K, c["xdist"])
        out.append(make_problem(config, p.M, p.K, c["ws"], a, c["xdist"], seed=seed, layer=layer,
                                proj=PROJ_IDS[p.name], mask_kind=c["mask"], x=xs[p.x_group]))
        out[-1].meta["proj_name"] = p.name
    return out


def headline_problem(seed: int = 0) -> Problem:
    h = HEADLINE
    return make_problem(h["config"], h["M"], h["K"], h["ws"], h["as_"], h["xdist"], seed=seed,
                        proj=PROJ_IDS["w"])


def random_small(seed: int, M: int, K: int, ws: float, as_: float, xdist: str = "laplace",
                 zero_weights: int = 0) -> Problem:
    """Small fuzz case; optionally plants ``zero_weights`` kept entries of value +-0."""
    p = make_problem(99, M, K, ws, as_, xdist, seed=seed)
    if zero_weights:
        rng = rng_for(98, seed)
        kept = np.flatnonzero(p.mask.ravel())
        if kept.size:
            pick = rng.choice(kept, size=min(zero_weights, kept.size), replace=False)
            sign = rng.integers(0, 2, size=pick.size).astype(np.uint16) << np.uint16(15)
            Wb = p.W.view(np.uint16).ravel().copy()
            Wb[pick] = sign
            p.W = Wb.view(np.float16).reshape(M, K)
    return p
