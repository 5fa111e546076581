"""Seeded synthetic inputs for the masking compressor and the spectral corrector.

This module only *draws inputs*: activations, low-rank-plus-noise gradient
matrices, mask keys and hyperparameters.  It holds none of the method's
arithmetic (no masking, packing, EMA, SVD, filtering or blending), so both the
CPU oracle and the HIP path can consume exactly the same bits from it.

Shapes follow the model classes the paper trains and evaluates:

* 1B class: Llama-3.2-1B, hidden size 2048, MLP width 8192, 2k context
  (Sec. 5.1 setup; App. H uses S = H = 2048).
* 8B class: hidden 4096, MLP 14336, GQA k/v projection 4096x1024 (Table 3
  covers 1B-8B models).
* 70B-class slice: hidden 8192, MLP 28672, four layers resident on one GPU.

Every tensor is drawn from a ``torch.Generator`` seeded from
``(2609, config, layer, tensor id)``; the same call on the same device gives
the same bits.  CPU and GPU generators produce different streams, so a test
draws on one device and copies to the other.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import torch

# Paper defaults (Table 2): mask probability p = 0.95 (keep 0.05), staleness
# 20 steps, filter damping 1e-3, blend alpha = 0.3.  beta_anc is not given
# (Sec. 3.2 only asks it to span several anchor cycles); 0.9 is our reading.
ALPHA = 0.3
TAU = 1e-3
BETA = 0.9


@dataclasses.dataclass(frozen=True)
class ActSpec:
    B: int
    S: int
    H: int
    dtype: torch.dtype
    keep: Tuple[float, ...]      # keep fractions (1 - p) swept for this config
    dist: str                    # "normal" or "student_t4"


@dataclasses.dataclass(frozen=True)
class GradSpec:
    shapes: Tuple[Tuple[int, int], ...]   # (m, n) per matrix of one layer
    rank: int                              # signal rank rho
    s_range: Tuple[float, float]           # log-spaced signal singular values
    r: Tuple[int, ...]                     # prior ranks swept
    dtype: torch.dtype
    anc_noise: Optional[float]             # absolute std; None -> 0.05 * ||S||_F / sqrt(mn)
    mask_noise: Optional[float]
    layers: int = 1
    rot_eps: Tuple[float, ...] = (0.0,)    # rotation of the masked signal subspace


@dataclasses.dataclass(frozen=True)
class Config:
    cid: int
    name: str
    act: ActSpec
    grad: GradSpec
    oversample: int
    power_iters: int


CONFIGS = {
    1: Config(1, "tiny-fp32",
              ActSpec(2, 64, 256, torch.float32, (0.1,), "normal"),
              GradSpec(((256, 256),), 8, (1.0, 10.0), (8,), torch.float32, 0.01, 0.1),
              oversample=8, power_iters=6),
    2: Config(2, "1b-bf16",
              ActSpec(8, 2048, 2048, torch.bfloat16, (0.05,), "normal"),
              GradSpec(((2048, 2048),) * 4 + ((2048, 8192), (8192, 2048)), 32, (1.0, 100.0),
                       (32,), torch.bfloat16, None, None),
              oversample=16, power_iters=2),
    3: Config(3, "8b-bf16",
              ActSpec(4, 4096, 4096, torch.bfloat16, (0.02, 0.05, 0.1), "student_t4"),
              GradSpec(((4096, 4096), (4096, 1024), (4096, 14336), (14336, 4096)), 64,
                       (1.0, 100.0), (64,), torch.bfloat16, None, None),
              oversample=16, power_iters=3),
    4: Config(4, "8b-staleness",
              ActSpec(4, 4096, 4096, torch.bfloat16, (0.05,), "student_t4"),
              GradSpec(((4096, 4096), (4096, 1024), (4096, 14336), (14336, 4096)), 64,
                       (1.0, 100.0), (16, 64, 128), torch.bfloat16, None, None,
                       rot_eps=(0.0, 0.05, 0.2)),
              oversample=16, power_iters=3),
    5: Config(5, "70b-slice-4layer-bf16",
              ActSpec(2, 8192, 8192, torch.bfloat16, (0.02,), "normal"),
              GradSpec(((8192, 8192), (8192, 28672), (28672, 8192)), 128, (1.0, 100.0),
                       (128,), torch.bfloat16, None, None, layers=4),
              oversample=16, power_iters=2),
}


def _gen(device, *ids: int) -> torch.Generator:
    """A generator seeded from (2609, *ids); deterministic per device type."""
    g = torch.Generator(device=device)
    seed = 2609
    for v in ids:
        seed = (seed * 1000003 + int(v) + 1) % (2 ** 62)
    g.manual_seed(seed)
    return g


def keep_count_plain(H: int, keep: float) -> int:
    """K = round(keep * H), ties away from zero, as a plain integer."""
    return int(math.floor(keep * H + 0.5))


def mask_key_fields(cid: int, layer: int = 0, step: int = 1, microbatch: int = 0):
    """Key fields (seed, layer, step, microbatch) used for config ``cid``."""
    return dict(seed=14339 + cid, layer=layer, step=step, microbatch=microbatch)


def activation(spec: ActSpec, cid: int, layer: int = 0, tensor_id: int = 0,
               device="cpu", rows: Optional[int] = None) -> torch.Tensor:
    """[B*S, H] activation (or activation gradient) in ``spec.dtype``.

    ``normal``: iid N(0, 1).  ``student_t4``: standard Student-t with 4 degrees
    of freedom, drawn as z / sqrt(chi2_4 / 4) with chi2_4 the sum of four
    squared standard normals (heavy tails, variance 2).
    """
    n_rows = spec.B * spec.S if rows is None else rows
    g = _gen(device, cid, layer, 100 + tensor_id)
    z = torch.randn(n_rows, spec.H, generator=g, device=device, dtype=torch.float32)
    if spec.dist == "student_t4":
        c = torch.zeros_like(z)
        for _ in range(4):
            e = torch.randn(n_rows, spec.H, generator=g, device=device, dtype=torch.float32)
            c.add_(e * e)
        z = z / torch.sqrt(c / 4.0)
    return z.to(spec.dtype)


def log_spaced(lo: float, hi: float, k: int, dtype=torch.float64, device="cpu") -> torch.Tensor:
    """k values log-spaced from hi down to lo (descending)."""
    if k == 1:
        return torch.tensor([hi], dtype=dtype, device=device)
    e = torch.linspace(math.log(hi), math.log(lo), k, dtype=dtype, device=device)
    return torch.exp(e)


def orthonormal(rows: int, cols: int, g: torch.Generator, device, dtype=torch.float64) -> torch.Tensor:
    """rows x cols matrix with orthonormal columns (QR of a Gaussian matrix)."""
    a = torch.randn(rows, cols, generator=g, device=device, dtype=dtype)
    q, r = torch.linalg.qr(a)
    # fix the sign so the factor is a deterministic function of the draw
    sgn = torch.sign(torch.diagonal(r))
    sgn[sgn == 0] = 1
    return q * sgn


def rotate_columns(Q: torch.Tensor, eps: float, g: torch.Generator) -> torch.Tensor:
    """exp(eps*A) @ Q for the skew generator A = W Q^T - Q W^T.

    W is a random orthonormal block orthogonal to span(Q).  Then
    exp(eps*A) Q = Q cos(eps) + W sin(eps) in closed form, so every principal
    angle between span(Q) and the result is exactly eps.
    """
    if eps == 0.0:
        return Q.clone()
    m, k = Q.shape
    Z = torch.randn(m, k, generator=g, device=Q.device, dtype=Q.dtype)
    Z = Z - Q @ (Q.T @ Z)
    Z = Z - Q @ (Q.T @ Z)
    W, R = torch.linalg.qr(Z)
    sgn = torch.sign(torch.diagonal(R))
    sgn[sgn == 0] = 1
    W = W * sgn
    return Q * math.cos(eps) + W * math.sin(eps)


@dataclasses.dataclass
class GradPair:
    """One weight matrix's gradients: anchor gradient and masked gradient."""
    G_anc: torch.Tensor      # [m, n] in the config dtype
    G_mask: torch.Tensor     # [m, n] in the config dtype
    s_signal: torch.Tensor   # [rho] float64, the constructed singular values
    U_sig: torch.Tensor      # [m, rho] float64 (anchor signal left basis)
    V_sig: torch.Tensor      # [n, rho] float64


def grad_pair(spec: GradSpec, cid: int, layer: int, mat: int, device="cpu",
              rot_eps: float = 0.0, keep_basis: bool = False) -> GradPair:
    """Low-rank signal S = U diag(s) V^T plus independent Gaussian noise.

    G_anc = S + sigma_a * N and G_mask = S' + sigma_m * N', where S' uses the
    signal subspaces rotated by ``rot_eps`` (zero means S' = S).  When the
    spec gives no absolute noise level, sigma = 0.05 * ||S||_F / sqrt(mn), the
    reading of "0.05 times the signal scale" as a per-entry standard deviation.
    """
    m, n = spec.shapes[mat]
    rho = spec.rank
    g = _gen(device, cid, layer, mat)
    U = orthonormal(m, rho, g, device)
    V = orthonormal(n, rho, g, device)
    s = log_spaced(spec.s_range[0], spec.s_range[1], rho, device=device)
    S = (U * s) @ V.T
    fro = float(torch.sqrt(torch.sum(s * s)))
    auto = 0.05 * fro / math.sqrt(m * n)
    sa = spec.anc_noise if spec.anc_noise is not None else auto
    sm = spec.mask_noise if spec.mask_noise is not None else auto
    Na = torch.randn(m, n, generator=g, device=device, dtype=torch.float32).double()
    G_anc = (S + sa * Na).to(spec.dtype)
    del Na
    if rot_eps != 0.0:
        U2 = rotate_columns(U, rot_eps, g)
        V2 = rotate_columns(V, rot_eps, g)
        S2 = (U2 * s) @ V2.T
    else:
        S2 = S
    Nm = torch.randn(m, n, generator=g, device=device, dtype=torch.float32).double()
    G_mask = (S2 + sm * Nm).to(spec.dtype)
    del Nm, S, S2
    return GradPair(G_anc, G_mask, s, U if keep_basis else U[:, :0], V if keep_basis else V[:, :0])


def anchor_arrival(spec: GradSpec, cid: int, layer: int, mat: int, arrival: int, drift: float,
                   device="cpu") -> Tuple[torch.Tensor, torch.Tensor]:
    """(G_anc, G_mask) of anchor arrival ``arrival`` (0, 1, ..) of a signal
    whose subspaces drift along one fixed geodesic.

    The signal basis of ``grad_pair`` (same seed) is rotated by
    arrival * drift for the anchor gradient and by (arrival + 1) * drift for
    the masked gradient that the arrival's prior will correct (one arrival
    ahead), always toward the same orthonormal directions, so the subspaces
    of consecutive arrivals sit ``drift`` apart.  Each arrival draws fresh
    noise at the spec's level.  float64 on ``device``, cast to spec.dtype."""
    m, n = spec.shapes[mat]
    rho = spec.rank
    g = _gen(device, cid, layer, mat)
    U = orthonormal(m, rho, g, device)
    V = orthonormal(n, rho, g, device)
    s = log_spaced(spec.s_range[0], spec.s_range[1], rho, device=device)
    fro = float(torch.sqrt(torch.sum(s * s)))
    auto = 0.05 * fro / math.sqrt(m * n)
    sa = spec.anc_noise if spec.anc_noise is not None else auto
    sm = spec.mask_noise if spec.mask_noise is not None else auto

    def signal(angle: float) -> torch.Tensor:
        gu = _gen(device, cid, layer, 500 + mat)      # the same directions at every angle
        Ua = rotate_columns(U, angle, gu)
        Va = rotate_columns(V, angle, gu)
        return (Ua * s) @ Va.T

    gn = _gen(device, cid, layer, 600 + 16 * mat + arrival)
    Na = torch.randn(m, n, generator=gn, device=device, dtype=torch.float32).double()
    G_anc = (signal(arrival * drift) + sa * Na).to(spec.dtype)
    Nm = torch.randn(m, n, generator=gn, device=device, dtype=torch.float32).double()
    G_mask = (signal((arrival + 1) * drift) + sm * Nm).to(spec.dtype)
    return G_anc, G_mask


def grad_pair_fast(spec: GradSpec, cid: int, layer: int, mat: int, device="cuda",
                   rot_eps: float = 0.0) -> Tuple[torch.Tensor, torch.Tensor]:
    """Same construction as ``grad_pair`` in float32 on ``device`` (for the
    large shapes, where float64 on the host would take minutes).  Returns
    (G_anc, G_mask) in the config dtype."""
    m, n = spec.shapes[mat]
    rho = spec.rank
    g = _gen(device, cid, layer, mat)
    U = orthonormal(m, rho, g, device, dtype=torch.float32)
    V = orthonormal(n, rho, g, device, dtype=torch.float32)
    s = log_spaced(spec.s_range[0], spec.s_range[1], rho, dtype=torch.float32, device=device)
    fro = float(torch.sqrt(torch.sum(s.double() * s.double())))
    auto = 0.05 * fro / math.sqrt(m * n)
    sa = spec.anc_noise if spec.anc_noise is not None else auto
    sm = spec.mask_noise if spec.mask_noise is not None else auto
    Us = U * s
    G = torch.randn(m, n, generator=g, device=device, dtype=torch.float32)
    G.mul_(sa).addmm_(Us, V.T)
    G_anc = G.to(spec.dtype)
    if rot_eps != 0.0:
        U2 = rotate_columns(U, rot_eps, g)
        V2 = rotate_columns(V, rot_eps, g)
        Us = U2 * s
        V = V2
    torch.randn(m, n, generator=g, device=device, dtype=torch.float32, out=G)
    G.mul_(sm).addmm_(Us, V.T)
    G_mask = G.to(spec.dtype)
    del G
    return G_anc, G_mask


def random_orthonormal_basis(m: int, n: int, r: int, seed: int, device="cpu"):
    """(U, s, V) with orthonormal U [m, r], V [n, r] and log-spaced s in
    [0.5, 5] (descending): an arbitrary prior basis for correction tests."""
    g = _gen(device, 77, seed, m * 131 + n)
    U = orthonormal(m, r, g, device)
    V = orthonormal(n, r, g, device)
    s = log_spaced(0.5, 5.0, r, device=device)
    return U, s, V


def gaussian(shape: Sequence[int], seed: int, device="cpu", dtype=torch.float32, std=1.0):
    g = _gen(device, 91, seed)
    return (torch.randn(*shape, generator=g, device=device, dtype=torch.float32) * std).to(dtype)
