"""Anchor-prior state over training steps (paper Sec. 3.2; Alg. 1; App. H).

For every targeted weight matrix the fast circuit keeps the anchor EMA
M^anc and the spectral basis of its top-r SVD.  Alg. 1 folds an anchor
gradient into M^anc whenever one arrives (asynchronously, every Delta ~ 20
fast steps) and corrects the masked gradient of every step with the basis of
the current M^anc.  M^anc changes only on arrival, so the basis is rebuilt
then and reused exactly on the steps in between; a rebuild starts its
subspace iteration from the previous right basis (warm start), which the
slow drift of the anchor subspace makes a good starting block.

Every operation is a batched library call (sc_build_prior_batched,
sc_correct_batched, sc_correct_adamw_batched) over all matrices at once;
this class holds the device buffers and the arrival bookkeeping.
"""
from __future__ import annotations

from typing import Optional, Sequence

import torch

from . import sc_build_prior_batched, sc_correct_adamw_batched, sc_correct_batched, workspace


class AnchorPrior:
    """The anchor EMA and its basis for a set of weight matrices.

    Before the first arrival M^anc = 0, so d = 0 and the correction returns
    alpha * G (the paper's formula on an empty prior)."""

    def __init__(self, shapes: Sequence[tuple], r: int, beta: float, tau: float, oversample: int,
                 power_iters: int, dtype: torch.dtype = torch.bfloat16, device="cuda",
                 warm_start: bool = True, seed: int = 0):
        self.shapes = [tuple(s) for s in shapes]
        self.r, self.beta, self.tau = r, beta, tau
        self.oversample, self.power_iters = oversample, power_iters
        self.dtype, self.device = dtype, torch.device(device)
        self.warm_start, self.seed = warm_start, seed
        self.arrivals = 0
        self.M = [torch.zeros(m, n, device=self.device) for m, n in self.shapes]
        self.U = [torch.zeros(m, r, device=self.device) for m, _ in self.shapes]
        self.s = [torch.zeros(r, device=self.device) for _ in self.shapes]
        self.V = [torch.zeros(n, r, device=self.device) for _, n in self.shapes]
        self.d = [torch.zeros(r, device=self.device) for _ in self.shapes]
        self.ws = [workspace(m, n, r, oversample, dtype, self.device) for m, n in self.shapes]

    def arrive(self, G_anc: Sequence[Optional[torch.Tensor]], stream=None) -> None:
        """An anchor gradient per matrix (None: no new gradient for that
        matrix, its EMA is kept): fold into M^anc, rebuild every basis."""
        if len(G_anc) != len(self.shapes):
            raise ValueError("one anchor gradient (or None) per matrix")
        items = []
        for i, g in enumerate(G_anc):
            it = dict(G_anc=g, M=self.M[i], out=(self.U[i], self.s[i], self.V[i], self.d[i]), ws=self.ws[i])
            if self.warm_start and self.arrivals > 0:
                it["V_warm"] = self.V[i].clone()
            items.append(it)
        # matrix i of arrival a draws its random columns from seed + a * count + i
        sc_build_prior_batched(items, self.r, self.beta, self.tau, self.oversample, self.power_iters,
                               seed=self.seed + self.arrivals * len(self.shapes), dtype=self.dtype,
                               stream=stream)
        self.arrivals += 1

    def prior(self, i: int):
        """(U, d, V) of matrix i."""
        return self.U[i], self.d[i], self.V[i]

    def correct(self, G: Sequence[torch.Tensor], alpha: float, out: Optional[Sequence[torch.Tensor]] = None,
                stream=None):
        """G_proj = alpha G + (1 - alpha) G_filt for every matrix, with the
        current basis.  Returns the G_proj tensors (out, or new tensors)."""
        if out is None:
            out = [torch.empty_like(g) for g in G]
        items = [dict(G=g, prior=self.prior(i), out=o, ws=self.ws[i]) for i, (g, o) in enumerate(zip(G, out))]
        sc_correct_batched(items, self.r, alpha, dtype=self.dtype, stream=stream)
        return list(out)

    def correct_adamw(self, G: Sequence[torch.Tensor], states: Sequence[tuple], alpha: float, lr: float,
                      step: int, norm_out: Optional[torch.Tensor] = None, stream=None, **hp) -> None:
        """The corrected AdamW step of every matrix (states: (W, m1, m2) fp32, in place)."""
        items = [dict(G=g, prior=self.prior(i), ws=self.ws[i], state=tuple(st))
                 for i, (g, st) in enumerate(zip(G, states))]
        sc_correct_adamw_batched(items, self.r, alpha, lr, step=step, dtype=self.dtype, norm_out=norm_out,
                                 stream=stream, **hp)
