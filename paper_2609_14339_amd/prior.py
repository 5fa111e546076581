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

Streams.  A build may run on a stream of its own beside the corrections (the
prior is built asynchronously).  Builds and corrections use separate
workspaces, and the basis is double-buffered: corrections read the front
buffer while a build writes the back one.  HIP events order what must be
ordered: a build waits for the work that produced its inputs (the caller's
current stream), for the previous build (the EMA state and the warm-start
basis) and for the last correction that read the buffer it overwrites; a
correction waits for the build that wrote the buffer it reads and for the
previous correction (they share the correction workspaces).  Tensors used
on a stream other than the current one are recorded on it, so the caching
allocator does not hand their memory out early.
"""
from __future__ import annotations

from typing import List, Optional, Sequence

import torch

from . import (sc_adamw_workspace_size, sc_build_prior_batched, sc_correct_adamw_batched, sc_correct_batched,
               workspace)


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
        dev = self.device
        self.M = [torch.zeros(m, n, device=dev) for m, n in self.shapes]
        # two bases per matrix: (U, s, V, d); corrections read buffer `front`
        self.bufs = [[(torch.zeros(m, r, device=dev), torch.zeros(r, device=dev), torch.zeros(n, r, device=dev),
                       torch.zeros(r, device=dev)) for m, n in self.shapes] for _ in range(2)]
        self.front = 0
        self._pending: Optional[int] = None
        self.ws = [workspace(m, n, r, oversample, dtype, dev) for m, n in self.shapes]
        self.cws = [torch.empty(max(sc_adamw_workspace_size(m, n, r, dtype), 256), dtype=torch.uint8, device=dev)
                    for m, n in self.shapes]
        self._written: List[Optional[torch.cuda.Event]] = [None, None]   # last build that wrote buffer b
        self._read: List[Optional[torch.cuda.Event]] = [None, None]      # last correction that read buffer b
        self._last_build: Optional[torch.cuda.Event] = None
        self._last_correct: Optional[torch.cuda.Event] = None

    # the basis the corrections use
    @property
    def U(self):
        return [b[0] for b in self.bufs[self.front]]

    @property
    def s(self):
        return [b[1] for b in self.bufs[self.front]]

    @property
    def V(self):
        return [b[2] for b in self.bufs[self.front]]

    @property
    def d(self):
        return [b[3] for b in self.bufs[self.front]]

    def _streams(self, stream):
        cur = torch.cuda.current_stream(self.device)
        return cur, (stream if stream is not None else cur)

    @staticmethod
    def _event(s) -> torch.cuda.Event:
        e = torch.cuda.Event()
        e.record(s)
        return e

    def arrive(self, G_anc: Sequence[Optional[torch.Tensor]], stream=None, publish: bool = True) -> None:
        """An anchor gradient per matrix (None: no new gradient for that
        matrix, its EMA is kept): fold into M^anc and rebuild every basis, on
        `stream` (default: the current stream).  With publish=False the new
        basis waits in the back buffer, and corrections keep using the
        previous one until publish()."""
        if len(G_anc) != len(self.shapes):
            raise ValueError("one anchor gradient (or None) per matrix")
        if self._pending is not None:
            self.publish()
        cur, s = self._streams(stream)
        G = [None if g is None else g.contiguous() for g in G_anc]   # any copy is made on `cur`
        back = 1 - self.front
        if s != cur:
            s.wait_stream(cur)
        for e in (self._last_build, self._read[back]):
            if e is not None:
                s.wait_event(e)
        items = []
        for i, g in enumerate(G):
            it = dict(G_anc=g, M=self.M[i], out=self.bufs[back][i], ws=self.ws[i])
            if self.warm_start and self.arrivals > 0:
                it["V_warm"] = self.bufs[self.front][i][2]       # read only; the build writes `back`
            items.append(it)
        # matrix i of arrival a draws its random columns from seed + a * count + i
        sc_build_prior_batched(items, self.r, self.beta, self.tau, self.oversample, self.power_iters,
                               seed=self.seed + self.arrivals * len(self.shapes), dtype=self.dtype, stream=s)
        if s != cur:
            for g in G:
                if g is not None:
                    g.record_stream(s)
        self._last_build = self._written[back] = self._event(s)
        self.arrivals += 1
        self._pending = back
        if publish:
            self.publish()

    def publish(self) -> None:
        """Make the last build's basis the one corrections use (they wait for
        that build to finish)."""
        if self._pending is not None:
            self.front, self._pending = self._pending, None

    def prior(self, i: int):
        """(U, d, V) of matrix i in the basis the corrections use."""
        U, _, V, d = self.bufs[self.front][i]
        return U, d, V

    def _begin_correction(self, tensors, stream):
        cur, s = self._streams(stream)
        if s != cur:
            s.wait_stream(cur)
        for e in (self._written[self.front], self._last_correct):
            if e is not None:
                s.wait_event(e)
        return cur, s

    def _end_correction(self, tensors, cur, s):
        if s != cur:
            for t in tensors:
                if t is not None:
                    t.record_stream(s)
        self._last_correct = self._read[self.front] = self._event(s)

    def correct(self, G: Sequence[torch.Tensor], alpha: float, out: Optional[Sequence[torch.Tensor]] = None,
                stream=None):
        """G_proj = alpha G + (1 - alpha) G_filt for every matrix, with the
        current basis.  Returns the G_proj tensors (out, or new tensors)."""
        G = [g.contiguous() for g in G]
        if out is None:
            out = [torch.empty_like(g) for g in G]
        cur, s = self._begin_correction(G, stream)
        items = [dict(G=g, prior=self.prior(i), out=o, ws=self.cws[i]) for i, (g, o) in enumerate(zip(G, out))]
        sc_correct_batched(items, self.r, alpha, dtype=self.dtype, stream=s)
        self._end_correction(list(G) + list(out), cur, s)
        return list(out)

    def correct_adamw(self, G: Sequence[torch.Tensor], states: Sequence[tuple], alpha: float, lr: float,
                      step: int, norm_out: Optional[torch.Tensor] = None, stream=None, **hp) -> None:
        """The corrected AdamW step of every matrix (states: (W, m1, m2) fp32, in place)."""
        G = [g.contiguous() for g in G]
        cur, s = self._begin_correction(G, stream)
        items = [dict(G=g, prior=self.prior(i), ws=self.cws[i], state=tuple(st))
                 for i, (g, st) in enumerate(zip(G, states))]
        sc_correct_adamw_batched(items, self.r, alpha, lr, step=step, dtype=self.dtype, norm_out=norm_out,
                                 stream=s, **hp)
        self._end_correction(list(G) + [t for st in states for t in st] + [norm_out], cur, s)
