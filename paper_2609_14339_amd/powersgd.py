"""PowerSGD state of one worker: the memory E, the factors P, Q and the
workspaces of a set of weight matrices, stepped by the library (the
data-parallel compressor the method is paired with: Sec. 3.3, App. J F3).

Ranks follow the compression ratio: r = floor(m n / (ratio (m + n))), at
least 1 and at most min(m, n, SC_KMAX); matrices of equal rank share one
library call.  Q starts Gaussian (seeded), E at zero.  Every operation is a
library call (psgd_step); this module only holds the buffers.
"""
from __future__ import annotations

from typing import List, Optional, Sequence, Tuple

import torch

from . import SC_KMAX, psgd_step, psgd_workspace


def rank_for_ratio(m: int, n: int, ratio: float = 64.0) -> int:
    r = int(m * n // (ratio * (m + n)))
    return max(1, min(r, m, n, SC_KMAX))


class PowerSGDState:
    def __init__(self, shapes: Sequence[Tuple[int, int]], ratio: float = 64.0, dtype=torch.bfloat16,
                 device="cuda", seed: int = 0, ranks: Optional[Sequence[int]] = None):
        self.shapes = [tuple(s) for s in shapes]
        self.dtype = dtype
        self.ranks = list(ranks) if ranks is not None else [rank_for_ratio(m, n, ratio) for m, n in self.shapes]
        gen = torch.Generator(device=device).manual_seed(seed)
        self.items = []
        for (m, n), r in zip(self.shapes, self.ranks):
            self.items.append(dict(E=torch.zeros(m, n, device=device), P=torch.zeros(m, r, device=device),
                                   Q=torch.randn(n, r, device=device, generator=gen),
                                   ws=psgd_workspace(m, n, r, dtype, device)))
        self.groups = {}
        for i, r in enumerate(self.ranks):
            self.groups.setdefault(r, []).append(i)

    def step(self, grads: Sequence[torch.Tensor], outs: Optional[Sequence[torch.Tensor]] = None,
             stream=None) -> List[torch.Tensor]:
        """One compressor step on every matrix: returns the decompressed
        gradients (outs, or new tensors; an out may be its grad)."""
        if outs is None:
            outs = [torch.empty_like(g) for g in grads]
        for r, idx in self.groups.items():
            items = [dict(self.items[i], G=grads[i], out=outs[i]) for i in idx]
            psgd_step(items, r, self.dtype, stream)
        return list(outs)

    def sent_elements(self) -> int:
        """Numbers a worker exchanges per step: m r + n r per matrix."""
        return sum(r * (m + n) for (m, n), r in zip(self.shapes, self.ranks))
