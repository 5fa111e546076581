"""CPU oracle of the paper's hot path: masking compressor and spectral corrector.

TEST INFRASTRUCTURE ONLY.  Plain, slow, obviously correct definitions written
from the paper (Sec. 3.1, Sec. 3.2, Alg. 1, App. E, App. F), used to check the
HIP library.  Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import it; the library never does, and the two share no
code.

Pins (tests run without a GPU) and their status:
  mask.*       pinned: published SplitMix64 / MurmurHash3 vectors, bijection and
               permutation brute force, subset-uniformity statistics,
               unbiasedness and variance of the rescaled mask (App. F), the
               paper's worked payload arithmetic (App. H), torch's bf16 rounding.
  spectral.*   pinned: closed forms for G = U S V^T, alpha = 1 identity,
               projector idempotence and self-adjointness at tau = 0,
               Lemma 1 (non-expansive) and Lemma 2 (noise contraction, Monte
               Carlo), EMA closed forms, SVD against eigh brute force.
  mask.bern_*  pinned (the per-entry draw is our specification): inclusion
               frequency per position, binomial row counts, independence of
               neighbouring entries, uniform patterns on a tiny row, keep = 1,
               App. F unbiasedness and variance (p / (1 - p)) h^2, layout.
  adamw.*      pinned: torch.optim.AdamW and torch.nn.utils.clip_grad_norm_ in
               float64 (independent library routines), the closed form of the
               first step from zero moments, clipping invariants, the norm
               identity the library clips with, planted-mistake checks.
  powersgd.*   pinned: numpy's Householder QR for the Gram-Schmidt step,
               dropped dependent columns (exact small case), exact
               reconstruction at rank <= r, least squares and Pythagoras for
               the output and memory, the rank-1 closed form, Eckart-Young
               (SVD) reached by the warm-started iteration, telescoping error
               feedback, brute-force rank for a compression ratio,
               planted-mistake checks.
"""
