"""Q-Mean auxiliary (Algorithm 1, the mu step and the score correction;
Section 4.6; Appendix C, "Q-Mean GEMV and coordinate consistency").

Test infrastructure: only the tests, the smoke check and the benchmark's CPU
baseline use this package.

The mean of each smoothed query row over the head dimension is removed before
HIF4 quantization, and the scores get the product of that mean with the sum
of the smoothed key's channels back, so that in exact arithmetic
Q_z K~^T + mu * sum_c K~ = Q~ K~^T.  Both sums run over the channels of one
(token, head) row; the correction uses the smoothed key K~ (the coordinate
frame of the quantized product), not K.

Readings fixed here (the paper names the operation but not its rounding):
  * mu_i = fp16(sum_c q~_ic / D): the sum of the fp16 values is exact (float64
    holds any sum of at most 2^11 fp16 values exactly) and the quotient is
    rounded once to fp16 (mu is an FP16 quantity of the GEMV);
  * Q_z = fp16(q~ - mu): the exact difference rounded once;
  * kappa_j = fp32(sum_c k~_jc): the exact sum rounded once to fp32;
  * the correction mu_i * kappa_j is added to the fp32 score accumulator
    after the group terms (Algorithm 1 adds it after the product), the exact
    product with one rounding, and is then scaled by c with the rest of the
    score: S2 = fp16(fp32(fp32(S_acc + mu_i*kappa_j) * c)).  Scaling it with
    the rest of S is what the identity above requires (Algorithm 1 writes the
    correction after the division by sqrt(d), which only holds once the
    correction carries the same scale).
"""
from __future__ import annotations

import numpy as np

from .fparith import fma_f32


def token_mean(q_tilde):
    """mu = fp16(exact sum over the last axis / D) of fp16 values."""
    x = np.asarray(q_tilde, np.float16).astype(np.float64)
    return (x.sum(axis=-1) / x.shape[-1]).astype(np.float16)


def zero_mean(q_tilde, mu):
    """Q_z = fp16(q~ - mu), mu broadcast over the last axis."""
    a = np.asarray(q_tilde, np.float16).astype(np.float64)
    b = np.asarray(mu, np.float16).astype(np.float64)[..., None]
    return (a - b).astype(np.float16)


def key_sums(k_tilde):
    """kappa = fp32(exact sum over the last axis) of fp16 values."""
    return np.asarray(k_tilde, np.float16).astype(np.float64).sum(axis=-1).astype(np.float32)


def add_correction(acc, mu, kappa):
    """fp32(acc[i, j] + mu_i * kappa_j): the exact product (fp16 times fp32)
    added to the fp32 score accumulator with one rounding."""
    return fma_f32(np.asarray(mu, np.float16).astype(np.float32)[:, None],
                   np.asarray(kappa, np.float32)[None, :], acc)
