"""Rounding bounds of the fp32 selection, used to judge near ties.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

The phase-2 argmin of Algorithm 1 (section 4) is a discrete decision taken on
floating-point scores.  The oracle computes the scores exactly (fp64 from the
exact inputs); a device computes them in fp32.  When two window keys score
within the device's rounding error of each other, either pick is a correct
execution of the rule.  This module bounds that error from the arithmetic
the device performs, so a test can accept a different pick only when it is
inside the bound (and then the oracle adopts the device's pick).

The fp32 computation bounded here, per query head ``h`` of a KV head and
window key ``j``:

1. logit ``s_hj = fl(sc * fl(q_h . k_j))``: a dot product of length ``d`` in
   fp32 with any summation order (each product of two bf16 or E4M3-derived
   values is exact in fp32), then one multiply by the fp32 scale ``sc``
   (for fp8 caches ``sc`` is itself the rounded product of the softmax scale
   and the K scale).  Error at most ``gamma_d * scale * sum_i |q_i k_i|``
   plus ``3u |s|`` with ``u = 2^-24`` (standard forward error analysis of
   recursive or tree summation).
2. group size 1: the argmin is taken on the logits themselves.
3. group size ``g > 1``: ``m_h = max_j s_hj``; ``e_hj = exp2(fl(L *
   fl(s_hj - m_h)))`` with ``L`` the fp32 value of ``log2 e`` and the
   hardware base-2 exponential, whose relative error is taken to be at most
   ``EXP2_REL`` (two units in the last place); ``Z_h`` the fp32 sum of the
   ``e_hj`` over the window (a tree of depth at most
   ``ceil(n / 64) + 6``), its reciprocal (correctly rounded division,
   error at most ``u``) and the products ``w_hj = fl(e_hj * (1 / Z_h))``;
   ``sigma_j`` the fp32 sum of the ``g`` weights.

Every bound below is rigorous, not first order (it keeps ``exp`` and
``gamma`` forms rather than linearising), and bounds the absolute error of
the fp32 ``sigma_j`` against the exact ``sigma_j`` of the same inputs.
"""

from __future__ import annotations

import math

import numpy as np

U = 2.0 ** -24                 # unit roundoff of fp32
EXP2_REL = 2.0 ** -22          # relative error allowed for the hardware exp2


def gamma(n: int) -> float:
    """``gamma_n = n u / (1 - n u)``."""
    return n * U / (1 - n * U)


def dot_band(q, keys, scale: float) -> np.ndarray:
    """Bound of the fp32 dot-product error per key, times the scale:
    ``gamma_d * scale * sum_i |q_i k_i|``."""
    q = np.asarray(q, np.float64)
    keys = np.asarray(keys, np.float64)
    return gamma(q.shape[-1]) * abs(scale) * (np.abs(keys) @ np.abs(q))


def logit_band(q, keys, scale: float) -> np.ndarray:
    """Bound of ``|fp32 logit - exact logit|`` per key (step 1): the dot
    product's error, plus three roundings of the scale path (the fp32 value
    of the softmax scale, its product with an fp8 K scale, and the final
    multiply), each relative ``u``."""
    s = float(scale) * (np.asarray(keys, np.float64) @ np.asarray(q, np.float64))
    return (dot_band(q, keys, scale) + 3 * U * np.abs(s)) * (1 + 8 * U)


def score_bounds(q_group, window_keys, scale: float):
    """Exact selection scores of the window keys and a bound of the fp32
    path's error on each.

    Returns ``(score, err)``: for one query head the exact logits and
    ``logit_band``; for a group the exact ``sigma_j`` (sum of the group's
    window softmaxes) and the bound of steps 1-3."""
    qg = np.atleast_2d(np.asarray(q_group, np.float64))
    keys = np.asarray(window_keys, np.float64)
    n = keys.shape[0]
    if qg.shape[0] == 1:
        s = float(scale) * (keys @ qg[0])
        return s, logit_band(qg[0], keys, scale)
    sigma = np.zeros(n)
    err = np.zeros(n)
    depth = -(-n // 64) + 6
    for q in qg:
        s = float(scale) * (keys @ q)
        beta = logit_band(q, keys, scale)
        x = np.abs(s - s.max()) + beta + beta.max()      # |computed s - computed max| bound
        # log-relative error of each exp: the logit error (the max's error
        # cancels in the normalisation but is counted once more here), the
        # subtraction and the two roundings in the exponent's argument
        # (relative 3u of |x|), and the exp2 itself.
        eta = beta + 3 * U * x * (1 + 1e-6) + -math.log1p(-EXP2_REL)
        H = eta.max()
        w = np.exp(s - s.max())
        w /= w.sum()
        # weight ratio computed / exact within exp(+-lam)
        lam = eta + H - math.log1p(-gamma(depth)) - 2 * math.log1p(-U)
        sigma += w
        err += w * np.expm1(lam)
    # the fp32 sum over the group
    g = qg.shape[0]
    err = err + gamma(g - 1) * (sigma + err)
    return sigma, err


def within_tie_band(q_group, window_keys, scale: float, j_gpu: int, j_ref: int) -> bool:
    """Is the device's argmin ``j_gpu`` a correct pick?  True when it equals
    the oracle's ``j_ref``, or when its exact score exceeds the minimum by no
    more than the two keys' fp32 error bounds together (so the fp32 scores
    can order them either way).  The device breaks exact ties towards the
    smaller index, which the bound covers too."""
    if j_gpu == j_ref:
        return True
    score, err = score_bounds(q_group, window_keys, scale)
    if not (0 <= j_gpu < len(score)):
        return False
    slack = err[j_gpu] + err[j_ref] + 4 * np.finfo(np.float64).eps * max(1.0, abs(score).max())
    return bool(score[j_gpu] - score[j_ref] <= slack)
