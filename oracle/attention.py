"""Single-query softmax attention and the phase-2 window weights, in fp64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

* ``attend`` is ``Attn(Q_t, K_p + K[idx], V_p + V[idx])`` of Algorithm 1
  (section 4): the keys are the full prompt KV followed by the kept decode
  KV ("+" is concatenation), scores are ``scale * q.k`` with the usual
  ``scale = 1/sqrt(d)`` (the algorithm box omits the scale), and the output
  is the softmax-weighted sum of the value rows.
* ``window_weights`` is the phase-2 selection score ``softmax(Q_t K[idx]^T)``
  of Algorithm 1, normalised over the kept *window* keys only (the prompt is
  not part of ``K[idx]``).  The same scaled logits as the attention are used.
* ``select`` returns ``j* = argmin_j w[j]``.  For a KV head shared by several
  query heads (GQA, which the paper does not treat) the score of a window key
  is the sum of the group's window weights; at group size 1 this is the
  paper's per-head rule.  Ties go to the first (oldest) position, as
  ``argmin`` over the ascending window does.

Everything is computed in float64 from float64 copies of the inputs.
"""

from __future__ import annotations

import numpy as np


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


def softmax(s: np.ndarray) -> np.ndarray:
    """softmax over the last axis, with the maximum subtracted first."""
    s = _f64(s)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def logits(q, keys, scale: float) -> np.ndarray:
    """``scale * keys @ q`` -- one score per key row."""
    return float(scale) * (_f64(keys) @ _f64(q))


def attend(q, keys, values, scale: float):
    """Return ``(out, w)``: ``w = softmax(scale * keys @ q)`` and
    ``out = w @ values``.  ``keys``/``values`` are ``[n, d]`` with ``n >= 1``."""
    keys, values = _f64(keys), _f64(values)
    if keys.shape[0] == 0:
        raise ValueError("attention over an empty key set")
    w = softmax(logits(q, keys, scale))
    return w @ values, w


def window_weights(q, window_keys, scale: float) -> np.ndarray:
    """Phase-2 score of Algorithm 1: softmax of the query's logits over the
    kept window keys only."""
    return softmax(logits(q, window_keys, scale))


def select(q_group, window_keys, scale: float):
    """``j* = argmin_j sigma_j`` with ``sigma_j = sum_h w_h[j]`` over the
    query heads ``h`` in ``q_group`` (shape ``[g, d]``).  Returns
    ``(j_star, sigma)``."""
    q_group = _f64(q_group)
    if q_group.ndim == 1:
        q_group = q_group[None, :]
    sigma = np.zeros(_f64(window_keys).shape[0])
    for q in q_group:
        sigma += window_weights(q, window_keys, scale)
    return int(np.argmin(sigma)), sigma
