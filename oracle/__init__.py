"""CPU oracle for diagonal-aware sparse decode attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code with the
HIP library (``paper_2609_19702_amd``): no kernels, headers, helpers, tables
or pre/post-processing.  The only module both sides read is the seeded input
generator ``paper_2609_19702_amd.synth``, which holds none of the method's
arithmetic.

What it computes, in plain slow fp64 (paper section 4, "Diagonal-Aware
Sparse Attention", Algorithm 1 and the "Detailed explanation" paragraph):

* ``alg1``      -- Algorithm 1's selection state, step by step: the
                   ``skip_idx`` list of absolute decode positions, shifted by
                   +1 every step, the window ``[max(0, t-N_r) .. t]``, the
                   eviction of ``K[t-N_r]`` in phase 3 and the phase-2
                   argmin append.  The argmin is supplied by the caller so the
                   same code runs with scripted, random or attention-derived
                   choices.
* ``attention`` -- single-query softmax attention over the prompt KV plus the
                   kept decode KV (``Attn(Q_t, K_p + K[idx], V_p + V[idx])``),
                   and the phase-2 window weights ``softmax(Q_t K[idx]^T)``
                   with their argmin.
* ``step``      -- one decode step (and whole trajectories) for one request,
                   per KV head, in diagonal or dense mode.
* ``params``    -- the parameter rules of the "Parameter selection"
                   paragraph and the sparsity definition of section 5.1.
* ``fp8``       -- exact decoding of an fp8 (OCP E4M3) KV cache with per-
                   (request, KV head) scales, the KV quantization the paper
                   calls orthogonal to its method (section 6).
* ``coracle``   -- the same Algorithm 1 and decode step restated in plain C
                   (``oracle/c/dsa_oracle.c``, fp64, OpenMP over KV heads),
                   for long selection histories and the timed CPU baseline;
                   pinned to the Python oracle and the worked example.
* ``tieband``   -- bounds of the fp32 rounding of the phase-2 scores, which
                   decide when a device's different argmin is still a
                   correct pick (a near tie); pinned by simulating the fp32
                   arithmetic it bounds.

Parity status: every function is pinned in ``tests/test_oracle_*.py`` except
the GQA aggregation of the selection weights (one skip set per KV head, score
= sum of the group's window softmaxes), which the paper does not define; its
reduction to the paper's per-head rule at group size 1 is pinned, the rest is
"parity unpinned".
"""

from . import alg1, attention, fp8, params, step, tieband  # noqa: F401
