"""Plain CPU fp64 oracle of one PACI pipeline stage.

TEST INFRASTRUCTURE ONLY. The only code allowed to import, call or execute
anything in this package is ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py``. The product path (the HIP library and its
Python binding) never touches it, and this package shares no code with it.

Contents
--------
schedule  the stage event rule (Alg. 1), the canonical asynchronous 1F1B order,
          version stamps and the inconsistency bound (Eq. 2), plus a brute-force
          enumerator of every admissible interleaving.
model     LayerNorm, tanh-GELU, causal attention, the pre-LN GPT block, the
          embedding front and the LM-head/cross-entropy back, forward and
          backward, written out from their definitions in float64.
adamw     the decoupled-weight-decay Adam update the paper trains with.
stage     one stage's state (single parameter copy, fp32-style accumulator G,
          moments, counters) and the replay of an event list under the drift
          semantics of Eq. (1): saved activations come from the forward,
          parameters read in the backward are the current version.
pipeline  bubble-efficiency formulas (Eqs. 3-5) used only to pin the paper's
          printed numbers.
partition the memory-constrained stage partitioning problem and its
          infeasibility fallback, solved by exhaustive search.

Every function states the passage of the paper it follows. Precision is
float64 throughout; inputs that the GPU sees in bf16 are handed to the oracle as
the exact bf16 values.
"""
