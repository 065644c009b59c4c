"""CPU oracle for the AceSpec cloud-side tree-verify step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import anything from this package; the
product path (the HIP library and its Python binding) never does.

What it computes, in plain numpy float64, following the paper:

* ``model``  -- one forward pass of a Llama-style decoder over a batch of
  drafted token trees, each attending to its session's KV prefix and to its
  own ancestors only (tree attention mask, Section III-C), plus the
  plain-definition twin: a token-by-token causal decode along one root-to-node
  path.
* ``verify`` -- per tree row, the target distribution reduced to what the
  cloud returns downlink (Section III-B and Algorithm 1): temperature and
  top-p, the min(1, p/q) acceptance test, the residual max(0, p - q)
  resample, a bonus sample, the top-k sparse distribution; then the
  per-session path walk with the sibling-hit rule of Algorithm 1
  (w = (pi, x_resampled) looked up in the drafted tree).

Readings where the paper is silent are documented in the design notes of the
repository and in each function's docstring.  Pins: every function here is
checked by the CPU test suite against closed forms, invariants, brute-force
enumeration and an independent library implementation of the decoder.
"""
from . import model, verify  # noqa: F401
