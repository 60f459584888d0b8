"""CPU oracle of the Gated VLA-Cache control step.  TEST INFRASTRUCTURE ONLY.

This package is the slow, plain reference that the HIP path is checked
against.  Only the tests, the smoke entry point and the benchmark's CPU
baseline leg may import it; the product path never does.  It shares no code
with the HIP library: it receives the same seeded inputs (from `synth`) and
recomputes everything with NumPy in float64, by default one token row at a
time, so a row's result never depends on which other rows are computed
alongside it.  At the 7B shape the tests run it in its batched mode, where
each projection and each head's attention is one library matrix product
over the recomputed rows (pinned against the row-at-a-time form and the
Hugging Face forward).

Contents (each function cites the passage it follows):
  patches  - Stage 1 static-patch detection (Sec. III-B) and the per-layer
             reuse proportion (Stage 3, applied).
  llama    - the Llama-2 decoder block (Sec. V-A names the backbone).
  margin   - the top-1/top-2 margin (Eq. 1) and the gate test of Alg. 1.
  vla      - the control step state machine of Alg. 1.
  flops    - the per-step compute accounting of Tables I-II.

Parity status: every function here is pinned by tests under tests/ against
closed forms, invariants, brute force or library routines, except the three
readings the paper leaves open (per-layer reuse base and order, token order,
hidden state of a reused token), which are pinned only by the invariants
they must satisfy ("parity unpinned" beyond those).
"""
