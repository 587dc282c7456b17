"""CPU oracle for the perturbation-propagation sensitivity profile (RippleKV).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link or
execute this package: only the tests, the smoke check and the CPU-baseline leg of
the benchmark use it.  It shares no code with the HIP library (kernels, headers,
helpers, tables or generators); the only common module is ``fixtures``, which
draws seeded inputs and holds none of the method's arithmetic.

It is plain, slow and written to be checked by eye against the paper:

* ``philox``  -- the counter-based Gaussian noise epsilon of the Value perturbation
  (Section 4.3, Eq. value-perturbation), Philox4x32-10 + Box-Muller.
* ``model``   -- the Llama-style decoder the problem statement assumes
  (Section 4.1): embedding, RMSNorm, rotary Q/K, grouped-query causal attention,
  SwiGLU, final norm and LM head; clean pass with cached per-layer inputs.
* ``profile`` -- ReferencePredict, PerturbedPredict resumed from layer l,
  WindowKL and the calibration mean (Algorithm 1, profiling half; Eqs.
  value-perturbation, sample-response and layer-sensitivity).
* ``budgets`` -- min-max normalisation, exponential mapping, ClipNormalize and
  the integer budgets (Algorithm 1, allocation half; Section 4.4, Eqs.
  sensitivity-normalization, sensitivity-mapping, weight-normalization and
  layer-budget).

Floating point: the forward runs in a caller-chosen numpy dtype (float64 by
default, float32 for the large workloads); log-softmax and KL always run in
float64; the mapping uses Python floats.
"""

