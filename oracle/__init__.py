"""Plain fp64 CPU oracle for routed pattern-sparse causal attention prefill.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or link this
package: only the tests, the package's ``smoke()`` entry and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library (no kernels, headers, helpers or
tables) and is written from the paper's definitions:

* ``attention``  dense causal attention (Sec. 2.1, Eq. 1), masked attention with the
  minus-infinity semantics (Sec. 2.1), the omitted-mass certificate (Sec. 3.3, Eq. 5) and
  the relative output error (Sec. 4.2, Eq. 9);
* ``patterns``   token-exact key sets of the A-shape, vertical-slash and block-sparse
  families (Sec. 2.1, Sec. 3.1);
* ``probe``      the shared sampled-row probe and the block-mean estimator (Sec. 3.1,
  Sec. 3.2, Eq. 3);
* ``indices``    the candidate index rules (Sec. 3.1);
* ``coverage``   covered probe mass, subset disagreement, lower mass and risk (Sec. 3.2,
  Sec. 3.3, Eq. 4);
* ``router``     the greedy latency-constrained router with expand/fallback and grouping
  (Sec. 3.4, Eqs. 6-8, and the inference-procedure table).

Where the paper leaves a choice open the reading used is stated in the function's
docstring.  Parity of the probe sampling mix, budget grids and router constants is
"parity by definition of this reading": nothing in the paper pins their values.
"""
