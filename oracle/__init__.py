"""Float64 CPU oracle for the JARQ refinement sweep.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the C-ABI library and
its Python binding) imports, links or calls this package; only the tests, the
smoke check and the CPU-baseline leg of the benchmark do.  It shares no code,
constants or helpers with the HIP path.

Modules
-------
jarq      The method in the Hessian form F_j = (w_j - what_j)^T H (w_j - what_j),
          float64, vectorised over rows (rows are independent, Sec. 3.3).
qrform    The paper's own least-squares form with A = [X; nu I], thin QR of
          each group block and v = U_i^T y / s (eqs. (3), (7)-(10)); used on
          small layers where X is available to pin the Hessian form.
replay    Teacher-forced re-evaluation of one code sweep conditioned on the
          decisions of another implementation (parity protocol).
hosts     Round-to-nearest host, and the GPTQ-style sequential-compensation
          host used for the wide-MLP layer (written from the GPTQ recursion).
hessian   The calibration Hessian H = X~^T X~ + nu^2 I (App. E.1) from
          chunks of tokens, with optional relative damping.
qep       The propagation-corrected weights of the mixed target (App. E.5).
post      After refinement: canonical positive scales (App. E.3), dequantized
          weights, packed codes, activation ordering.
"""

from . import jarq, qrform, replay, hosts, hessian, qep, post  # noqa: F401
