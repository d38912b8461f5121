"""fp64 CPU oracle for the output-layer training step -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check of the package entry file and the CPU
baseline leg of the benchmark may import this package.  The product path (the
HIP library and its Python binding) never imports, calls or links it, and the
oracle shares no code, table or helper with that path.

  dense     -- the plain definition: an explicit D x d matrix W, the full output
               O = W H, the loss, its gradient with respect to H and the
               gradient-descent update of W (sections 2.3 and 4 of the paper).
  factored  -- the paper's factored algorithms (Algorithm 3 and Algorithm 4 with
               V, U, U^{-T} and Q) in fp64, used to check the paper's algebra
               against the dense definition and to expose the intermediates
               (H^, G, Z^, M, the Woodbury matrices, P) when a GPU kernel has to
               be examined step by step.
  stabilize -- section 5: the pristine restore, the recomputed U^{-T}, power
               iteration for the extreme singular values of U, Algorithm 5's
               fix-singular-value and the stabilisation loop around them.

All inputs are float64 upcasts of the float32 arrays the GPU receives.
"""
from .dense import (dense_targets, dense_step, spherical_softmax_step, squared_error_step,
                    taylor_softmax_step)
from .factored import FactoredState, factored_init, factored_step

__all__ = [
    "dense_targets", "dense_step", "squared_error_step", "spherical_softmax_step",
    "taylor_softmax_step",
    "FactoredState", "factored_init", "factored_step",
]
