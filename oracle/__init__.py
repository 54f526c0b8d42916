"""Slow, plain fp64 CPU reference of the large-sparse-target output-layer step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link or
execute anything in this package: only the test suite, the smoke check of the
entry module and the CPU-baseline leg of the benchmark use it.  It shares no
code with the GPU library; both sides receive their inputs from the `synth`
generators, which hold none of the method's arithmetic.

Modules
  explicit  the plain definition: W kept explicit, O(Dd) per example
            (sections 2.3, 3.1 and 3.2 of the paper, and its loss-family
            extension in section 3.6 for the spherical softmax, in the
            (o_c^2 + eps) form and in the shifted (o_c + eps)^2 form the
            section prints).
  factored  the paper's factored algorithm in fp64 (Algorithm 1, the minibatch
            algorithm of Appendix A, the pristine restore of Appendix C), used
            only to check the paper's identities against the explicit
            definition: W = VU, Q = W^T W, U (U^{-T})^T = I.
  stabilize Appendix C's correction of out-of-range singular values of U
            (fix-singular-value, with a full SVD or with power iterations),
            and the recomputation of U^{-T}.
  input_layer  the sparse input layer of section 2.2 (forward A = X W_in and
            the update of the rows of W_in the inputs refer to).

Pin status (what fixes each function other than itself) is listed in each
function's docstring; the only function without a pin by the paper is the
minibatch forms of the two spherical-softmax factored steps, which are pinned
by the explicit definition (itself pinned by closed forms, finite differences
and the normalisation of the class probabilities) instead.
"""
from . import explicit, factored, input_layer, stabilize  # noqa: F401
