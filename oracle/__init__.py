"""CPU oracle for optimizer fusion (arXiv 2104.00237) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 numpy implementation of what the fused training path
computes, written from the paper:

  * eager training: forward of every operator, then backward accumulating
    every gradient, then one optimizer step over every parameter
    (Section 1 and Fig. 1(b));
  * forward-fusion (Appendix B.1, Alg. 2) and backward-fusion (Appendix B.2,
    Alg. 3, with the dependency rule stated after Alg. 3);
  * the optimizer policies of Appendix A (Alg. 1, gradient descent and
    momentum) plus Adam / AdamW as used by the workloads, and Adagrad,
    RMSprop and Adadelta, the other optimizers of the comparison in Fig. 7;
  * global-norm gradient clipping (the global-information step forward-fusion
    permits, Appendix B.1, Table 1) and parameters shared by two layers (the
    `updated` flag of Alg. 2 and `count` of Alg. 3);
  * the depthwise 3x3 convolution of the small-parameter layers (MobileNetV2,
    Fig. 3 and Table 2), pinned to the full convolution's direct loops.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product (the HIP library and its Python binding)
never imports it, and it imports nothing from the product.  Both read their
inputs from the separate `workloads` package.

Parity status per function is stated in each module's header; whole K-step
trajectories are pinned transitively (component pins + the ordering
invariant), since the paper prints no worked numeric example.
"""
from .train import (run, new_model, ambiguous_relu_decisions, candidate_steps,  # noqa: F401
                    DecisionSearch)
