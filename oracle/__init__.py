"""Plain, slow CPU oracle for conv_einsum (arXiv 2401.03384).

TEST INFRASTRUCTURE.  Only the test-suite, the package smoke check and the
benchmark's CPU-baseline leg may import this package.  The HIP product path
never imports, links or executes anything here, and nothing here imports the
product path.

Everything is float64 NumPy (Python ints for costs) written from the paper:

  notation   conv_einsum strings (Section 2.2, Appendix A.3) and size binding
             (Appendix A, sizes of non-convolved modes must agree; Appendix B,
             'Convolution Varieties': the larger size is the feature side)
  cost       tnn-cost of a pairwise step (Appendix B, the contraction, batch,
             outer-product and convolution cost equations) and the training
             variant cost(f)+cost(g1)+cost(g2) (Appendix B, 'Modification of
             the cost model for training')
  sequencer  brute-force search over every pairwise evaluation tree
             (Section 3.2, optimal sequencer) plus the left-to-right baseline
  evaluate   the plain definition of the result (direct sums), the pairwise
             evaluation along any tree (Section 3.1 atomic operations), and the
             reconstructed-dense-kernel evaluation
  gradients  reverse-mode gradients along a tree (Appendix B, g1 / g2) and via
             the reconstructed dense kernel

Convolution convention (readings of the paper, listed with the design notes):
cross-correlation, stride 1, zero 'same' padding with floor((K-1)/2) zeros
before and K-1-floor((K-1)/2) after; the output keeps the feature size.
"""
from .notation import Expr, parse, bind
from .cost import step_cost, kept_labels, label_size, tree_cost, step_costs
from .sequencer import (all_trees, optimal_tree, left_to_right_tree, leaves,
                        post_order_steps, count_trees, intermediate_size, max_intermediate,
                        checkpoint_choice)
from .evaluate import eval_definition, eval_pairwise, eval_dense, dense_kernel
from .gradients import grads_pairwise, grads_dense

__all__ = [
    "Expr", "parse", "bind", "step_cost", "kept_labels", "label_size",
    "tree_cost", "step_costs", "all_trees", "optimal_tree", "left_to_right_tree",
    "leaves", "post_order_steps", "count_trees", "intermediate_size", "max_intermediate",
    "checkpoint_choice",
    "eval_definition",
    "eval_pairwise", "eval_dense", "dense_kernel", "grads_pairwise", "grads_dense",
]
