"""CPU oracle for the pruned RNN-T loss (Kuang et al., arXiv 2206.13236).

TEST INFRASTRUCTURE ONLY. This package is a plain, slow, fp64 NumPy
restatement of what the paper defines. Only the test suite, the smoke check
in ``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import
it. The product package (``paper_2206_13236_amd``) never imports, links or
runs anything here, and nothing here imports the product: the two share no
code. Inputs come from the separate ``workloads`` generator, which holds none
of the loss arithmetic.

Every public function names the passage of the paper it follows. Where the
paper is silent or ambiguous the reading taken is stated in the docstring.
"""
from .rnnt import (  # noqa: F401
    NEG_INF,
    log_add,
    log_normalizer,
    trivial_joiner_logprobs,
    lattice_forward_backward,
    lattice_loss,
    trivial_joiner_grad,
    pruning_window_scores,
    raw_pruning_bounds,
    monotonic_lower_bound,
    adjust_pruning_bounds,
    prune_ranges,
    joiner_hidden,
    pruned_joiner_logits,
    pruned_joiner_logprobs,
    pruned_loss,
    pruned_joiner_grad,
    full_joiner_logprobs,
    full_joiner_loss,
    simple_stage,
    smoothed_joiner_logprobs,
    smoothed_simple_stage,
    pruned_stage,
)
