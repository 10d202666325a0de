"""CPU oracle for the Pruned CTC head-and-loss path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports, calls or
links anything in this directory; only the tests, the smoke check of the build
entry point and the CPU-baseline leg of the benchmark may use it.  It shares no
code with the HIP path: it is a plain, slow, fp64 NumPy rendering of the
paper's definitions, written so that it can be checked against the paper by eye.
"""
from .prunedctc_oracle import (  # noqa: F401
    OracleError,
    PCTC_OK, PCTC_EINVAL, PCTC_ELABEL, PCTC_ELENGTH,
    STATUS_OK, STATUS_NOT_ALIGNABLE, STATUS_NONFINITE,
    beam_round_tol,
    validate,
    union_remap,
    log_normalizer,
    selected_logprobs,
    extended_labels,
    ctc_utterance,
    ctc_from_scores,
    discarded_mass,
    head_backward,
    head_backward_rows,
    grouped_logprobs,
    grouped_gradient,
    grouped_backward,
    fwd_bwd,
    ctc_collapse,
    greedy_decode,
)
