"""fp64 CPU oracle for IPPD decode-step and prefill attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the CPU-baseline leg of the benchmark may import or call anything here.  The
GPU library never does, and this package imports nothing from the GPU
library: the two share only the seeded input generator in ``workload``.

Every function is plain numpy in float64 and cites the passage of the paper
it follows (Intra-Prompt Parallel Decoding, arXiv 2609.05707).
"""
from .ippd import (  # noqa: F401
    INT_MAX,
    inv_freq,
    rope,
    attend,
    standard_prompting_question,
    KVState,
    Instructions,
    decode_step_standard,
    stacked_prompt_step,
    build_stacked_metadata,
    mask_predicates,
    decode_run,
)
from . import prefill  # noqa: F401,E402
