"""fp64 CPU oracle for the prefix-shared attention hot path.

TEST INFRASTRUCTURE ONLY: the test-suite, the smoke check and the benchmark's
CPU-baseline leg are the only code that may import or run anything here.  The
oracle shares no code with the GPU library (it reads inputs from the
``synthetic`` generator only) and the product path never routes through it.
"""
from .attention import (causal_attention, dense_group_reference,
                        three_phase_reference, group_loss)
from .compare import max_abs_rel, paper_pass_fraction

__all__ = ["causal_attention", "dense_group_reference", "three_phase_reference",
           "group_loss", "max_abs_rel", "paper_pass_fraction"]
