"""CPU oracle of MemDecay's retention step — TEST INFRASTRUCTURE ONLY.

Import it only from the test suite, the package entry's smoke check and the
benchmark's CPU-baseline leg.  The device path never imports it.
"""
from .memdecay import (Session, StepRecord, aligned_page_sizes, quantise_block, select_pages,  # noqa: F401
                       session_from_workload, softmax, widen_bf16)
