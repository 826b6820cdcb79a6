"""CPU oracle of MemDecay's retention step — TEST INFRASTRUCTURE ONLY.

Import it only from the test suite, the package entry's smoke check and the
benchmark's CPU-baseline leg.  The device path never imports it.
"""
from .memdecay import (Session, StepRecord, aligned_page_sizes, e4m3_decode, e4m3_encode,  # noqa: F401
                       quantise_block, select_pages,
                       session_from_workload, softmax, widen_bf16)
