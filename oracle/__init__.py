"""CPU oracle for the linear-layer online prefill (test infrastructure only).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It shares no code with the GPU library.
"""
from .core import (gdn_scan, gdn_transition, ssd_scan, ssd_log_decay, init_single,
                   compose_gdn, compose_ssd, gdn_decode, ssd_decode, load)
from .gather import gather_rows, gather_selected
from .bf16 import round_bf16
from .diagnostic import mismatch_recursion, rel_error

__all__ = ["gdn_scan", "gdn_transition", "ssd_scan", "ssd_log_decay", "init_single",
           "compose_gdn", "compose_ssd", "gdn_decode", "ssd_decode", "load", "gather_rows", "gather_selected",
           "round_bf16", "rel_error", "mismatch_recursion"]
