"""CPU oracle of the CLEAR-MoE FFN forward (test infrastructure only).

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  It computes every step in IEEE double from the stored
inputs; see ``clearmoe_ref.c`` for the paper passage each function follows.
"""
from .ref import *  # noqa: F401,F403
