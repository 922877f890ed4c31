"""CPU fp64 oracle of the Token Radius Attention hot path (test infrastructure).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package.  The GPU library never does, and the two share no code.

Parity status of every function: pinned by the CPU tests against closed forms,
invariants and brute force (see the test module for the oracle).  The paper
prints no worked numerical example, so no pin uses a value printed in the
paper; hand-derived fixtures live in the golden folder of the tests.
"""
from .tra_oracle import *  # noqa: F401,F403
from .tra_oracle import __all__  # noqa: F401
