"""CPU oracle for PaDoc tree attention (TEST INFRASTRUCTURE ONLY).

Importable only by the tests, the smoke check and the benchmark's CPU-baseline
leg.  See :mod:`oracle.dense` for the definitions it follows.
"""
from .dense import *  # noqa: F401,F403
from .dense import __all__  # noqa: F401
from .backward import masked_attention_backward, tree_attention_backward  # noqa: F401,E402
