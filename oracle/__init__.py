"""CPU oracle for the MoARa optimizer hot path -- TEST INFRASTRUCTURE ONLY.

Imported only by tests/, __graft_entry__.smoke() and bench.py's CPU-baseline
leg. The product path never imports, links or executes anything here, and this
package imports nothing from the product package.
"""
from .moara_oracle import *  # noqa: F401,F403
from . import moara_oracle  # noqa: F401
