"""CPU oracle of the Skip-Conv layer -- test infrastructure, not part of the product path.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may import it.
"""
from .skipconv_oracle import *  # noqa: F401,F403
