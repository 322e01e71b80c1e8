"""CPU oracle of TreeFlash drafting: test infrastructure, never used by the library.

Only the tests, the entry module's smoke check and the benchmark's CPU-baseline
leg import this package.
"""
from .treeflash_oracle import *  # noqa: F401,F403
from .treeflash_oracle import __all__  # noqa: F401
