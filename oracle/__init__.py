"""TwinKV reference oracle -- TEST INFRASTRUCTURE ONLY.

Importable only from tests/, __graft_entry__.smoke() and bench.py's cpu_baseline
leg.  See twinkv_oracle.py for the definitions, citations and readings.
"""
from .twinkv_oracle import *  # noqa: F401,F403
from .twinkv_oracle import __all__  # noqa: F401
