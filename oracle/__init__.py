"""CPU oracle of the FlashDecoder decoder forward -- test infrastructure only.

Importable by tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg;
never by the product path.
"""
from .decoder import *  # noqa: F401,F403
