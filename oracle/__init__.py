"""CPU oracle of the compressed-KV path (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package; the GPU path never does.
"""
from .fdkv_oracle import *  # noqa: F401,F403
from . import fdkv_oracle as core  # noqa: F401
