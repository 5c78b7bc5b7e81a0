"""CPU oracle (float64) for budgeted in-place KV-cache repair.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it; the library never does,
and the oracle shares no code with the HIP path.
"""
from .decoder import (DenseWeights, attend, empty_cache, layer_forward, prefill, repair,
                      repaired_set, rms_norm, rope, silu, transplant)
from .select import SplitMix64, pool, select_edit_local, select_random, select_to_boundary
from . import scoring

__all__ = [
    "DenseWeights", "attend", "empty_cache", "layer_forward", "prefill", "repair",
    "repaired_set", "rms_norm", "rope", "silu", "transplant",
    "SplitMix64", "pool", "select_edit_local", "select_random", "select_to_boundary", "scoring",
]
