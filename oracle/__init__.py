"""CPU oracle (float64 numpy) for compiled structured-sparse decode.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py``, never by the product library or its binding.

* ``reference``: the oracle proper (closure, zero-masked dequantised layer, decode, prefill,
  stack, FLOP and byte ledgers);
* ``compact``: the same layer from physically compacted panels (mask-as-zero invariant and
  byte-exact panel checks);
* ``dense``: a textbook dense layer with no mask logic (all-kept invariant);
* ``scalar``: pure-Python loops for tiny shapes (brute-force cross-check).
"""
from . import reference, compact, dense, scalar  # noqa: F401
from .reference import *  # noqa: F401,F403
