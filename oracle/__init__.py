"""CPU oracle for the CompAct compressed linear layer — TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct fp64 (numpy) statement of what
the CompAct layer computes (forward Alg. 1, backward Alg. 2, Adam step Alg. 3 of
"CompAct: Compressed Activations for Memory-Efficient LLM Training", §3.2-§3.3),
plus an independent implementation of the projection streams (Philox4x32-10, a
fixed fp32 Box-Muller transform for the Gaussian, and the hashed signed draws of
the sparse Johnson-Lindenstrauss projection of the ablation, §5).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  It shares no code with the HIP path and the HIP path
never imports it: the product fails loudly when its HIP library is missing and
never falls back to anything here.

Modules
-------
pstream  : the P stream (seed, i, j) -> N(0,1) float32, and P = G/sqrt(r);
           the sparse JL stream S (integers), and P = S/sqrt(s).
compact  : Alg. 1-3 in fp64, the seed schedule and the Table 1 memory model.
"""
from . import pstream, compact  # noqa: F401
