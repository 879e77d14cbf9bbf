"""Plain, slow fp64 CPU oracle for FAVOR attention (arXiv 2006.03555).

THIS PACKAGE IS TEST INFRASTRUCTURE. Only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import or call it. The product
path (``paper_2006_03555_amd``, the HIP library) never imports it and shares no
code, constant table or helper with it; the two meet only on the seeded host
arrays made by ``workloads.py``.

Modules
-------
philox   Philox4x64-10 counter-based generator (Salmon et al., SC'11) and the
         uniform / Box-Muller streams the orthogonal-random-feature draw uses.
favor    The method: ORF draw (Sec. 2.4), feature map (Sec. 2.3, Eqs. b, dqdk,
         qkprime), bidirectional FAVOR (Sec. 2.5, Algorithm 1), unidirectional
         FAVOR by sequential prefix aggregation (Sec. 2.5.1, Eq. cumsum; Sec. 2.6),
         the explicit L x L estimator and exact softmax attention (Sec. 2.1).
backward Gradients of both directions with respect to Q, K, V (and the causal
         state), the steps of Algorithm 1 / Eq. cumsum taken in reverse.
metrics  Parity metrics (row-relative error and a conditioning-aware error).

Every function is fp64 and follows the paper's order of operations; no blocking,
fusion or reordering beyond what the definitions state.
"""
from . import philox, favor, backward, metrics  # noqa: F401
