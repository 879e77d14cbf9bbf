"""The measurement entry points the benchmark relies on: the microbenchmark
probes behind the measured peaks (favor_probe) and the per-launch event timing
(favor_timing_*). Timing counts exactly the launches of the calls made while it
is enabled; a reset clears it.
"""
import ctypes

import numpy as np
import pytest

from helpers import to_dev
from oracle import favor

pytestmark = pytest.mark.gpu

S64 = 64 ** -0.25


def _fv():
    import paper_2006_03555_amd as fv
    return fv


@pytest.mark.parametrize("kind", [0, 1, 2])
def test_probe_runs(kind):
    import torch
    fv = _fv()
    sink = torch.zeros(512, dtype=torch.float32, device="cuda")
    st = torch.cuda.current_stream()
    assert fv.lib().favor_probe(kind, 2, ctypes.c_void_p(sink.data_ptr()),
                                ctypes.c_void_p(st.cuda_stream)) == 0
    torch.cuda.synchronize()
    assert torch.isfinite(sink).all()


def test_timing_counts_the_launches_of_a_call():
    import torch
    fv = _fv()
    W, b = favor.orf_draw(3, 2, 128, 64)
    rng = np.random.default_rng(4)
    q, k, v = (to_dev(rng.standard_normal((1, 2, 300, 64)).astype(np.float32) * s, "bf16")
               for s in (S64, S64, 1.0))
    args = (q, k, v, to_dev(W.astype(np.float32)), to_dev(b.astype(np.float32)), S64)
    fv.attn_bidir(*args)          # first call outside the timed window
    torch.cuda.synchronize()
    fv.timing_reset()
    fv.timing_enable(True)
    fv.attn_bidir(*args)
    fv.timing_enable(False)
    fv.attn_causal(*args)         # not counted
    t = fv.timing_read()
    counted = {name: v for name, v in t.items() if v[1] > 0}
    assert set(counted) == {"k_kside", "k_finalize", "k_qside"}, counted
    for name, (ms, n) in counted.items():
        assert n == 1 and ms > 0.0, name
    fv.timing_reset()
    assert all(n == 0 for _, n in fv.timing_read().values())
