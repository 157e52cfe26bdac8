"""The compute accounting entry point (tasq_schedule_cost, host only) against
the oracle's accounting on every workload and step range, the paper's
printed Eff. W-bit -> Rel. BitOPs pairs, and its argument checks."""
import ctypes

import numpy as np
import pytest

import oracle
import paper_2608_03057_amd as T
from paper_2608_03057_amd import _lib, inputs

FIELDS = ("macs", "b_eff", "b_mean", "bitops", "rel_bitops", "rel_cycles_measured",
          "rel_cycles_as_a4")


def shapes(wl):
    return [(s.M, s.N, s.K) for s in wl.layers]


@pytest.mark.parametrize("cfg", range(5))
@pytest.mark.parametrize("act_bits", [4, 8, 16])
def test_matches_oracle_on_workloads(cfg, act_bits):
    wl = inputs.workload(cfg)
    table = inputs.b_table(wl).numpy()
    macs = [M * N * K for (M, N, K) in shapes(wl)]
    for t0, t1 in [(0, wl.T), (0, 1), (wl.T - 1, wl.T), (0, 0)]:
        got = T.schedule_cost(shapes(wl), table, wl.S, wl.T, t0, t1, act_bits)
        ref = oracle.schedule_cost(macs, table, wl.S, wl.T, t0, t1, act_bits)
        assert got["macs"] == ref["macs"] and got["bitops"] == ref["bitops"]
        for f in FIELDS:
            assert got[f] == pytest.approx(ref[f], rel=1e-12, abs=0), (cfg, t0, t1, f)


def test_printed_pair_5_91_to_0_74():
    """Layers of 9 and 91 MACs at 5 and 6 bits give Eff. W 5.91, and at A8
    the printed Rel. BitOPs 0.74 of the SVDQuant+TASQ W8A8 row."""
    c = T.schedule_cost([(1, 1, 9), (1, 1, 91)], [[5], [6]], 1, 1, 0, 1, 8)
    assert c["b_eff"] == pytest.approx(5.91, abs=1e-12)
    assert round(c["rel_bitops"], 2) == 0.74
    assert c["rel_cycles_measured"] == pytest.approx(5.91 / 8)


def test_rejects():
    L = _lib.lib()
    lay = (_lib.Layer * 1)()
    lay[0].M, lay[0].N, lay[0].K = 2, 3, 4
    tab = (ctypes.c_uint8 * 4)(8, 7, 6, 5)
    out = _lib.Cost()
    f = L.tasq_schedule_cost
    assert f(lay, 1, tab, 4, 20, 0, 20, 8, None) == _lib.TASQ_ERR_NULL
    assert f(lay, 1, tab, 4, 20, 0, 21, 8, ctypes.byref(out)) == _lib.TASQ_ERR_RANGE
    assert f(lay, 1, tab, 5, 4, 0, 4, 8, ctypes.byref(out)) == _lib.TASQ_ERR_RANGE
    assert f(lay, 1, tab, 4, 20, 0, 20, 0, ctypes.byref(out)) == _lib.TASQ_ERR_RANGE
    assert f(None, 1, tab, 4, 20, 0, 20, 8, ctypes.byref(out)) == _lib.TASQ_ERR_NULL
    bad = (ctypes.c_uint8 * 4)(8, 7, 9, 5)
    assert f(lay, 1, bad, 4, 20, 0, 20, 8, ctypes.byref(out)) == _lib.TASQ_ERR_BITS
    lay[0].K = -1
    assert f(lay, 1, tab, 4, 20, 0, 20, 8, ctypes.byref(out)) == _lib.TASQ_ERR_DIM
    assert f(None, 0, None, 4, 20, 0, 20, 8, ctypes.byref(out)) == _lib.TASQ_OK
    assert out.macs == 0.0
