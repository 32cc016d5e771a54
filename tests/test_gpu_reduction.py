"""Algorithm 2 (bit-precision level reduction) and the memory model
(Eq. 26-30) on the GPU against the oracle, on ResNet-18 (2 images, 16 x 16)
from the forward optimizer's 8-bit design.

Bit-exact: every trial (data structure, theta, fractional lengths, accuracy,
validity), every applied change, every candidate of Algorithm 1 inside the
trials, and the memory model; costs agree to a relative 1e-9 (fp64 sums in
different orders).  The run is capped at three changes, then the FC bias
(G2, 32 bits) runs one Reduce with its binary search at threshold 0."""
import pytest

from gpu_util import DEV, note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fx():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2203_12091_amd import fxpq
    return fxpq


def same_trace(a, b):
    assert len(a) == len(b)
    for (l1, d1, f1, c1), (l2, d2, f2, c2) in zip(a, b):
        assert (l1, d1, f1) == (l2, d2, f2)
        assert abs(c1 - c2) <= 1e-9 * max(abs(c2), 1e-30), (l1, d1, f1, c1, c2)


def test_reduction_matches_oracle(fx):
    from oracle import qparams as OQ
    from oracle import reduction as OR
    from paper_2203_12091_amd import qparams as GQ
    from paper_2203_12091_amd import reduction as GR
    note("reduction oracle resnet18 2x16 w8")
    ref = OQ.ForwardOptimizer("resnet18", batch=2, image=16, w_wl=8)
    want = ref.run()
    note("reduction gpu resnet18 2x16 w8")
    fo = GQ.ForwardOptimizer("resnet18", batch=2, image=16, device=DEV, w_wl=8)
    got = fo.run()
    assert got == {k: tuple(v) for k, v in want.items()}
    rr, rg = OR.QReduction(ref, 0.5, max_changes=3), GR.QReduction(fo, 0.5, max_changes=3)
    assert rg.nu == rr.nu and rg.clusters == rr.clusters
    n0 = len(ref.trace)
    note("reduction run oracle")
    fr = rr.run()
    note("reduction run gpu")
    fg = rg.run()
    assert fx.sync_status(fo.h) == 0
    assert rg.trials == rr.trials
    assert rg.changes == rr.changes and len(rg.changes) == 3
    assert fg == fr
    same_trace(fo.trace[n0:], ref.trace[n0:])
    assert rg.accuracy() == rr.accuracy()
    assert GR.memory_model(fo) == OR.memory_model(ref)
    # G2: the FC bias from 32 bits, binary search at threshold 0
    n1, t1 = len(ref.trace), len(rr.trials)
    note("reduction g2 reduce")
    sr = rr.reduce(rr.clusters[2][0], 0.0, 1)
    sg = rg.reduce(rg.clusters[2][0], 0.0, 1)
    assert sg == sr
    assert rg.trials[t1:] == rr.trials[t1:] and len(rr.trials) - t1 >= 4
    same_trace(fo.trace[n1:], ref.trace[n1:])
    assert fx.sync_status(fo.h) == 0
    fo.close()
