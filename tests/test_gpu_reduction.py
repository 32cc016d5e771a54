"""Algorithm 2 (bit-precision level reduction) and the memory model
(Eq. 26-30) on the GPU against the oracle, on ResNet-18 (2 images, 16 x 16)
from the forward optimizer's 8-bit design.

Bit-exact: every trial (data structure, theta, fractional lengths, accuracy,
validity), every applied change, every candidate of Algorithm 1 inside the
trials, and the memory model; costs agree to a relative 1e-9 (fp64 sums in
different orders).  The run is capped at three changes, then the FC bias
(G2, 32 bits) and two Scale parameters of the 512-channel layers (G2, 16 and
32 bits) run Reduce with its binary search at threshold 0."""
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
    # G2 holds the Scale parameters too (Eq. 22): the first two members of
    # the 512-channel sub-cluster (aleph_1 from 16 bits, aleph_2 from 32)
    sub_r, sub_g = rr.clusters[2][1][:2], rg.clusters[2][1][:2]
    assert sub_r == sub_g and [d for _, d in sub_r] == ["s1", "s2"]
    n2, t2 = len(ref.trace), len(rr.trials)
    note("reduction g2 scale reduce")
    assert rg.reduce(sub_g, 0.0, 1) == rr.reduce(sub_r, 0.0, 1)
    assert rg.trials[t2:] == rr.trials[t2:] and len(rr.trials) - t2 >= 6
    same_trace(fo.trace[n2:], ref.trace[n2:])
    assert fx.sync_status(fo.h) == 0
    fo.close()


@pytest.mark.parametrize("flw", [32, 16])
def test_wide_first_last_layers_match_oracle(fx, flw):
    """The paper's initial design with wide first / last layers (the input,
    the first and last weights and the last layer's input at 32 bits, as the
    paper starts them, and at 16; wide C-Blocks on the GPU): the forward
    optimizer, two changes of Algorithm 2, then the binary searches of the
    wide input and FC weights from their initial word length."""
    from oracle import qparams as OQ
    from oracle import reduction as OR
    from paper_2203_12091_amd import qparams as GQ
    from paper_2203_12091_amd import reduction as GR
    note("wide first/last oracle resnet18 2x16", flw)
    ref = OQ.ForwardOptimizer("resnet18", batch=2, image=16, w_wl=8, first_last_wl=flw)
    want = ref.run()
    note("wide first/last gpu resnet18 2x16", flw)
    fo = GQ.ForwardOptimizer("resnet18", batch=2, image=16, device=DEV, w_wl=8, first_last_wl=flw)
    got = fo.run()
    assert got == {k: tuple(v) for k, v in want.items()}
    assert got[("input", "a")][0] == flw and got[("fc", "w")][0] == flw
    same_trace(fo.trace, ref.trace)
    assert fo.top1_agreement() == ref.top1(ref.q[ref.last][0])
    rr, rg = OR.QReduction(ref, 0.5, max_changes=2), GR.QReduction(fo, 0.5, max_changes=2)
    n0 = len(ref.trace)
    note("wide first/last reduction")
    assert rg.run() == rr.run()
    assert rg.trials == rr.trials and rg.changes == rr.changes
    for key in (("input", "a"), ("fc", "w")):
        t0 = len(rr.trials)
        note("wide first/last reduce", key)
        cr = [c for c in rr.clusters[1] if key in c][0]
        cg = [c for c in rg.clusters[1] if key in c][0]
        assert rg.reduce(cg, 0.5, 1) == rr.reduce(cr, 0.5, 1)
        assert rg.trials[t0:] == rr.trials[t0:] and len(rr.trials) - t0 >= 3
    same_trace(fo.trace[n0:], ref.trace[n0:])
    assert GR.memory_model(fo) == OR.memory_model(ref)
    assert fx.sync_status(fo.h) == 0
    fo.close()


@pytest.mark.parametrize("name,image", [("alexnet", 63), ("vgg16", 32)])
def test_alexnet_vgg_match_oracle(fx, name, image):
    """The paper's other two networks (2 images, small enough that the FC
    input is 1x1): the forward optimizer's candidates and formats, one
    change of Algorithm 2 and the memory model, identical to the oracle."""
    from oracle import qparams as OQ
    from oracle import reduction as OR
    from paper_2203_12091_amd import qparams as GQ
    from paper_2203_12091_amd import reduction as GR
    note("optimizer oracle", name, image)
    ref = OQ.ForwardOptimizer(name, batch=2, image=image, w_wl=8)
    want = ref.run()
    note("optimizer gpu", name, image)
    fo = GQ.ForwardOptimizer(name, batch=2, image=image, device=DEV, w_wl=8)
    got = fo.run()
    assert got == {k: tuple(v) for k, v in want.items()}
    same_trace(fo.trace, ref.trace)
    assert fo.top1_agreement() == ref.top1(ref.q[ref.last][0])
    rr, rg = OR.QReduction(ref, 0.5, max_changes=1), GR.QReduction(fo, 0.5, max_changes=1)
    note("reduction", name)
    assert rg.run() == rr.run()
    assert rg.trials == rr.trials and rg.changes == rr.changes and len(rr.changes) == 1
    assert GR.memory_model(fo) == OR.memory_model(ref)
    assert fx.sync_status(fo.h) == 0
    fo.close()
