"""Whole calibration forwards on the GPU against the exact CPU oracle.

Every chosen format (weights, biases, Scale parameters, every activation),
every activation code and the final integer logits must be bit-identical.
Sizes are small enough for the oracle to finish in seconds but span many
tiles of every kernel; odd image sizes give ragged tails everywhere.
"""
import numpy as np
import pytest

from gpu_util import note

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mods():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import oracle
    from paper_2203_12091_amd import nets
    return nets, oracle


def compare(res, ref):
    assert res["flags"] == 0, f"device flags {res['flags']:#x}"
    assert set(res["fmts"]) == set(ref["fmts"])
    bad = {k: (res["fmts"][k], ref["fmts"][k]) for k in ref["fmts"] if res["fmts"][k] != ref["fmts"][k]}
    assert not bad, bad
    for name, want in ref.get("codes", {}).items():
        got = res["codes"][name]
        got = np.transpose(got, (0, 3, 1, 2)) if got.ndim == 4 else got
        if name == "input":
            got = got[:, :3]
        assert got.size == want.size, name
        assert np.array_equal(got.reshape(want.shape), want), name
    assert res["logit_fl"] == ref["logit_fl"]
    assert np.array_equal(res["logits"], ref["logits"])


def test_fc_config(mods):
    nets, oracle = mods
    note("net fc")
    res = nets.run_config("fc")
    ref = oracle.nets.run_config("fc")
    assert res["flags"] == 0
    assert res["fmts"] == ref["fmts"]
    for wl in (8, 6, 4):
        assert np.array_equal(res["outs"][wl]["acc"], ref["outs"][wl]["acc"])
        assert np.array_equal(res["outs"][wl]["y"], ref["outs"][wl]["y"])


@pytest.mark.parametrize("name,batch,image", [
    ("resnet50", 2, 64), ("resnet50", 1, 67), ("resnet18", 3, 64), ("resnet18", 2, 75),
    ("alexnet", 2, 67), ("alexnet", 1, 99), ("vgg16", 2, 64), ("vgg16", 1, 48)])
def test_network_bit_exact(mods, name, batch, image):
    nets, oracle = mods
    note("net", name, batch, image)
    res = nets.run_config(name, batch=batch, image=image, with_codes=True)
    ref = oracle.nets.run_config(name, batch=batch, image=image)
    compare(res, ref)
    np.testing.assert_allclose(res["input_error"][:3], ref["input_error"][:3], rtol=1e-9)


def test_fused_paths_match_two_call_forward(mods):
    # the fused C-Block calls and the fused FxP-QLayer calls against the
    # qconv -> fl_search -> requant sequence over whole ResNet-50 forwards, at
    # a size beyond the oracle's; two forwards each (the second one's
    # FxP-QLayers start from the formats the first one chose)
    nets, _ = mods
    res = {}
    for fused, qlayer, predict, defer in ((True, True, False, True), (False, True, False, True),
                                          (False, False, False, True), (False, True, True, True),
                                          (False, True, True, False)):
        note("net resnet50 8x112 fused", fused, "qlayer", qlayer, "predict", predict, "defer", defer)
        net = nets.CalibNet("resnet50", batch=8, image=112, fused=fused, qlayer=qlayer,
                            predict=predict, defer=defer)
        plan = net._plan()
        assert any(c[0] == "cblock" for c in plan) == fused
        assert any(c[2].__name__ == "fxpq_qlayer" for c in plan) == qlayer
        assert net.predict == predict
        for _ in range(2):
            net.forward()
            res[(fused, qlayer, predict, defer, _)] = net.results(with_codes=True)
        if predict:
            # the first forward has no predictions; a layer whose window
            # cannot decide alone misses once more, then runs unpredicted
            assert net.misses <= 2
            m = net.misses
            net.forward()
            assert net.misses == m
            res[(fused, qlayer, predict, defer, 2)] = net.results(with_codes=True)
        net.close()
    b = res[(False, False, False, True, 1)]
    for key, a in res.items():
        assert a["flags"] == 0, key
        assert a["fmts"] == b["fmts"], key
        for name in b["codes"]:
            assert np.array_equal(a["codes"][name], b["codes"][name]), (key, name)
        assert np.array_equal(a["logits"], b["logits"]), key


@pytest.mark.parametrize("name,batch,image", [
    ("resnet50", 2, 64), ("resnet18", 2, 75), ("alexnet", 2, 67), ("vgg16", 2, 64)])
def test_predicted_forward_bit_exact(mods, name, batch, image):
    """Predicted C-Blocks (fxpq_cblock_predicted): the first forward has no
    prediction (every predicted C-Block misses and the standard calls run
    again from the first), the second is predicted from the first; both
    bit-identical to the oracle.  Then another batch (the images scaled by
    1.5, predictions from the first batch) against the standard calls on that
    batch."""
    nets, oracle = mods
    net = nets.CalibNet(name, batch=batch, image=image)
    net._plan()
    assert net.predict and any(c[0] == "cblock_pred" for c in net.pcalls)
    ref = oracle.nets.run_config(name, batch=batch, image=image)
    for k in range(2):
        note("net predicted", name, batch, image, "forward", k)
        net.forward()
        compare(net.results(with_codes=True), ref)
    assert net.misses >= 1
    std = nets.CalibNet(name, batch=batch, image=image, predict=False)
    for t in (net, std):
        t.x_dev.mul_(1.5)
    note("net predicted", name, "other batch")
    net.forward()
    std.forward()
    a, b = net.results(with_codes=True), std.results(with_codes=True)
    assert a["flags"] == 0 and a["fmts"] == b["fmts"]
    for nm in b["codes"]:
        assert np.array_equal(a["codes"][nm], b["codes"][nm]), nm
    assert np.array_equal(a["logits"], b["logits"])
    net.close()
    std.close()
