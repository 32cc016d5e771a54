"""The oracle of the bit-precision level reduction (Algorithm 2) and of the
memory model (Eq. 26-30).

The traversal and Reduce rules are pinned on stub accuracy functions worked
by hand (binary search over 32-bit word lengths, gradual steps, the size
restriction of the first G1 visit, the zero threshold of G2, hill climbing,
removal at the lowest level, the ranking of candidates); the memory model on
the paper's worked saving (tests/golden/memory_model.txt), a hand-built
graph and ResNet-18's parameter count; the composed run on a tiny ResNet-18
by invariants: every applied change is valid, and the network the change
leaves behind reproduces the cost and accuracy its trial measured."""
import pytest

from conftest import read_golden
from oracle import reduction as R


class FakeFO:
    def __init__(self, qp):
        self.qp, self.order = qp, list(qp)

    def refinalize(self, ln):
        pass


class Stub(R.QReduction):
    """Algorithm 2 over given data structures and an accuracy function of
    all word lengths (no network)."""

    def __init__(self, members, acc, thld, floor=None):
        self.fo = FakeFO({u: [wl, 10, 1] for u, wl, _ in members})
        self.thld, self.max_changes = thld, None
        self.nu = {u: nu for u, _, nu in members}
        self.layer_id = {}
        for u, _, _ in members:
            self.layer_id.setdefault(u[0], len(self.layer_id))
        self.floor = floor or {}
        G1, G2 = R.level1([u for u, _, _ in members])
        self.nu_sum = {d: sum(v for k, v in self.nu.items() if k[1] == d) for d in R.TYPE_ORDER}
        self.clusters = {1: R.level2(G1, self.nu), 2: R.level2(G2, self.nu)}
        self.acc_fp32 = 1.0
        self.trials, self.changes, self.calls = [], [], []
        self.acc = acc

    def trial(self, u, theta):
        wl, fl, _ = self.fo.qp[u]
        self.calls.append((u, theta))
        state = {v: q[0] for v, q in self.fo.qp.items()}
        state[u] = wl - theta
        return fl - theta, self.acc(state)


A, B, C = ("l2", "w"), ("l1", "a"), ("l3", "b")


def test_level1_clusters():
    """Eq. 22 worked by hand: activations and conv / FC weights in G1; the
    bias and both Scale parameters (multiplier, offset) in G2."""
    order = [("input", "a"), ("c1", "w"), ("c1", "s1"), ("c1", "s2"), ("c1", "a"),
             ("fc", "w"), ("fc", "b")]
    G1, G2 = R.level1(order)
    assert G1 == [("input", "a"), ("c1", "w"), ("c1", "a"), ("fc", "w")]
    assert G2 == [("c1", "s1"), ("c1", "s2"), ("fc", "b")]


def test_level2_clusters():
    nu = {("x", "a"): 5, ("y", "w"): 9, ("z", "a"): 5, ("q", "w"): 7}
    G = [("x", "a"), ("y", "w"), ("z", "a"), ("q", "w")]
    assert R.level2(G, nu) == [[("y", "w")], [("q", "w")], [("x", "a"), ("z", "a")]]


def test_binary_search_over_32_bits():
    # valid while the word length stays >= 19, i.e. theta <= 13
    s = Stub([(C, 32, 10)], lambda st: 1.0 if st[C] >= 19 else 0.0, 0.5)
    sol = s.reduce([C], 0.5, 1)
    assert [t for _, t in s.calls] == [16, 8, 12, 14, 13]
    assert sol == (C, 13, 0.0, 10 - 13)
    # the midpoint rounds up: 10 bits, valid only at theta 1
    s = Stub([(C, 10, 10)], lambda st: 1.0 if st[C] >= 9 else 0.0, 0.5)
    sol = s.reduce([C], 0.5, 1)
    assert [t for _, t in s.calls] == [5, 3, 2, 1] and sol[1] == 1


def test_gradual_step_at_8_bits_and_ranking():
    # both valid at theta 1: equal drops, the deeper layer (l2) wins
    s = Stub([(B, 8, 50), (A, 8, 50)], lambda st: 1.0, 0.5)
    sol = s.reduce([B, A], 0.5, 1)
    assert s.calls == [(B, 1), (A, 1)] and sol[0] == A and sol[1] == 1
    # ranking order: theta, then drop, then layer, then type w / a / b
    s.layer_id = {"l1": 1, "l2": 2}
    c = [(("l1", "a"), 2, 0.1, 0), (("l2", "w"), 1, 0.0, 0)]
    assert s.select(c)[0] == ("l1", "a")
    c = [(("l1", "a"), 1, 0.1, 0), (("l1", "w"), 1, 0.2, 0)]
    assert s.select(c)[0] == ("l1", "a")
    c = [(("l1", "a"), 1, 0.1, 0), (("l2", "a"), 1, 0.1, 0)]
    assert s.select(c)[0] == ("l2", "a")
    c = [(("l1", "b"), 1, 0.1, 0), (("l1", "a"), 1, 0.1, 0), (("l1", "w"), 1, 0.1, 0)]
    assert s.select(c)[0] == ("l1", "w")


def test_first_visit_size_restriction_and_hill_climbing():
    # drop 0.1 everywhere; A holds half of all weights
    W2 = ("l9", "w")
    s = Stub([(A, 6, 50), (W2, 6, 50)], lambda st: 0.9, 0.15)
    # lambda = 0: phi = theta * 1/2; theta 1 gives 0.075 < 0.1 for both, the
    # hill-climbing round at theta 2 gives 0.15 >= 0.1: the deeper one wins
    sol = s.reduce([A, W2], 0.15, 0)
    assert s.calls == [(A, 1), (W2, 1), (A, 2), (W2, 2)]
    assert sol[0] == W2 and sol[1] == 2
    # lambda = 1: phi = 1, theta 1 is valid
    s.calls = []
    sol = s.reduce([A], 0.15, 1)
    assert s.calls == [(A, 1)] and sol[1] == 1
    # nothing valid at all: None after both rounds
    s2 = Stub([(A, 6, 50)], lambda st: 0.0, 0.15)
    assert s2.reduce([A], 0.15, 1) is None and s2.calls == [(A, 1), (A, 2)]


def test_traversal_worked_by_hand():
    # accuracy 1 while A >= 2, B >= 1 and C >= 3 bits, else 0
    def acc(st):
        return 1.0 if (st[A] >= 2 and st[B] >= 1 and st[C] >= 3) else 0.0

    s = Stub([(B, 3, 50), (A, 3, 100), (C, 4, 10)], acc, 0.5)
    out = s.run()
    assert [(c[0], c[1], c[2], c[3]) for c in s.changes] == [
        ("l2", "w", 1, 2), ("l1", "a", 1, 2), ("l1", "a", 1, 1), ("l3", "b", 1, 3)]
    assert out == {A: (2, 9, 1), B: (1, 8, 1), C: (3, 9, 1)}
    # B reached 1 bit and left its sub-cluster; A and C stayed
    assert s.clusters[1] == [[A], []] and s.clusters[2] == [[C]]


def test_g2_needs_zero_drop_and_floors():
    # a bias whose every reduction costs 0.01 accuracy is never reduced, even
    # with a large threshold
    s = Stub([(A, 3, 100), (C, 8, 10)], lambda st: 1.0 if st[C] == 8 else 0.99, 0.5)
    s.run()
    assert all(c[1] != "b" for c in s.changes)
    # a floor of 2 bits stops the reduction there and removes the member
    s = Stub([(A, 4, 100)], lambda st: 1.0, 0.5, floor={A: 2})
    s.run()
    assert s.fo.qp[A][0] == 2 and s.clusters[1] == [[]]


def test_memory_model_pins():
    for row in read_golden("memory_model.txt"):
        _, nu, k0, k1, kb = row
        saved = R.mfp(int(nu), int(k0)) - R.mfp(int(nu), int(k1))
        assert round(saved * 1024, 2) == float(kb)
    # Eq. 26 on a hand-built graph: the eltwise step holds both inputs
    nu = {"in": 100, "c1": 200, "c2": 200, "add": 200}
    k = {"in": 8, "c1": 8, "c2": 4, "add": 8}
    layers = [("c1", ["in"]), ("c2", ["c1"]), ("add", ["c1", "c2"])]
    assert R.rw_required(layers, nu, k) == (200 * 8 + 200 * 4 + 200 * 8) / 2 ** 23
    assert R.ro_required([("p", "w"), ("p", "b")], {("p", "w"): 10, ("p", "b"): 2},
                         {("p", "w"): 4, ("p", "b"): 32}) == (40 + 64) / 2 ** 23


def resnet18_parameter_count():
    """Weights, FC bias and Scale (two per channel) of ResNet-18, by hand."""
    convs = [(64, 3, 7)]
    cin = 64
    for width, stride in ((64, 1), (128, 2), (256, 2), (512, 2)):
        for b in range(2):
            convs += [(width, cin, 3), (width, width, 3)]
            if b == 0 and (stride != 1 or cin != width):
                convs.append((width, cin, 1))
            cin = width
    w = sum(k * c * r * r for k, c, r in convs) + 512 * 1000
    return w + 1000 + sum(2 * k for k, _, _ in convs)


@pytest.fixture(scope="module")
def tiny():
    from oracle import qparams as Q
    fo = Q.ForwardOptimizer("resnet18", batch=2, image=16, w_wl=8)
    fo.run()
    return fo


def test_memory_model_of_resnet18(tiny):
    assert resnet18_parameter_count() == 11_689_512
    m = R.memory_model(tiny)
    assert m["ro_fp32"] == 11_689_512 * 32 / 2 ** 23
    # every activation at 8 bits (logits at 32): the widest step is early
    assert m["comp_act"] == 4.0
    scale = sum(v.size for sp in tiny.spec.values() for d, v in sp.items() if d in ("a1",))
    params = 11_689_512 - 2 * scale - 1000
    bias_bits = tiny.qp[("fc", "b")][0] * 1000
    want = (params * 8 + bias_bits + scale * 16 + scale * 32) / 2 ** 23
    assert m["ro_fxp"] == pytest.approx(want, rel=1e-15)


def test_composed_run_invariants(tiny):
    r = R.QReduction(tiny, 0.5, max_changes=2)
    r.run()
    assert len(r.changes) == 2
    fo = tiny
    for (ln, d, theta, wl, fl, drop) in r.changes:
        u = (ln, d)
        # the trial that produced the change was valid under its phi
        t = [x for x in r.trials if x[:3] == (ln, d, theta) and x[4] == fl and x[6]]
        assert t, (ln, d, theta)
        assert wl >= r.min_wl(u)
    # the finalized network reproduces the last change's trial: same
    # accuracy, and the same cost for the chosen candidate
    ln, d, theta, wl, fl, drop = r.changes[-1]
    assert r.accuracy() == pytest.approx(1.0 - drop, abs=0)
    cost, acc = fo.evaluate_quant(ln)
    seen = [c for (l2, d2, f2, c) in fo.trace if (l2, d2, f2) == (ln, d, fl)]
    assert cost in seen and acc == 1.0 - drop
    assert tuple(fo.qp[(ln, d)][:2]) == (wl, fl)


def test_scale_parameters_reduced_in_g2(tiny):
    """A G2 visit reduces Scale parameters (Eq. 22): with G1 left out, the
    first change comes from G2's largest sub-cluster (the FC bias, 1000
    values, then the 512-channel Scale parameters), at zero accuracy drop."""
    import copy
    fo = copy.deepcopy(tiny)
    r = R.QReduction(fo, 0.5, max_changes=3)
    scale = [u for u in fo.order if u[1] in ("s1", "s2")]
    assert scale and all(any(u in c for c in r.clusters[2]) for u in scale)
    assert not any(u in c for c in r.clusters[1] for u in scale)
    r.clusters[1] = []
    r.run()
    assert r.changes and all(d in ("b", "s1", "s2") and drop <= 0 for _, d, _, _, _, drop in r.changes)
    assert any(d in ("s1", "s2") for _, d, _, _, _, _ in r.changes)
    for ln, d, theta, wl, fl, drop in r.changes:
        assert tuple(fo.qp[(ln, d)][:2]) == (wl, fl)
