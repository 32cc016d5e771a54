"""The oracle of Algorithm 1 (QParamsOpt) and the forward optimizer.

The search rule is pinned on cost curves worked by hand (directional
expansion: a direction is followed K steps past its last improvement, so
K = 1 stops at the first local minimum while a large K reaches the global
one), and on a tiny ResNet-18 against brute force: the chosen fractional
length of the first data structure is a local minimum of its full cost
curve, every chosen format is the cheapest of the candidates evaluated for
it, and no chosen format costs more than the preprocessor's."""
import pytest

from oracle import qparams as Q


class Stub(Q.ForwardOptimizer):
    """The search loop over a given cost curve (no network)."""

    def __init__(self, curve, fl0, K):
        self.curve, self.K, self.trace = curve, K, []
        self.qp = {("x", "w"): [8, fl0, 1]}

    def evaluate(self, ln):
        return self.curve(self.qp[("x", "w")][1])


@pytest.mark.parametrize("curve,fl0,K,want", [
    # convex, minimum 3 steps up: followed step by step
    (lambda f: (f - 3) ** 2, 0, 1, 3),
    # convex, minimum 2 steps down
    (lambda f: (f + 2) ** 2, 0, 1, -2),
    # start at the minimum
    (lambda f: abs(f - 5), 5, 1, 5),
    # a bump one step up hides a deeper minimum two steps up: K = 1 stops,
    # K = 2 looks one step further
    (lambda f: {0: 4.0, 1: 5.0, 2: 1.0}.get(f, 9.0), 0, 1, 0),
    (lambda f: {0: 4.0, 1: 5.0, 2: 1.0}.get(f, 9.0), 0, 2, 2),
    # equal cost is not an improvement: the first (initial) candidate stays
    (lambda f: 1.0, 4, 3, 4),
    # both directions improve: the downward search runs first, the upward one
    # must beat its result
    (lambda f: {-1: 2.0, 0: 3.0, 1: 1.0}.get(f, 9.0), 0, 1, 1),
    # the range ends at -8 / 15
    (lambda f: float(f), -7, 1, -8),
    (lambda f: float(-f), 14, 1, 15),
])
def test_search_rule(curve, fl0, K, want):
    s = Stub(curve, fl0, K)
    assert s.qparams_opt("x", "w") == want
    assert s.qp[("x", "w")][1] == want


def test_tiny_resnet18_against_brute_force():
    fo = Q.ForwardOptimizer("resnet18", batch=1, image=16)
    # brute force over the whole range for the first data structure
    key = ("input", "a")
    fl0 = fo.qp[key][1]
    curve = {}
    for fl in range(-8, 16):
        fo.qp[key][1] = fl
        curve[fl] = fo.evaluate("input")
    fo.qp[key][1] = fl0
    res = fo.run()
    got = res[key][1]
    for nb in (got - 1, got + 1):
        if nb in curve:
            assert curve[got] <= curve[nb]
    assert curve[got] <= curve[fl0]
    # every choice is the cheapest candidate evaluated for it, never worse
    # than the initial format
    by = {}
    for ln, d, fl, cost in fo.trace:
        by.setdefault((ln, d), []).append((fl, cost))
    for k, cands in by.items():
        first = cands[0]
        best = min(c for _, c in cands)
        chosen = [c for f, c in cands if f == res[k][1]]
        assert chosen and chosen[0] == best and best <= first[1], k
    assert len(by) == len(fo.order)


def _golden_layers():
    from fractions import Fraction

    import numpy as np

    from conftest import read_golden
    samples, params, errs, expect = {}, {}, {}, []
    for r in read_golden("importance_pi.txt"):
        if r[0] == "sample":
            samples.setdefault((r[1], r[2]), []).append([float(Fraction(v)) for v in r[3:]])
        elif r[0] == "param":
            params[(r[1], r[2])] = [float(Fraction(v)) for v in r[3:]]
        elif r[0] == "err":
            errs[(r[1], r[2])] = float(Fraction(r[3]))
        else:
            expect.append((r[1], r[2], r[3], Fraction(r[4])))
    stat = {k: Q._stats(np.array(v), per_sample=True) for k, v in samples.items()}
    stat.update({k: Q._stats(np.array(v)) for k, v in params.items()})
    return stat, errs, expect


def test_importance_pinned_by_hand():
    """Eq. 15-18 on the hand-worked layers of tests/golden/importance_pi.txt:
    sigma of activations per sample then averaged, nu per sample, pi
    normalized per layer, E summed over the layers from l on."""
    stat, errs, expect = _golden_layers()
    pi = {}
    for layer in {k[0] for k in stat}:
        pi.update(Q.importance({k: v for k, v in stat.items() if k[0] == layer}))
    field = {"sigma": 0, "nu": 1, "range": 2}
    n = 0
    for what, layer, d, want in expect:
        if what in field:
            got = stat[(layer, d)][field[what]]
        elif what == "pi":
            got = pi[(layer, d)]
        else:  # E(., l): the layers from l on
            got = Q.distillation_error(pi, stat, {k: e for k, e in errs.items() if int(k[0]) >= int(layer)})
        assert abs(got - float(want)) <= 1e-15 * max(1.0, abs(float(want))), (what, layer, d, got, want)
        n += 1
    assert n == 19


def test_importance_is_not_whole_batch():
    """The per-sample reading differs from the whole-batch statistics on the
    golden layer (so a regression to those fails the pin above)."""
    import numpy as np
    a = np.array([[0, 2, 0, 2], [4, 4, 4, 4]], np.float64)
    sig, nu, _ = Q._stats(a, per_sample=True)
    assert (sig, nu) == (0.5, 4)
    assert abs(a.std() - 11 ** 0.5 / 2) < 1e-15 and a.size == 8


def test_forward_optimizer_uses_eq15_statistics():
    """The forward optimizer's statistics are Eq. 16's (per sample for
    activations), its pi normalized per layer over every data structure of
    the layer, Scale parameters included."""
    import numpy as np
    fo = Q.ForwardOptimizer("resnet18", batch=2, image=16)
    acts = [k for k in fo.stat if k[1] == "a" and k[0] != "input"]
    assert acts
    for k in acts:
        assert fo.stat[k] == Q._stats(fo.g.act[k[0]], per_sample=True)
    assert fo.stat[("input", "a")] == Q._stats(fo.g.x, per_sample=True)
    assert fo.stat[("input", "a")][1] == 3 * 16 * 16
    layers = {k[0] for k in fo.pi}
    for ln in layers:
        tot = sum(v for k, v in fo.pi.items() if k[0] == ln)
        assert abs(tot - 1.0) < 1e-12, ln
    # every BN-as-Scale C-Block has both Scale parameters as data structures
    scaled = [ln for ln, sp in fo.spec.items() if "a1" in sp]
    assert scaled and all((ln, "s1") in fo.order and (ln, "s2") in fo.order for ln in scaled)
    assert all(fo.qp[(ln, "s1")][0] == 16 and fo.qp[(ln, "s2")][0] == 32 for ln in scaled)
    np.testing.assert_equal(sorted(d for ln, d in fo.order if ln == scaled[0]),
                            sorted(["w", "s1", "s2", "a"]))
