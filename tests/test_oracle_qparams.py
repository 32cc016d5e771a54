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
