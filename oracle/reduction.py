"""Oracle of the bit-precision level reduction (Algorithm 2, parts 1 and 2)
and of the memory model (Eq. 26-30) -- TEST INFRASTRUCTURE ONLY.

Sec. "Bit-Precision Level Reduction": the data structures of a quantized
network are clustered (Eq. 22: G1 = activations and conv / FC weights, G2 =
the other learnable parameters, i.e. biases and Scale parameters; Eq. 23:
within each, one sub-cluster per distinct size, larger sizes first).  The traversal visits G1's sub-clusters
in order; in a sub-cluster, every data structure competes (Reduce): it tries
word length k - theta with its fractional length lowered by theta (the
integer length stays), re-optimizes the fractional length with Algorithm 1
and measures the accuracy; theta is 1 when k <= 8 and binary-searched in
[1, k - 1] otherwise (2 when hill climbing after a round without
candidates).  A trial is valid when the accuracy drop is at most
phi * threshold, phi = lambda + (1 - lambda) * theta * size / (sum of the
sizes of that type), lambda = 0 on the first visit of G1 and 1 afterwards
(Eq. 24); G2 gets threshold 0.  The best valid candidate (largest theta,
then smallest drop, then deepest layer, then type) is applied and the
sub-cluster is visited again; a data structure that reaches 1 bit leaves its
sub-cluster.  The traversal alternates between G1 and G2 until an episode
changes nothing.

Readings (the GPU driver takes the same):
  * the network is the forward optimizer's result (Algorithm 1 on every data
    structure) from 8-bit weights and activations, 32-bit biases and the
    Scale parameters at 16 (multiplier aleph_1) and 32 (offset aleph_2)
    bits; the Scale parameters are G2 members like the biases (Eq. 22);
  * accuracy without labels is the top-1 agreement with the FP32 teacher on
    the calibration batch, so the FP32 accuracy is 1;
  * a trial's Algorithm 1 runs the whole network quantized (the prefix at
    its formats, the data structure at the candidate, every later layer at
    its formats), its cost summing the errors of all data structures from
    the trial's layer on;
  * a trial whose lowered fractional length falls below the format range is
    not valid (no candidate at that theta);
  * in the hill-climbing round theta = 2 is tried only where k - 2 is
    allowed;
  * the input and the first layer's weights stop at 2 bits: the GPU layout
    pads the RGB input to four channels with zeros, and a 1-bit code (Eq. 13)
    has no zero;
  * sizes are per image for activations (C x H x W, the input's three
    channels), the model's counts for parameters; the sums in phi run over
    the data structures of that type taking part (G1 / G2 members), the
    Scale multipliers and offsets each forming a type of their own;
  * select()'s last tie rule orders w / a / b / aleph_1 / aleph_2.

parity unpinned for the composed run over a network (the paper prints
none); the Reduce / select / traversal rules are pinned on stub accuracy
functions worked by hand, the memory model on the paper's CONV-1 saving and
ResNet-18's parameter count, the composed run by invariants
(tests/test_oracle_reduction.py).
"""
import math

from .nets import FL
from .qparams import PARAM

# tie order of select(): conv / FC weights, activations, bias, then the Scale
# multiplier and offset
TYPE_ORDER = {"w": 0, "a": 1, "b": 2, "s1": 3, "s2": 4}


def level1(order):
    """Eq. 22: (G1, G2) of the data structures in network order: G1 holds
    every activation and the conv / FC weights, G2 every other learnable
    parameter (biases, Scale multipliers and offsets)."""
    G1 = [k for k in order if k[1] in ("a", "w")]
    G2 = [k for k in order if k[1] not in ("a", "w")]
    return G1, G2


def level2(G, nu):
    """Eq. 23: one sub-cluster per distinct size, larger sizes first; members
    keep the network order."""
    sizes = sorted({nu[k] for k in G}, reverse=True)
    return [[k for k in G if nu[k] == v] for v in sizes]


class QReduction:
    def __init__(self, fo, delta_thld, max_changes=None):
        """fo: an oracle ForwardOptimizer whose run() has finished."""
        self.fo, self.thld, self.max_changes = fo, float(delta_thld), max_changes
        g = fo.g
        self.layer_id = {"input": 0}
        for op, nm, _ in g.nodes:
            if op == "conv":
                self.layer_id[nm] = len(self.layer_id)
        self.nu = {}
        for (ln, d) in fo.order:
            if ln == "input":
                self.nu[(ln, d)] = int(g.x[0].size)
            elif d == "a":
                self.nu[(ln, d)] = int(g.act[ln][0].size)
            else:
                self.nu[(ln, d)] = int(fo.spec[ln][PARAM.get(d, d)].size)
        first = [nm for op, nm, _ in g.nodes if op == "conv"][0]
        self.floor = {("input", "a"): 2, (first, "w"): 2}
        G1, G2 = level1(fo.order)
        self.nu_sum = {d: sum(v for k, v in self.nu.items() if k[1] == d) for d in TYPE_ORDER}
        self.clusters = {1: level2(G1, self.nu), 2: level2(G2, self.nu)}
        self.acc_fp32 = 1.0
        self.trials = []   # (ln, d, theta, fl_start, fl_chosen, acc, valid)
        self.changes = []  # (ln, d, theta, wl, fl, delta)

    # -- one trial: Algorithm 1 at word length k - theta ------------------------------
    def trial(self, u, theta):
        """(fractional length, accuracy) Algorithm 1 reaches for u at word
        length k - theta from fl - theta, or None when fl - theta is out of
        range; the format of u is restored afterwards."""
        fo = self.fo
        wl, fl, sign = fo.qp[u]
        if fl - theta < FL[0]:
            return None
        fo.qp[u] = [wl - theta, fl - theta, sign]
        fl_new = fo.qparams_opt(u[0], u[1], quantized=True)
        acc = fo.acc_best
        fo.qp[u] = [wl, fl, sign]
        return fl_new, acc

    # -- Algorithm 2, part 2 ------------------------------------------------------------
    def reduce(self, G, thld, lam):
        climb = False
        while True:
            cand = []
            for u in G:
                k = self.fo.qp[u][0]
                if climb:
                    lo, hi = 2, 2
                elif k <= 8:
                    lo = hi = 1
                else:
                    lo, hi = 1, k - 1
                hi = min(hi, k - self.min_wl(u))
                sol = None
                while lo <= hi:
                    theta = (lo + hi + 1) // 2
                    r = self.trial(u, theta)
                    valid = False
                    if r is not None:
                        fl_new, acc = r
                        delta = self.acc_fp32 - acc
                        phi = lam + (1 - lam) * theta * self.nu[u] / self.nu_sum[u[1]]
                        valid = delta <= phi * thld
                        self.trials.append((u[0], u[1], theta, self.fo.qp[u][1] - theta, fl_new, acc, valid))
                    if valid:
                        sol = (u, theta, delta, fl_new)
                        lo = theta + 1
                    else:
                        hi = theta - 1
                if sol is not None:
                    cand.append(sol)
            if cand:
                return self.select(cand)
            if climb:
                return None
            climb = True

    def min_wl(self, u):
        return self.floor.get(u, 1)

    def select(self, cand):
        """Largest reduction, then smallest accuracy drop, then deepest
        layer, then weights / activations / biases."""
        return min(cand, key=lambda c: (-c[1], c[2], -self.layer_id[c[0][0]], TYPE_ORDER[c[0][1]]))

    def apply(self, sol, cluster):
        u, theta, delta, fl_new = sol
        fo = self.fo
        wl, _, sign = fo.qp[u]
        fo.qp[u] = [wl - theta, fl_new, sign]
        fo.refinalize(u[0])
        if wl - theta == self.min_wl(u):
            cluster.remove(u)
        self.changes.append((u[0], u[1], theta, wl - theta, fl_new, delta))

    def capped(self):
        return self.max_changes is not None and len(self.changes) >= self.max_changes

    # -- Algorithm 2, part 1 ------------------------------------------------------------
    def run(self):
        visit = {1: True, 2: True}
        t, lam = 1, 0
        while True:
            visit[t] = False
            j = 0
            while j < len(self.clusters[t]):
                if self.capped():
                    return self.formats()
                sol = self.reduce(self.clusters[t][j], self.thld if t != 2 else 0.0, lam)
                if sol is not None:
                    self.apply(sol, self.clusters[t][j])
                    visit = {1: True, 2: True}
                else:
                    j += 1
            if not visit[t]:
                t = 2 if t == 1 else 1
            lam = 1
            if not visit[t]:
                return self.formats()

    def formats(self):
        return {k: tuple(self.fo.qp[k]) for k in self.fo.order}

    def accuracy(self):
        """Top-1 agreement of the finalized network."""
        return self.fo.top1(self.fo.q[self.fo.last][0])


# ---------------------------------------------------------------------------------
# Memory model (Sec. "Memory Requirements", Eq. 26-30)
# ---------------------------------------------------------------------------------
def mfp(nu, k):
    """Eq. 28: footprint in MB (2^23 bits) of nu values of k bits."""
    return nu * k / 2.0 ** 23


def rw_required(layers, nu, k):
    """Eq. 26: the largest sum over layers of the footprints of a layer's
    input activations and of its output.  layers: [(name, [inputs])]."""
    return max(sum(mfp(nu[i], k[i]) for i in ins) + mfp(nu[l], k[l]) for l, ins in layers)


def ro_required(params, nu, k):
    """Eq. 27: the footprints of every learnable data structure."""
    return math.fsum(mfp(nu[p], k[p]) for p in params)


def memory_model(fo, formats=None):
    """RW / RO requirements (MB) of the oracle network at FP32 and at the
    given formats, and the compression rates of Eq. 29-30.  Activations of
    the output layer stay at 32 bits; max-pool outputs keep their input's
    word length; eltwise / avg-pool outputs have their 8-bit FxP-QLayers;
    Scale parameters count at their formats' word lengths."""
    qp = fo.qp if formats is None else formats
    g = fo.g
    nu, k, layers = {}, {}, []
    nu["input"], k["input"] = int(g.x[0].size), qp[("input", "a")][0]
    params = []
    for op, nm, sp in g.nodes:
        if op == "input":
            continue
        nu[nm] = int(g.act[nm][0].size)
        if op == "conv":
            ins = [sp["src"]]
            k[nm] = 32 if sp["last"] else qp[(nm, "a")][0]
            for d in ("w", "b"):
                if d in sp:
                    nu[(nm, d)], k[(nm, d)] = int(sp[d].size), qp[(nm, d)][0]
                    params.append((nm, d))
            if "a1" in sp:
                for d in ("s1", "s2"):
                    nu[(nm, d)], k[(nm, d)] = int(sp[PARAM[d]].size), qp[(nm, d)][0]
                    params.append((nm, d))
        elif op == "maxpool":
            ins = [sp["src"]]
            k[nm] = k[sp["src"]]
        elif op == "add":
            ins = [sp["a"], sp["b"]]
            k[nm] = 8
        else:
            ins = [sp["src"]]
            k[nm] = fo.fl_wl or 8
        layers.append((nm, ins))
    k32 = {key: 32 for key in k}
    rw_fp, rw_q = rw_required(layers, nu, k32), rw_required(layers, nu, k)
    ro_fp, ro_q = ro_required(params, nu, k32), ro_required(params, nu, k)
    return {"rw_fp32": rw_fp, "rw_fxp": rw_q, "ro_fp32": ro_fp, "ro_fxp": ro_q,
            "comp_act": rw_fp / rw_q, "comp_model": ro_fp / ro_q}
