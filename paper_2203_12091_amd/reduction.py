"""Bit-precision level reduction (Algorithm 2, parts 1 and 2) and the memory
model (Eq. 26-30) over the GPU forward optimizer.

Sec. "Bit-Precision Level Reduction": the data structures of the quantized
network are clustered (Eq. 22: G1 holds the activations and the conv / FC
weights, G2 the other learnable parameters, i.e. biases and the Scale
multipliers and offsets; Eq. 23: one sub-cluster per distinct size, larger
first).  Sub-clusters are visited in order; inside one,
every member tries a lower word length k - theta (fractional length lowered
by theta, integer length kept), re-optimized by Algorithm 1 with the whole
network quantized, and is scored by its accuracy drop.  theta is 1 for
k <= 8 and binary-searched in [1, k - 1] above 8; when no member succeeds,
one hill-climbing round tries theta = 2.  A trial is valid when its drop is
at most phi * threshold with phi = lambda + (1 - lambda) * theta * size /
(sum of the sizes of its type) (Eq. 24; lambda = 0 only on the first visit
of G1, and G2 gets threshold 0).  Of the valid trials the one with the
largest theta, then the smallest drop, then the deepest layer, then type
(w / a / b / aleph_1 / aleph_2) is applied; the sub-cluster is visited again
until nothing changes, and the traversal alternates between G1 and G2 until an episode
changes nothing.

Readings: the network is the forward optimizer's result from 8-bit weights
and activations, 32-bit biases and the Scale parameters at 16 (aleph_1) and
32 (aleph_2) bits; accuracy is the top-1 agreement with the FP32 teacher on the calibration
batch (no labels), so the FP32 accuracy is 1; a trial whose lowered
fractional length falls below the format range is not valid; hill climbing
tries theta = 2 only where k - 2 is allowed; the input and the first layer's
weights stop at 2 bits (the RGB input is padded to four channels with zeros,
which a 1-bit code cannot hold); sizes are per image for activations; the
sums in phi run over the data structures of the same type, the Scale
multipliers and offsets each forming a type of their own.

Every evaluation is a sequence of libfxpq calls; the host only keeps the
clusters, compares accuracies and ranks the candidates.
"""
import math

from .nets import FL_LO

TYPE_ORDER = {"w": 0, "a": 1, "b": 2, "s1": 3, "s2": 4}


def level1(order):
    """Eq. 22: (G1, G2) in network order; G1 = activations and conv / FC
    weights, G2 = every other learnable parameter."""
    return ([u for u in order if u[1] in ("a", "w")],
            [u for u in order if u[1] not in ("a", "w")])


def sub_clusters(G, nu):
    """Eq. 23: members of G grouped by size, larger sizes first, network
    order inside a group."""
    out = {}
    for u in G:
        out.setdefault(nu[u], []).append(u)
    return [out[v] for v in sorted(out, reverse=True)]


class QReduction:
    def __init__(self, fo, delta_thld, max_changes=None):
        """fo: a qparams.ForwardOptimizer whose run() has finished."""
        self.fo, self.thld, self.max_changes = fo, float(delta_thld), max_changes
        convs = [n for n in fo.nodes if n.op in ("conv", "fc")]
        self.layer_id = {"input": 0}
        self.layer_id.update({n.name: i for i, n in enumerate(convs, 1)})
        self.nu = {}
        for (ln, d) in fo.order:
            if ln == "input":
                _, H, W, _ = fo.act["input"].shape
                self.nu[(ln, d)] = 3 * H * W
            elif d == "a":
                self.nu[(ln, d)] = math.prod(fo.act[ln].shape[1:])
            elif d == "w":
                self.nu[(ln, d)] = int(fo.L[ln]["w_host"].size)
            else:
                self.nu[(ln, d)] = fo.L[ln]["node"].cout
        self.floor = {("input", "a"): 2, (convs[0].name, "w"): 2}
        G1, G2 = level1(fo.order)
        self.type_size = {t: sum(v for u, v in self.nu.items() if u[1] == t) for t in TYPE_ORDER}
        self.clusters = {1: sub_clusters(G1, self.nu), 2: sub_clusters(G2, self.nu)}
        self.acc_fp32 = 1.0
        self.trials = []   # (layer, d, theta, fl start, fl chosen, accuracy, valid)
        self.changes = []  # (layer, d, theta, new word length, fl, accuracy drop)

    def min_wl(self, u):
        return self.floor.get(u, 1)

    def trial(self, u, theta):
        """Algorithm 1 for u at word length k - theta from fl - theta:
        (chosen fl, its accuracy), or None if fl - theta is out of range.
        The format of u is restored afterwards."""
        fo = self.fo
        wl, fl, _ = fo.qp[u]
        if fl - theta < FL_LO:
            return None
        fo._set(u, fl - theta, wl - theta)
        fl_new, _ = fo.qparams_opt(u[0], u[1], quantized=True)
        acc = fo.acc_best
        fo._set(u, fl, wl)
        return fl_new, acc

    def reduce(self, G, thld, lam):
        """Algorithm 2, part 2: the selected candidate of sub-cluster G, or
        None."""
        for climb in (False, True):
            cand = []
            for u in G:
                k = self.fo.qp[u][0]
                if climb:
                    lo = hi = 2
                elif k <= 8:
                    lo = hi = 1
                else:
                    lo, hi = 1, k - 1
                hi = min(hi, k - self.min_wl(u))
                best = None
                while lo <= hi:
                    theta = (lo + hi + 1) // 2
                    r = self.trial(u, theta)
                    ok = False
                    if r is not None:
                        fl_new, acc = r
                        drop = self.acc_fp32 - acc
                        phi = lam + (1 - lam) * theta * self.nu[u] / self.type_size[u[1]]
                        ok = drop <= phi * thld
                        self.trials.append((u[0], u[1], theta, self.fo.qp[u][1] - theta, fl_new, acc, ok))
                    if ok:
                        best, lo = (u, theta, drop, fl_new), theta + 1
                    else:
                        hi = theta - 1
                if best is not None:
                    cand.append(best)
            if cand:
                return min(cand, key=lambda c: (-c[1], c[2], -self.layer_id[c[0][0]], TYPE_ORDER[c[0][1]]))
        return None

    def apply(self, sol, cluster):
        u, theta, drop, fl_new = sol
        wl = self.fo.qp[u][0] - theta
        self.fo._set(u, fl_new, wl)
        self.fo.refinalize(u[0])
        if wl == self.min_wl(u):
            cluster.remove(u)
        self.changes.append((u[0], u[1], theta, wl, fl_new, drop))

    def run(self):
        """Algorithm 2, part 1; returns the final formats."""
        visit = {1: True, 2: True}
        t, lam = 1, 0
        while True:
            visit[t] = False
            j = 0
            while j < len(self.clusters[t]):
                if self.max_changes is not None and len(self.changes) >= self.max_changes:
                    return self.formats()
                sol = self.reduce(self.clusters[t][j], self.thld if t == 1 else 0.0, lam)
                if sol is None:
                    j += 1
                    continue
                self.apply(sol, self.clusters[t][j])
                visit = {1: True, 2: True}
            if not visit[t]:
                t = 3 - t
            lam = 1
            if not visit[t]:
                return self.formats()

    def formats(self):
        return {u: tuple(self.fo.qp[u]) for u in self.fo.order}

    def accuracy(self):
        return self.fo.top1_agreement()


# ---------------------------------------------------------------------------------
# Memory model (Sec. "Memory Requirements", Eq. 26-30)
# ---------------------------------------------------------------------------------
def footprint_mb(count, bits):
    """Eq. 28: MB (2^23 bits) taken by count values of the given width."""
    return count * bits / 2.0 ** 23


def memory_model(fo):
    """Read-write (Eq. 26) and read-only (Eq. 27) requirements in MB at FP32
    and at the current formats of fo, and the compression rates (Eq. 29-30).
    Output-layer activations stay at 32 bits, max-pool outputs keep their
    input's word length, eltwise / avg-pool outputs are 8-bit FxP-QLayers,
    Scale parameters count at their formats' word lengths."""
    size, bits, steps, params = {}, {}, [], []
    _, H, W, _ = fo.act["input"].shape
    size["input"], bits["input"] = 3 * H * W, fo.qp[("input", "a")][0]
    for n in fo.nodes:
        if n.op == "input":
            continue
        size[n.name] = math.prod(fo.act[n.name].shape[1:])
        ins = [n.inp] + ([n.other] if n.op == "add" else [])
        if n.op in ("conv", "fc"):
            L = fo.L[n.name]
            bits[n.name] = 32 if n.last else fo.qp[(n.name, "a")][0]
            size[(n.name, "w")], bits[(n.name, "w")] = int(L["w_host"].size), fo.qp[(n.name, "w")][0]
            params.append((n.name, "w"))
            if n.bias:
                size[(n.name, "b")], bits[(n.name, "b")] = n.cout, fo.qp[(n.name, "b")][0]
                params.append((n.name, "b"))
            if "a1_f32" in L:
                for d in ("s1", "s2"):
                    size[(n.name, d)], bits[(n.name, d)] = n.cout, fo.qp[(n.name, d)][0]
                    params.append((n.name, d))
        elif n.op == "maxpool":
            bits[n.name] = bits[n.inp]
        elif n.op == "avgpool" and fo.fl_wl is not None:
            bits[n.name] = fo.fl_wl  # the last layer's input
        else:
            bits[n.name] = 8
        steps.append((n.name, ins))

    def rw(b):
        return max(sum(footprint_mb(size[i], b[i]) for i in ins) + footprint_mb(size[o], b[o])
                   for o, ins in steps)

    def ro(b):
        return math.fsum(footprint_mb(size[p], b[p]) for p in params)

    full = {key: 32 for key in bits}
    r = {"rw_fp32": rw(full), "rw_fxp": rw(bits), "ro_fp32": ro(full), "ro_fxp": ro(bits)}
    r["comp_act"] = r["rw_fp32"] / r["rw_fxp"]
    r["comp_model"] = r["ro_fp32"] / r["ro_fxp"]
    return r
