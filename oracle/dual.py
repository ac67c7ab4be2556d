"""Dual-number evaluation of masked softmax attention.  TEST INFRASTRUCTURE ONLY.

Forward-mode differentiation by construction: every scalar carries a pair
(value, tangent) and each arithmetic step applies its own derivative rule
(sum, product, quotient, exp, log).  The masked attention map of the paper's
App. B (masked-attention equation; the mask is a fixed routing object with no
tangent) is then evaluated element by element with plain Python loops.  No
closed-form tangent expression appears here, so agreement with the closed form
in ``attention.py`` pins that closed form.

Only for tiny inputs: the cost is O(L^2 D) Python operations per head.
"""
import math

from .masks import allowed_mask


class Dual:
    __slots__ = ("x", "t")

    def __init__(self, x, t=0.0):
        self.x = float(x)
        self.t = float(t)

    def __add__(self, o):
        o = o if isinstance(o, Dual) else Dual(o)
        return Dual(self.x + o.x, self.t + o.t)

    __radd__ = __add__

    def __sub__(self, o):
        o = o if isinstance(o, Dual) else Dual(o)
        return Dual(self.x - o.x, self.t - o.t)

    def __mul__(self, o):
        o = o if isinstance(o, Dual) else Dual(o)
        return Dual(self.x * o.x, self.t * o.x + self.x * o.t)

    __rmul__ = __mul__

    def __truediv__(self, o):
        o = o if isinstance(o, Dual) else Dual(o)
        return Dual(self.x / o.x, (self.t * o.x - self.x * o.t) / (o.x * o.x))

    def exp(self):
        e = math.exp(self.x)
        return Dual(e, e * self.t)

    def log(self):
        return Dual(math.log(self.x), self.t / self.x)


def attention_dual(Q, K, V, dQ, dK, dV, kind, offsets=None, scale=None):
    """Returns nested lists O[b][h][a][d], dO[b][h][a][d], LSE[b][h][a], dLSE[b][h][a].

    Inputs are array-likes of shape [B, H, L, D] (values read with float()).
    """
    B, H, L, D = len(Q), len(Q[0]), len(Q[0][0]), len(Q[0][0][0])
    s = float(scale) if (scale is not None and scale > 0) else 1.0 / math.sqrt(D)
    allowed = allowed_mask(kind, offsets, L)
    O, dO, LSE, dLSE = [], [], [], []
    for b in range(B):
        Ob, dOb, Lb, dLb = [], [], [], []
        for h in range(H):
            q = [[Dual(Q[b][h][a][d], dQ[b][h][a][d]) for d in range(D)] for a in range(L)]
            k = [[Dual(K[b][h][a][d], dK[b][h][a][d]) for d in range(D)] for a in range(L)]
            v = [[Dual(V[b][h][a][d], dV[b][h][a][d]) for d in range(D)] for a in range(L)]
            Oh, dOh, Lh, dLh = [], [], [], []
            for a in range(L):
                keys = [c for c in range(L) if allowed[a, c]]
                if not keys:
                    Oh.append([0.0] * D); dOh.append([0.0] * D)
                    Lh.append(-math.inf); dLh.append(0.0)
                    continue
                scores = {}
                for c in keys:
                    acc = Dual(0.0)
                    for d in range(D):
                        acc = acc + q[a][d] * k[c][d]
                    scores[c] = acc * s
                # a constant shift (zero tangent) leaves softmax and its derivative unchanged
                shift = max(sc.x for sc in scores.values())
                w = {c: (scores[c] - shift).exp() for c in keys}
                den = Dual(0.0)
                for c in keys:
                    den = den + w[c]
                row, drow = [], []
                for d in range(D):
                    num = Dual(0.0)
                    for c in keys:
                        num = num + w[c] * v[c][d]
                    o = num / den
                    row.append(o.x); drow.append(o.t)
                lse = den.log() + shift
                Oh.append(row); dOh.append(drow); Lh.append(lse.x); dLh.append(lse.t)
            Ob.append(Oh); dOb.append(dOh); Lb.append(Lh); dLb.append(dLh)
        O.append(Ob); dO.append(dOb); LSE.append(Lb); dLSE.append(dLb)
    return O, dO, LSE, dLSE
