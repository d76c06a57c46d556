"""Writes the hand-derived alpha-entmax fixtures in this folder.

Every value below is the closed-form solution of Eq. 3 (sum_j [x_j - tau]_+^gamma
= 1, gamma = 1/(alpha-1)) on a support found by hand; the `derivation` string
records the algebra.  The `alg1_*` fixtures hold the iterates of Algorithm 1
(Halley-bisection, Sec. 3.1) in exact rational arithmetic, on rows whose
bracket ends are rational; their first iterate is also derived by hand.
Nothing here calls the GPU path or the oracle.
Run from the repository root: python tests/golden/make_golden.py
"""
import json
import math
import os
from fractions import Fraction

HERE = os.path.dirname(os.path.abspath(__file__))


def examples():
    ex = []
    ex.append(dict(name="sparsemax_three", alpha=2.0, x=[0.8, 0.4, 0.0],
                   derivation="gamma=1; support {0,1}: (0.8-t)+(0.4-t)=1 -> t=0.1; x_2=0 <= t",
                   tau=0.1, p=[0.7, 0.3, 0.0],
                   cite="Eq. 2, Eq. 3 (alpha=2: Euclidean projection onto the simplex, Sec. 3.1)"))
    t = (3 - math.sqrt(7)) / 4
    ex.append(dict(name="entmax15_three", alpha=1.5, x=[1.0, 0.5, 0.0],
                   derivation="gamma=2; support {0,1}: (1-t)^2+(0.5-t)^2=1 -> 2t^2-3t+1/4=0 "
                              "-> t=(3-sqrt(7))/4; x_2=0 <= t",
                   tau=t, p=[(1 - t) ** 2, (0.5 - t) ** 2, 0.0], cite="Eq. 2, Eq. 3 with alpha=1.5"))
    ex.append(dict(name="entmax15_uniform", alpha=1.5, x=[0.3, 0.3, 0.3, 0.3],
                   derivation="gamma=2; all equal: 4 (0.3-t)^2 = 1 -> t = 0.3 - 1/2 = -0.2 "
                              "(= max - n^(1-alpha))",
                   tau=-0.2, p=[0.25] * 4, cite="Eq. 3; upper end of the bracket of Algorithm 1"))
    ex.append(dict(name="entmax15_onehot", alpha=1.5, x=[2.0, 1.0, 0.25],
                   derivation="gamma=2; support {0}: (2-t)^2 = 1 -> t = 1 (= max - 1); x_1 = 1 <= t",
                   tau=1.0, p=[1.0, 0.0, 0.0],
                   cite="Eq. 2 (s <= tau/(alpha-1) gives zero); lower end of the bracket of Algorithm 1"))
    a = 0.9
    t4 = a - 2 ** -0.25
    ex.append(dict(name="entmax125_pair", alpha=1.25, x=[a, a, -1.0],
                   derivation="gamma=4; support {0,1}: 2 (0.9-t)^4 = 1 -> t = 0.9 - 2^(-1/4); x_2=-1 <= t",
                   tau=t4, p=[0.5, 0.5, 0.0], cite="Eq. 2, Eq. 3 with alpha=1.25"))
    ex.append(dict(name="sparsemax_five", alpha=2.0, x=[0.6, -3.0, 1.0, -0.2, 0.9],
                   derivation="gamma=1; support {0,2,4}: 2.5 - 3t = 1 -> t = 0.5; -0.2 <= t",
                   tau=0.5, p=[0.1, 0.0, 0.5, 0.0, 0.4], cite="Eq. 2, Eq. 3 (alpha=2)"))
    return ex


def alg1_exact(x, gamma, n_pow, iters):
    """Algorithm 1 in exact arithmetic for an integer gamma: the bracket
    [max x - 1, max x - n^(1-alpha)] (n_pow = n^(1-alpha), rational here),
    tau = its midpoint; each iteration evaluates f, f', f'' (Eq. 3, 6, 7) over
    the strict support x > tau, applies B_f (Eq. 4; hi <- tau if f < 0, else
    lo <- tau), then takes the Halley value H_f (Eq. 5) if it lies in
    [lo, hi], else the midpoint.  Returns tau before each iteration and after
    the last."""
    m = max(x)
    lo, hi = m - 1, m - n_pow
    tau = (lo + hi) / 2
    out = []
    for _ in range(iters):
        out.append(tau)
        z = [xi - tau for xi in x if xi > tau]
        f = sum(zi ** gamma for zi in z) - 1
        f1 = -gamma * sum(zi ** (gamma - 1) for zi in z)
        f2 = gamma * (gamma - 1) * sum(zi ** (gamma - 2) for zi in z)
        if f < 0:
            hi = tau
        else:
            lo = tau
        den = 2 * f1 * f1 - f * f2
        th = tau - 2 * f * f1 / den if den != 0 else None
        tau = th if th is not None and lo <= th <= hi else (lo + hi) / 2
    out.append(tau)
    return out


def alg1_examples():
    ex = []
    x = [Fraction(1), Fraction(3, 4), Fraction(1, 4), Fraction(0)]
    it = alg1_exact(x, 2, Fraction(1, 2), 3)
    ex.append(dict(name="alg1_trace_a15", alpha=1.5, x=[float(v) for v in x], iters=3,
                   tau=[float(t) for t in it], tau_exact_first=[str(t) for t in it[:2]],
                   derivation="gamma=2, n=4: lo=1-1=0, hi=1-4^(-1/2)=1/2, tau0=1/4; support {1, 3/4}: "
                              "f=(3/4)^2+(1/2)^2-1=-3/16 -> hi=1/4; f'=-2(3/4+1/2)=-5/2; "
                              "f''=2*1*2=4; H=1/4-2(-3/16)(-5/2)/(2(25/4)+(3/16)4)=1/4-15/212=19/106 "
                              "in [0, 1/4] (a Newton step would give 1/4-(3/16)/(5/2)=7/40)",
                   cite="Algorithm 1 (Sec. 3.1), Eq. 3-7"))
    x = [Fraction(1), Fraction(3, 4)] + [Fraction(0)] * 14
    it = alg1_exact(x, 4, Fraction(1, 2), 3)
    ex.append(dict(name="alg1_trace_a125", alpha=1.25, x=[float(v) for v in x], iters=3,
                   tau=[float(t) for t in it], tau_exact_first=[str(t) for t in it[:2]],
                   derivation="gamma=4, n=16: lo=0, hi=1-16^(-1/4)=1/2, tau0=1/4; support {1, 3/4}: "
                              "f=(3/4)^4+(1/2)^4-1=-159/256 -> hi=1/4; f'=-4((3/4)^3+(1/2)^3)=-35/16; "
                              "f''=12((3/4)^2+(1/2)^2)=39/4; H=1/4-2(-159/256)(-35/16)/"
                              "(2(35/16)^2+(159/256)(39/4))=4871/64004 "
                              "(f'' with gamma instead of gamma(gamma-1) would differ)",
                   cite="Algorithm 1 (Sec. 3.1), Eq. 3-7"))
    return ex


if __name__ == "__main__":
    for e in examples() + alg1_examples():
        with open(os.path.join(HERE, e["name"] + ".json"), "w") as f:
            json.dump(e, f, indent=1)
