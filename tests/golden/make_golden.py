"""Writes the hand-derived alpha-entmax fixtures in this folder.

Every value below is the closed-form solution of Eq. 3 (sum_j [x_j - tau]_+^gamma
= 1, gamma = 1/(alpha-1)) on a support found by hand; the `derivation` string
records the algebra.  Nothing here calls the GPU path or the oracle.
Run from the repository root: python tests/golden/make_golden.py
"""
import json
import math
import os

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


if __name__ == "__main__":
    for e in examples():
        with open(os.path.join(HERE, e["name"] + ".json"), "w") as f:
            json.dump(e, f, indent=1)
