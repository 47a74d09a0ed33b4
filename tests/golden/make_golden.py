"""Writes tiny_exact.json: a tiny rational codec case and its exact results.

The expected values are computed only by the oracle's exact (Fraction)
implementation.  Inputs are dyadic rationals that bf16 and fp32 represent
exactly; U's columns are orthonormal with entries in {0, +-1/2}.

Run from the repository root:  python tests/golden/make_golden.py
"""
import json
import os
import sys
from fractions import Fraction as F

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))))
from oracle import exact  # noqa: E402

h = F(1, 2)
# d = 8, k = 3: three orthonormal columns with entries 0 or +-1/2.
U = [[h, h, 0], [h, -h, 0], [h, h, 0], [h, -h, 0],
     [0, 0, h], [0, 0, h], [0, 0, -h], [0, 0, -h]]
# vocab 5, n_pos 3, N = 4 rows; values on a 1/8 grid.
E = [[F(((3 * v + 5 * r) % 11) - 5, 8) for r in range(8)] for v in range(5)]
P = [[F(((7 * p + 3 * r) % 9) - 4, 16) for r in range(8)] for p in range(3)]
tok = [4, 0, 2, 4]
pos = [0, 1, 2, 0]
Ctrue = [[F(3, 2), F(-1, 4), F(5, 8)], [F(0), F(7, 4), F(-2)],
         [F(-9, 8), F(1, 2), F(1, 4)], [F(2), F(-3, 8), F(-1, 2)]]
# X = E[tok] + P[pos] + Ctrue U^T + an off-subspace term on coordinates
# orthogonal to every column (e.g. e0 - e2 is orthogonal to all three).
off = [[F(1, 8), 0, F(-1, 8), 0, 0, 0, 0, 0], [0, 0, 0, 0, 0, 0, 0, 0],
       [0, F(1, 4), 0, F(-1, 4), 0, 0, 0, 0], [0, 0, 0, 0, F(1, 8), F(-1, 8), 0, 0]]
X = exact.decompress(Ctrue, U, tok, E, P, pos)
X = [[X[i][r] + off[i][r] for r in range(8)] for i in range(4)]
G = [[F(((5 * i + 3 * r) % 13) - 6, 4) for r in range(8)] for i in range(4)]
W = [[F(((2 * r + 7 * c) % 9) - 4, 8) for c in range(6)] for r in range(8)]

C = exact.compress(X, U, tok, E, P, pos)
Xrec = exact.decompress(C, U, tok, E, P, pos)
Cg = exact.compress(G, U)
Grec = exact.decompress(Cg, U)
Wp = exact.project_weights(W, U)


def s(m):
    return [[str(F(v)) for v in row] for row in m]


out = {
    "about": "Tiny exact codec case; expected values from oracle.exact (Fraction).",
    "d": 8, "k": 3, "vocab": 5, "n_pos": 3, "N": 4,
    "U": s(U), "E": s(E), "P": s(P), "tok": tok, "pos": pos, "X": s(X), "G": s(G), "W": s(W),
    "C_true": s(Ctrue),
    "expect": {"C": s(C), "X_rec": s(Xrec), "Cg": s(Cg), "G_rec": s(Grec), "W_proj": s(Wp)},
}
path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_exact.json")
with open(path, "w") as f:
    json.dump(out, f, indent=1)
print("wrote", path)
