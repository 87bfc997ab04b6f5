"""Winograd transform matrices, exact rationals (Sec. II, "Beyond Winograd 2x2").

The F(4x4,3x3) matrices are the ones printed in Sec. II; the text there names
the root points {0, 1, -1, 1/2, 1/2}, which is garbled (a point is repeated),
so the printed matrices are taken as authoritative.  G is printed as
(1/3) * [[3/4,0,0], [-1/2,-1/2,-1/2], [-1/2,1/2,-1/2], [1/8,1/4,1/2],
[1/8,-1/4,1/2], [0,0,3]]; it is stored here entry by entry as Fractions.

Conventions used throughout the oracle:
  * a tile d is 6x6 with d[r][c], r the row (height) index;
  * V = B^T d B, tap t = 6*a + b addresses V[a][b];
  * U = G f G^T for a 3x3 kernel f;
  * Y = A^T M A is the 4x4 output tile (Eq. winograd).
"""
from fractions import Fraction as Fr

import numpy as np

# --- F(4x4, 3x3) -----------------------------------------------------------
BT4 = [
    [4, 0, -5, 0, 1, 0],
    [0, -4, -4, 1, 1, 0],
    [0, 4, -4, -1, 1, 0],
    [0, -2, -1, 2, 1, 0],
    [0, 2, -1, -2, 1, 0],
    [0, 4, 0, -5, 0, 1],
]

_third = Fr(1, 3)
G4 = [
    [_third * Fr(3, 4), Fr(0), Fr(0)],
    [_third * Fr(-1, 2), _third * Fr(-1, 2), _third * Fr(-1, 2)],
    [_third * Fr(-1, 2), _third * Fr(1, 2), _third * Fr(-1, 2)],
    [_third * Fr(1, 8), _third * Fr(1, 4), _third * Fr(1, 2)],
    [_third * Fr(1, 8), _third * Fr(-1, 4), _third * Fr(1, 2)],
    [Fr(0), Fr(0), _third * 3],
]

AT4 = [
    [1, 1, 1, 1, 1, 0],
    [0, 1, -1, 2, -2, 0],
    [0, 1, 1, 4, 4, 0],
    [0, 1, -1, 8, -8, 1],
]

# --- F(2x2, 3x3), same section ---------------------------------------------
BT2 = [
    [1, 0, -1, 0],
    [0, 1, 1, 0],
    [0, -1, 1, 0],
    [0, 1, 0, -1],
]
G2 = [
    [Fr(1), Fr(0), Fr(0)],
    [Fr(1, 2), Fr(1, 2), Fr(1, 2)],
    [Fr(1, 2), Fr(-1, 2), Fr(1, 2)],
    [Fr(0), Fr(0), Fr(1)],
]
AT2 = [
    [1, 1, 1, 0],
    [0, 1, -1, -1],
]


def g_times(k, G):
    """k * G as a list of integers; raises if any entry is not an integer."""
    out = []
    for row in G:
        r = []
        for v in row:
            s = v * k
            if s.denominator != 1:
                raise ValueError("k*G is not integral")
            r.append(int(s))
        out.append(r)
    return out


# 24 * G4 is integral; the exact weight transform works with it and divides
# by 24^2 = 576 at the end.
G4_DEN = 24
G4_INT = g_times(G4_DEN, G4)


def as_int_array(m):
    return np.array(m, dtype=np.int64)


def as_f64_array(m):
    return np.array([[float(v) for v in row] for row in m], dtype=np.float64)


BT4_I = as_int_array(BT4)
AT4_I = as_int_array(AT4)
G4_F = as_f64_array(G4)
G4_INT_I = as_int_array(G4_INT)
