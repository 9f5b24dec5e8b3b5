"""Exact transform synthesis for F(m, r) (oracle; test infrastructure only).

Follows §2.1: the fast vector convolution of Algorithm 1 reduces the
polynomial product s(x) = g(x) d(x) modulo m(x) = prod_k m^(k)(x) with pairwise
coprime factors (Theorem 1):

  (1) residues          g^(k) = g mod m^(k),  d^(k) = d mod m^(k)
  (2) residue products  s^(k) = g^(k) d^(k) mod m^(k)
  (3) reconstruction    s = sum_k s^(k) a^(k)  (mod m),
                        a^(k) = 1 mod m^(k), 0 mod m^(j) (j != k)

With linear factors m^(k)(x) = x - p_k the residues are evaluations and each
residue product is one scalar multiplication (the Cook-Toom case the paper's
matrices come from, §2.2).  Using alpha-1 finite points for a product of degree
alpha-1 leaves the top coefficient undetermined (Theorem 1 needs deg m >= deg s
with uniqueness only below), so, as in the printed matrices of §2.2 and §3.3,
the leading coefficient g_{r-1} u_{mo-1} is carried by one extra product, the
"point at infinity":  s = [sum_k s^(k) a^(k) mod m] + g_{r-1} u_{mo-1} m(x).

That gives the convolution form of eq. (1), s = A_cv[(C g) . (B u)], for a
length-mo vector u.  The layer of eq. (2) is a correlation; correlation with
g is the transpose of convolution with g, so

  A^T (m x alpha)      = B^T        (evaluation of u, transposed)
  B^T (alpha x alpha)  = A_cv^T     (reconstruction polynomials as rows)
  G   (alpha x r)      = C          (evaluation of g)

and y_i = sum_j A^T[i,j] (G g)_j (B^T d)_j = sum_k g_k d_{i+k}.

Two readings fix the remaining freedom (any diagonal rescaling of the three
matrices is equally correct):

* the CRT constant 1/M_k(p_k) of each reconstruction polynomial is moved from
  B^T into G (the cached kernel side), as the printed matrices do;
* if the x^1 coefficient of m(x) is negative, B^T rows 0 and alpha-1, G row 0
  and A^T column alpha-1 are negated.  This is the sign convention under which
  the F(2,3) matrices printed in §2.2 are reproduced entry for entry.

Pins: tests/test_oracle_toomcook.py checks the printed F(2,3) (§2.2) and
F(4,3) (§3.3) matrices entry for entry, Table 1's zero fractions and speed-ups,
and A^T[(G g) . (B^T d)] == correlation(g, d) exactly by brute force.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple

Poly = List[Fraction]          # ascending coefficients
Mat = List[List[Fraction]]


# ---------------------------------------------------------------- polynomials
def _trim(p: Sequence[Fraction]) -> Poly:
    p = list(p)
    while len(p) > 1 and p[-1] == 0:
        p.pop()
    return p


def poly_mul(a: Sequence[Fraction], b: Sequence[Fraction]) -> Poly:
    out = [Fraction(0)] * (len(a) + len(b) - 1)
    for i, ai in enumerate(a):
        for j, bj in enumerate(b):
            out[i + j] += ai * bj
    return _trim(out)


def poly_add(a: Sequence[Fraction], b: Sequence[Fraction]) -> Poly:
    n = max(len(a), len(b))
    return _trim([(a[i] if i < len(a) else 0) + (b[i] if i < len(b) else 0)
                  for i in range(n)])


def poly_scale(a: Sequence[Fraction], s) -> Poly:
    return _trim([Fraction(s) * c for c in a])


def poly_divmod(a: Sequence[Fraction], b: Sequence[Fraction]) -> Tuple[Poly, Poly]:
    a = _trim(a)
    b = _trim(b)
    if len(b) == 1 and b[0] == 0:
        raise ZeroDivisionError("polynomial division by zero")
    db = len(b) - 1
    rem = [Fraction(c) for c in a]
    if len(rem) - 1 < db:
        return [Fraction(0)], _trim(rem)
    q = [Fraction(0)] * (len(rem) - db)
    for shift in range(len(rem) - 1 - db, -1, -1):      # schoolbook long division
        coef = rem[shift + db] / b[db]
        q[shift] = coef
        for i, bi in enumerate(b):
            rem[shift + i] -= coef * bi
    return _trim(q), _trim(rem[:db] if db > 0 else [Fraction(0)])


def poly_mod(a, b) -> Poly:
    return poly_divmod(a, b)[1]


def poly_inverse_mod(a, mod) -> Poly:
    """a^{-1} mod `mod` by the extended Euclidean algorithm (a, mod coprime)."""
    r0, r1 = _trim(mod), poly_mod(a, mod)
    s0, s1 = [Fraction(0)], [Fraction(1)]
    while not (len(r1) == 1 and r1[0] == 0):
        q, r2 = poly_divmod(r0, r1)
        s2 = poly_add(s0, poly_scale(poly_mul(q, s1), -1))
        r0, r1, s0, s1 = r1, r2, s1, s2
    if len(r0) != 1:
        raise ValueError("moduli are not coprime")
    return poly_mod(poly_scale(s0, 1 / r0[0]), mod)


def poly_eval(a, x) -> Fraction:
    acc = Fraction(0)
    for c in reversed(a):
        acc = acc * x + c
    return acc


def _pad(p: Sequence[Fraction], n: int) -> Poly:
    p = list(p)
    if len(p) > n:
        if any(c != 0 for c in p[n:]):
            raise ValueError("polynomial does not fit")
        p = p[:n]
    return p + [Fraction(0)] * (n - len(p))


def residue_map(mod: Sequence[Fraction], n_coeffs: int) -> Mat:
    """Matrix of the linear map (coefficients of a degree < n_coeffs polynomial)
    -> (coefficients of its remainder mod `mod`): column j = x^j mod `mod`."""
    deg = len(_trim(mod)) - 1
    cols = []
    for j in range(n_coeffs):
        xj = [Fraction(0)] * j + [Fraction(1)]
        cols.append(_pad(poly_mod(xj, mod), max(deg, 1)))
    return [[cols[j][i] for j in range(n_coeffs)] for i in range(max(deg, 1))]


# -------------------------------------------------------- Algorithm 1 (conv)
def as_fraction(p) -> Fraction:
    if isinstance(p, Fraction):
        return p
    if isinstance(p, str):
        return Fraction(p)
    if isinstance(p, int):
        return Fraction(p)
    f = Fraction(p).limit_denominator(1 << 20)
    if float(f) != float(p):
        raise ValueError(f"point {p!r} is not a small rational")
    return f


def toom_cook_convolution(mo: int, r: int, points: Sequence) -> Tuple[Mat, Mat, Mat]:
    """Convolution form s = A_cv[(C g) . (B u)] for len(u)=mo, len(g)=r, built
    by the three steps of Algorithm 1 over m^(k)(x) = x - p_k plus infinity.

    Returns (A_cv alpha x alpha, B alpha x mo, C alpha x r)."""
    alpha = mo + r - 1
    pts = [as_fraction(p) for p in points]
    if len(pts) != alpha - 1:
        raise ValueError(f"F({mo},{r}) needs {alpha - 1} finite points, got {len(pts)}")
    if len(set(pts)) != len(pts):
        raise ValueError("interpolation points must be distinct")
    moduli = [[-p, Fraction(1)] for p in pts]            # m^(k)(x) = x - p_k
    m_full = [Fraction(1)]
    for mk in moduli:
        m_full = poly_mul(m_full, mk)                    # m(x) = prod_k m^(k)(x)

    # Step (1): residue maps of g and d for every modulus (evaluations here).
    C_rows, B_rows = [], []
    for mk in moduli:
        C_rows.append(residue_map(mk, r)[0])
        B_rows.append(residue_map(mk, mo)[0])
    # The point at infinity picks the leading coefficients.
    C_rows.append([Fraction(0)] * (r - 1) + [Fraction(1)])
    B_rows.append([Fraction(0)] * (mo - 1) + [Fraction(1)])

    # Step (2) is the element-wise product of the residues (one scalar each).
    # Step (3): CRT reconstruction polynomials a^(k) = M_k * (M_k^{-1} mod m^(k)).
    cols = []
    for k, mk in enumerate(moduli):
        Mk = [Fraction(1)]
        for j, mj in enumerate(moduli):
            if j != k:
                Mk = poly_mul(Mk, mj)
        ak = poly_mod(poly_mul(Mk, poly_inverse_mod(Mk, mk)), m_full)
        cols.append(_pad(ak, alpha))
    cols.append(_pad(m_full, alpha))                     # infinity: + lead * m(x)
    A_cv = [[cols[j][i] for j in range(alpha)] for i in range(alpha)]
    return A_cv, B_rows, C_rows


def _transpose(M: Mat) -> Mat:
    return [list(row) for row in zip(*M)]


def winograd_matrices(m: int, r: int, points: Sequence) -> Tuple[Mat, Mat, Mat]:
    """Exact (A^T, B^T, G) for the correlation F(m, r) from `points`
    (alpha-1 distinct finite points; infinity is implied).

    A^T is m x alpha, B^T is alpha x alpha, G is alpha x r, so that
    y = A^T [(G g) . (B^T d)] for a length-alpha input window d."""
    alpha = m + r - 1
    A_cv, B, C = toom_cook_convolution(m, r, points)
    AT = _transpose(B)                   # m x alpha
    BT = _transpose(A_cv)                # alpha x alpha
    G = [list(row) for row in C]         # alpha x r
    # Move each reconstruction polynomial's constant factor into G.
    pts = [as_fraction(p) for p in points]
    for k, pk in enumerate(pts):
        Nk = Fraction(1)
        for j, pj in enumerate(pts):
            if j != k:
                Nk *= (pk - pj)
        BT[k] = [c * Nk for c in BT[k]]
        G[k] = [c / Nk for c in G[k]]
    # Sign convention that reproduces the printed F(2,3) matrices.
    m_full = [Fraction(1)]
    for p in pts:
        m_full = poly_mul(m_full, [-p, Fraction(1)])
    x1 = m_full[1] if len(m_full) > 1 else Fraction(0)
    if x1 < 0:
        BT[0] = [-c for c in BT[0]]
        BT[alpha - 1] = [-c for c in BT[alpha - 1]]
        G[0] = [-c for c in G[0]]
        for i in range(m):
            AT[i][alpha - 1] = -AT[i][alpha - 1]
    return AT, BT, G


# Default interpolation points (infinity implied).  F(2,3) uses the set of the
# printed §2.2 matrices; F(4,3) uses {0, 1, -1, 2, -2}, which keeps the fp32
# error of the 3-D case well inside the m = 4 tolerance (the paper's printed
# F(4,3) set {0, 1, -1, 1/3, -1/3} is supported as an explicit choice).
DEFAULT_POINTS = {
    (2, 3): (0, 1, -1),
    (4, 3): (0, 1, -1, 2, -2),
    (2, 2): (0, 1),
    (3, 2): (0, 1, -1),
}

PAPER_F43_POINTS = (0, 1, -1, Fraction(1, 3), Fraction(-1, 3))


def default_points(m: int, r: int):
    if (m, r) in DEFAULT_POINTS:
        return DEFAULT_POINTS[(m, r)]
    # A symmetric ladder 0, 1, -1, 2, -2, 1/2, -1/2, ... for other sizes.
    ladder = [Fraction(0), Fraction(1), Fraction(-1), Fraction(2), Fraction(-2),
              Fraction(1, 2), Fraction(-1, 2), Fraction(3), Fraction(-3),
              Fraction(1, 3), Fraction(-1, 3)]
    need = m + r - 2
    if need > len(ladder):
        raise ValueError("no default points for this size")
    return tuple(ladder[:need])


def to_float(M: Mat) -> List[List[float]]:
    """Round every exact entry once to the nearest double."""
    return [[float(c) for c in row] for row in M]
