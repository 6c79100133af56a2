"""+-1 Hadamard matrices used by the online rotations R3 and R4.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper uses Hadamard matrices for the two online rotations (Sec. 3.1, "Additional
unabsorbed rotations"; Sec. 3.2 keeps R3/R4 as Hadamard) and defines a Hadamard
matrix in the footnote of Sec. 2.2.  That footnote's "entries +-sqrt(n)" is read as
"+-1 entries, applied as H / sqrt(n)" so that the rotation is orthonormal.  The paper
names no construction for sizes that are not powers of two; any Hadamard matrix is a
valid choice.  This module builds:

  * Sylvester S_b, b = 2^k, natural order: S[i, j] = (-1)^popcount(i & j).
  * Paley type II of order 2(q+1) for a prime q = 1 (mod 4)  (order 28 from q = 13).
  * Williamson of order 4m from four symmetric circulants of order m (order 172
    from m = 43), found by a deterministic meet-in-the-middle search over sign
    sequences that are constant on the cosets of a subgroup of (Z/m)* containing -1.

Every matrix returned satisfies H H^T = n I exactly (checked here and in the tests).
"""

from functools import lru_cache

import numpy as np


def sylvester(b: int) -> np.ndarray:
    """Sylvester-Hadamard matrix of order b = 2^k: S[i, j] = (-1)^popcount(i & j)."""
    if b < 1 or (b & (b - 1)) != 0:
        raise ValueError(f"Sylvester order must be a power of two, got {b}")
    i = np.arange(b, dtype=np.int64)
    bits = i[:, None] & i[None, :]
    pop = np.zeros_like(bits)
    while np.any(bits):
        pop += bits & 1
        bits >>= 1
    return np.where(pop % 2 == 0, 1, -1).astype(np.int8)


def _is_prime(q: int) -> bool:
    return q >= 2 and all(q % d for d in range(2, int(q ** 0.5) + 1))


def paley2(q: int) -> np.ndarray:
    """Paley type II Hadamard matrix of order 2(q+1), q prime with q = 1 (mod 4).

    chi is the quadratic character of GF(q); the Jacobsthal matrix is
    Q[i, j] = chi(j - i); the conference matrix is C = [[0, 1^T], [1, Q]], and
    H = C (x) [[1, 1], [1, -1]] + I (x) [[1, -1], [-1, -1]].
    """
    if not _is_prime(q) or q % 4 != 1:
        raise ValueError(f"Paley II needs a prime q = 1 mod 4, got {q}")
    squares = {(x * x) % q for x in range(1, q)}
    chi = np.array([0] + [1 if r in squares else -1 for r in range(1, q)], dtype=np.int64)
    idx = np.arange(q)
    jac = chi[(idx[None, :] - idx[:, None]) % q]
    conf = np.zeros((q + 1, q + 1), dtype=np.int64)
    conf[0, 1:] = 1
    conf[1:, 0] = 1
    conf[1:, 1:] = jac
    h = np.kron(conf, np.array([[1, 1], [1, -1]])) + np.kron(
        np.eye(q + 1, dtype=np.int64), np.array([[1, -1], [-1, -1]]))
    return h.astype(np.int8)


def _primitive_root(m: int) -> int:
    phi = m - 1
    factors = {p for p in range(2, phi + 1) if phi % p == 0 and _is_prime(p)}
    for g in range(2, m):
        if all(pow(g, phi // p, m) != 1 for p in factors):
            return g
    raise ValueError(f"no primitive root mod {m}")


def _circulant(first_row: np.ndarray) -> np.ndarray:
    m = first_row.shape[0]
    i = np.arange(m)
    return first_row[(i[None, :] - i[:, None]) % m]


def williamson(m: int, subgroup_order: int = 6) -> np.ndarray:
    """Williamson Hadamard matrix of order 4m (m prime), by deterministic search.

    Four symmetric +-1 circulants A, B, C, D of order m with A^2+B^2+C^2+D^2 = 4m I
    give the Hadamard matrix
        [[ A,  B,  C,  D],
         [-B,  A, -D,  C],
         [-C,  D,  A, -B],
         [-D, -C,  B,  A]].
    The condition is that the periodic autocorrelations of the four first rows sum to
    zero at every nonzero shift.  Candidates are first rows constant on each coset of
    the subgroup G of (Z/m)* of the given order (G must contain -1, which makes the
    circulant symmetric); their autocorrelation is then constant on cosets too, so one
    shift per coset is checked.  Candidate t has sign (-1)^bit0(t) at index 0 and
    (-1)^bit(j+1)(t) on coset g^j G.  The quadruple returned is the first one, in
    lexicographic order of (tA, tB, tC, tD) with tA <= tB <= tC <= tD, that satisfies
    the condition.
    """
    if not _is_prime(m) or (m - 1) % subgroup_order != 0:
        raise ValueError(f"unsupported Williamson order m={m}")
    g = _primitive_root(m)
    ncos = (m - 1) // subgroup_order
    h = pow(g, ncos, m)  # generator of the subgroup of the given order
    sub = {pow(h, k, m) for k in range(subgroup_order)}
    if (m - 1) not in sub:
        raise ValueError("subgroup must contain -1 for symmetric circulants")
    coset_of = np.full(m, -1, dtype=np.int64)
    for j in range(ncos):
        for s in sub:
            coset_of[(pow(g, j, m) * s) % m] = j
    ncand = 1 << (ncos + 1)

    def row(t: int) -> np.ndarray:
        signs = np.array([1 - 2 * ((t >> k) & 1) for k in range(ncos + 1)], dtype=np.int64)
        r = np.empty(m, dtype=np.int64)
        r[0] = signs[0]
        r[1:] = signs[1 + coset_of[1:]]
        return r

    reps = [pow(g, j, m) for j in range(ncos)]
    rows = [row(t) for t in range(ncand)]
    paf = np.array([[int(np.dot(r, np.roll(r, -s))) for s in reps] for r in rows], dtype=np.int64)

    pairs = {}
    for c in range(ncand):
        for d in range(c, ncand):
            pairs.setdefault(tuple(paf[c] + paf[d]), []).append((c, d))
    found = None
    for a in range(ncand):
        for b in range(a, ncand):
            for (c, d) in pairs.get(tuple(-(paf[a] + paf[b])), ()):
                if c >= b:
                    found = (a, b, c, d)
                    break
            if found:
                break
        if found:
            break
    if found is None:
        raise ValueError(f"no coset-constant Williamson quadruple for m={m}")
    A, B, C, D = (_circulant(rows[t]) for t in found)
    H = np.block([[A, B, C, D], [-B, A, -D, C], [-C, D, A, -B], [-D, -C, B, A]])
    return H.astype(np.int8)


@lru_cache(maxsize=None)
def _dense_factor_cached(n: int) -> np.ndarray:
    if n == 1:
        return np.ones((1, 1), dtype=np.int8)
    if n == 28:
        return paley2(13)
    if n == 172:
        return williamson(43)
    raise ValueError(f"no dense Hadamard factor registered for order {n}")


def dense_factor(n: int) -> np.ndarray:
    """The non-power-of-two Hadamard factor of order n (1, 28 or 172), as int8 +-1."""
    h = _dense_factor_cached(n).copy()
    check(h)
    return h


def check(h: np.ndarray) -> None:
    """Raise unless h is square with +-1 entries and H H^T = n I exactly."""
    n = h.shape[0]
    if h.shape != (n, n) or not np.all(np.abs(h.astype(np.int64)) == 1):
        raise ValueError("not a square +-1 matrix")
    g = h.astype(np.int64) @ h.astype(np.int64).T
    if not np.array_equal(g, n * np.eye(n, dtype=np.int64)):
        raise ValueError("H H^T != n I")
