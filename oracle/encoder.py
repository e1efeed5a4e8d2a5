"""Nearest-point encoder of 24-weight blocks and its retention (oracle,
test-only).

Paper passages followed:
* Sec. 3.1, Eq. 2 (shape-gain): a block is rebuilt as
  w_j = y_j / ||y|| * gain[g] * sigma_row, so the encoder looks for the kept
  lattice point whose direction is closest to the block, then for the gain.
* Sec. 3.1: the search is not exhaustive; at two trial scales it keeps
  candidates per section and joins the best of them over the trellis.
* Sec. 3.2-3.3: a kept point is a trellis path (three pattern bytes of a
  Golay codeword), a parity p and three rank rows: sections 1 and 3 read the
  2,048 cheapest rows of their class (class r, and r3 = p xor r xor delta by
  Eq. 3), the middle section its own list of the 2,048 cheapest overall,
  whose position gives its class delta.
* Sec. 3.5: retention is the rate the Gaussian rate-distortion limit needs
  for the encoder's mean squared error, as a fraction of the rate the code
  spends (48 bits per 24 weights); 88.80 % on 20,000 Gaussian blocks.

Reading (the paper gives no more than the sentences above):
1. The norm of the block, n2 = sum_j w_j^2, and every dot product below are
   float64 sums in coordinate order j = 0..23.
2. For each trial radius a: integer targets T_j = rint(w_j * (a * 2^16 /
   sqrt(n2))) and the kept point y maximising
       S(y) = sum_j (2 T_j y_j - 2^16 y_j^2),
   i.e. the kept point nearest to a w / ||w|| on a grid of 2^-16.  S splits
   over the sections: for every parity p, pattern byte P and class, the
   best row of the section's list of that class (the first of equal
   scores); then the best sum over the 4096 trellis paths and the parities
   r, delta.  Equal sums go to the smallest key
       (s8 | p << 6 | r << 7 | b1 << 8 | b2 << 9 | b3 << 13) * 2 + delta.
   Every score is an exact integer.
3. Of the two trial points, the one with the larger <w, y> / ||y|| (the
   first on equality).
4. The gain bit g minimising (gain[g] sigma - <w, y> / ||y||)^2 (g = 0 on
   equality).  A block whose n2 is zero or not finite gives the word 0
   (the origin, g = 0).
5. The word is the one that decodes to (y, g).

Pins (tests): with the trial radius equal to ||y|| of a decoded word y, and
sigma = 1 with ||w|| = gain[g], the encoder returns that word (every field
of every section, through the search); the result beats every word that
differs from it in one field (each row index over its whole list, each
trellis edge) and a random sample of words; retention is compared with the
paper's figure on the GPU path's 20,000 blocks.
"""

import math

import numpy as np

from . import codec, tables

SCALE = 1 << 16


def _lists():
    """The row lists of the three sections, per class: sections 1 and 3 use
    the two halves of the table, the middle section its own list."""
    rt = tables.rank_table()
    rows, mid, n0 = rt["rows"], rt["middle"], rt["n0"]
    outer = (rows[:tables.N_ROWS_HALF], rows[tables.N_ROWS_HALF:])
    middle = (mid[:n0], mid[n0:])
    return (outer, middle, outer), n0


def _ranks(lst) -> np.ndarray:
    lst = np.asarray(lst, dtype=np.int64)
    return (lst[:, None] >> (4 * np.arange(8))) & 0xF


def section_best(T8, lists):
    """best[p, P, c], arg[p, P, c]: the best score of a section with integer
    targets T8 over the class-c list for parity p and pattern byte P, and
    the index in that list of the first row reaching it."""
    V = tables.value_lists()
    T8 = np.asarray(T8, dtype=np.int64)
    E = 2 * T8[:, None, None] * V[None] - SCALE * V[None] ** 2       # [j, o, rank]
    bits = (np.arange(256)[:, None] >> np.arange(8)) & 1             # [P, j]
    best = np.zeros((2, 256, 2), dtype=np.int64)
    arg = np.zeros((2, 256, 2), dtype=np.int64)
    for p in (0, 1):
        O = p + 2 * bits
        for c in (0, 1):
            rk = _ranks(lists[c])
            S = np.zeros((256, rk.shape[0]), dtype=np.int64)
            for j in range(8):
                S += E[j][O[:, j]][:, rk[:, j]]
            best[p, :, c] = S.max(axis=1)
            arg[p, :, c] = S.argmax(axis=1)
    return best, arg


def _paths():
    """All 4096 trellis paths: (s8, b1, b2, b3) and their pattern bytes."""
    s8, b1, b2, b3 = np.meshgrid(np.arange(64), np.arange(2), np.arange(16), np.arange(2), indexing="ij")
    s8, b1, b2, b3 = (a.ravel() for a in (s8, b1, b2, b3))
    P1, P2, P3, _ = tables.walk(s8, b1, b2, b3)
    return s8, b1, b2, b3, P1.astype(np.int64), P2.astype(np.int64), P3.astype(np.int64)


def nearest_point(T):
    """The kept point maximising S for integer targets T (24 values, block
    order): returns (score, fields dict without g, y)."""
    (l1, l2, l3), n0 = _lists()
    T = np.asarray(T, dtype=np.int64)
    b = [section_best(T[8 * s:8 * s + 8], lst) for s, lst in enumerate((l1, l2, l3))]
    s8, b1, b2, b3, P1, P2, P3 = _paths()
    best, key, pick = None, None, None
    for p in (0, 1):
        for r in (0, 1):
            for d in (0, 1):
                r3 = p ^ r ^ d
                tot = b[0][0][p, P1, r] + b[1][0][p, P2, d] + b[2][0][p, P3, r3]
                k = (s8 | p << 6 | r << 7 | b1 << 8 | b2 << 9 | b3 << 13) * 2 + d
                m = tot.max()
                i = np.flatnonzero(tot == m)
                i = i[np.argmin(k[i])]
                if best is None or m > best or (m == best and k[i] < key):
                    best, key, pick = int(m), int(k[i]), (p, r, d, int(i))
    p, r, d, i = pick
    r3 = p ^ r ^ d
    rows = (l1[r][b[0][1][p, P1[i], r]], l2[d][b[1][1][p, P2[i], d]], l3[r3][b[2][1][p, P3[i], r3]])
    V = tables.value_lists()
    y = np.zeros(24, dtype=np.int64)
    for s, (P, row) in enumerate(zip((P1[i], P2[i], P3[i]), rows)):
        for t in range(8):
            o = p + 2 * ((int(P) >> t) & 1)
            y[8 * s + t] = V[o, (int(row) >> (4 * t)) & 0xF]
    i2 = b[1][1][p, P2[i], d] + (n0 if d else 0)
    f = {"s8": int(s8[i]), "p": p, "r": r, "b1": int(b1[i]), "b2": int(b2[i]), "b3": int(b3[i]),
         "i1": int(b[0][1][p, P1[i], r]), "i2": int(i2), "i3": int(b[2][1][p, P3[i], r3])}
    return best, f, y


def score(T, y) -> int:
    """S(y) for integer targets T (the quantity the search maximises)."""
    T = np.asarray(T, dtype=np.int64)
    y = np.asarray(y, dtype=np.int64)
    return int(np.sum(2 * T * y - SCALE * y * y))


def _seq_dot(a, b) -> float:
    s = 0.0
    for u, v in zip(a, b):
        s += float(u) * float(v)
    return s


def targets(w, alpha):
    """Integer targets of a block at trial radius alpha (reading 1-2)."""
    n2 = _seq_dot(w, w)
    f = float(alpha) * float(SCALE) / math.sqrt(n2)
    return np.array([int(np.rint(float(v) * f)) for v in w], dtype=np.int64)


def encode_block(w, sigma, alphas):
    """Canonical word of one block of 24 float32 weights (block order) with
    row scale sigma (float32), searched at the trial radii `alphas`."""
    w = np.asarray(w, dtype=np.float32)
    n2 = _seq_dot(w, w)
    if not (n2 > 0.0 and n2 <= 1e300):        # zero or non-finite block
        return 0
    best_c, best_y, best_f = None, None, None
    for a in alphas:
        _, f, y = nearest_point(targets(w, a))
        ny = math.sqrt(_seq_dot(y, y))
        c = _seq_dot(w, y) / ny if ny > 0 else -math.inf
        if best_c is None or c > best_c:
            best_c, best_y, best_f = c, y, f
    G = tables.gain()
    gs = float(np.float32(sigma))
    e = [float(G[g]) * gs - best_c for g in (0, 1)]
    g = 1 if e[1] * e[1] < e[0] * e[0] else 0
    word = codec.encode(best_y, g)
    assert word is not None
    assert word == int(codec.pack_fields(g=g, **best_f))
    return word


def encode_blocks(w, sigma, alphas) -> np.ndarray:
    """uint64 words of blocks w [n, 24] with per-block scales sigma [n]."""
    w = np.asarray(w, dtype=np.float32).reshape(-1, 24)
    sigma = np.broadcast_to(np.asarray(sigma, dtype=np.float32), (w.shape[0],))
    return np.array([encode_block(w[i], sigma[i], alphas) for i in range(w.shape[0])], dtype=np.uint64)


def reconstruct(words, sigma) -> np.ndarray:
    """float64 [n, 24]: y / ||y|| * gain[g] * sigma (Eq. 2), the origin for y = 0."""
    y = np.asarray(codec.decode(words)[0], dtype=np.float64).reshape(-1, 24)
    g = codec.fields(words)["g"].reshape(-1)
    ny = np.sqrt((y * y).sum(axis=1))
    G = tables.gain().astype(np.float64)[g]
    s = np.where(ny > 0, G / np.where(ny > 0, ny, 1.0), 0.0)
    return y * (s * np.asarray(sigma, dtype=np.float64).reshape(-1))[:, None]


def retention(mse_per_weight: float, variance: float = 1.0, bits_per_weight: float = 2.0) -> float:
    """Rate of the Gaussian rate-distortion limit at this error, 0.5 log2(var / D),
    as a fraction of the rate spent."""
    return 0.5 * math.log2(variance / mse_per_weight) / bits_per_weight
