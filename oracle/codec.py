"""Decode and encode of the 48-bit Tetra word (oracle, test-only).

Paper passages followed:
* Sec. 3.3: the word holds eight bits of state (s8, the shared parity p, and
  r, the k-parity of section 1), the edge choices b1, b2, b3, the gain bit g
  and three 11-bit row indices.  Eq. 3: the k-parity of section 3 is
  r3 = p xor r xor delta, where delta is the class of the middle row.
* Sec. 3.4 and Fig. 4: three trellis reads give the pattern bytes, three row
  reads give the rank vectors; the 24 values are then scaled by
  gain[g] * 1/sqrt(16m), with m recomputed from the decoded values.
* Eq. 1: y lies in the lattice when y_j = p + 2 c_j + 4 k_j with c a Golay
  codeword and sum_j k_j = p (mod 2).
* Eq. 2: the reconstructed weight is y_j / ||y|| * gain[g] * sigma_row with
  ||y|| = sqrt(16m).

Reading of the word layout (the drawing of the word is lost; ten fields,
8 + 6 + 33 + 1 = 48 bits; every 48-bit value is legal):
    bits 0-5 s8 | 6 p | 7 r | 8 b1 | 9-12 b2 | 13 b3 | 14 g |
    15-25 i1 | 26-36 i2 | 37-47 i3
stored as 6 little-endian bytes.  Block coordinate j = 8*s + t (section s,
position t) multiplies activation 24*blk + j.

Reading of the scale: s_blk = fl32(gain[g] * invnorm[m]) and the weight is
w_j = fl32(fl32(y_j * s_blk) * sigma_row) with sigma_row the fp16 row scale
widened to f32.

Pins (tests): every decoded point passes ``in_leech`` (independent of the
tables); nonzero points have m >= 2; the word 0 decodes to the origin;
``encode(decode(w)) == w`` for random words; bounds m <= 26, max|y| = 10.
"""

import numpy as np

from . import golay, tables

FIELDS = {  # name: (lsb, width)
    "s8": (0, 6), "p": (6, 1), "r": (7, 1), "b1": (8, 1), "b2": (9, 4),
    "b3": (13, 1), "g": (14, 1), "i1": (15, 11), "i2": (26, 11), "i3": (37, 11),
}


def fields(words) -> dict:
    w = np.asarray(words, dtype=np.uint64)
    return {k: ((w >> np.uint64(lsb)) & np.uint64((1 << n) - 1)).astype(np.int64)
            for k, (lsb, n) in FIELDS.items()}


def pack_fields(**f) -> np.ndarray:
    w = np.zeros(np.shape(f["s8"]), dtype=np.uint64)
    for k, (lsb, n) in FIELDS.items():
        v = np.asarray(f[k], dtype=np.uint64)
        assert np.all(v < (1 << n))
        w |= v << np.uint64(lsb)
    return w


def words_from_bytes(b: np.ndarray) -> np.ndarray:
    """[..., 6] uint8 little-endian -> uint64 words."""
    b = np.asarray(b, dtype=np.uint64)
    w = np.zeros(b.shape[:-1], dtype=np.uint64)
    for i in range(6):
        w |= b[..., i] << np.uint64(8 * i)
    return w


def words_to_bytes(w: np.ndarray) -> np.ndarray:
    w = np.asarray(w, dtype=np.uint64)
    return np.stack([((w >> np.uint64(8 * i)) & np.uint64(0xFF)).astype(np.uint8)
                     for i in range(6)], axis=-1)


def decode(words):
    """Decode words (any shape) into (y int8 [..., 24], m int, s_blk f32)."""
    words = np.asarray(words, dtype=np.uint64)
    shape = words.shape
    f = fields(words.reshape(-1))
    t = tables.trellis()
    rt = tables.rank_table()
    rows, middle = rt["rows"].astype(np.int64), rt["middle"].astype(np.int64)
    V = tables.value_lists()

    # trellis walk: the suffix read waits for s16 from the branch read
    p1 = t["prefixes"][2 * f["s8"] + f["b1"]].astype(np.int64)
    br = t["branches"][16 * f["s8"] + f["b2"]].astype(np.int64)
    p2, s16 = br & 0xFF, br >> 8
    p3 = t["suffixes"][2 * s16 + f["b3"]].astype(np.int64)

    # rank rows; the middle row's class is delta, Eq. 3 gives section 3's half
    rho1 = rows[N_HALF * f["r"] + f["i1"]]
    rho2 = middle[f["i2"]]
    delta = tables.cls_of(rho2)
    r3 = f["p"] ^ f["r"] ^ delta
    rho3 = rows[N_HALF * r3 + f["i3"]]

    n = words.size
    y = np.zeros((n, 24), dtype=np.int64)
    for s, (pat, rho) in enumerate(((p1, rho1), (p2, rho2), (p3, rho3))):
        for tt in range(8):
            c = (pat >> tt) & 1
            o = f["p"] + 2 * c
            rank = (rho >> (4 * tt)) & 0xF
            y[:, 8 * s + tt] = V[o, rank]

    sq = (y * y).sum(axis=1)
    assert np.all(sq % 16 == 0), "norm of a decoded point is not a multiple of 16"
    m = sq // 16
    assert np.all(m < 32)
    s_blk = (tables.gain()[f["g"]] * tables.invnorm()[m]).astype(np.float32)
    return (y.reshape(shape + (24,)).astype(np.int8), m.reshape(shape),
            s_blk.reshape(shape))


N_HALF = tables.N_ROWS_HALF


# --------------------------------------------------------------------------
# Lattice membership (Eq. 1), independent of the decoder tables
# --------------------------------------------------------------------------

def _golay_member(c: np.ndarray) -> np.ndarray:
    """Vectorised membership in the extended cyclic Golay code by polynomial
    division (same definition as ``golay.is_codeword``)."""
    a = (c & ((1 << 23) - 1)).astype(np.int64)
    g = golay.GEN_POLY
    for bit in range(22, 10, -1):
        a ^= ((a >> bit) & 1) * (g << (bit - 11))
    par = np.zeros_like(c)
    for i in range(24):
        par ^= (c >> i) & 1
    return (a == 0) & (par == 0)


def in_leech(y) -> np.ndarray:
    """Eq. 1 membership of integer vectors y [..., 24] given in block
    coordinate order; returns a bool array."""
    y = np.asarray(y, dtype=np.int64)
    flat = y.reshape(-1, 24)
    p = flat[:, 0] & 1
    same = np.all((flat & 1) == p[:, None], axis=1)
    cbits = ((flat - p[:, None]) >> 1) & 1
    k = (flat - p[:, None] - 2 * cbits) // 4
    perm = golay.block_order()
    c = np.zeros(flat.shape[0], dtype=np.int64)
    for j in range(24):
        c |= cbits[:, j] << perm[j]
    ok = same & _golay_member(c) & (((k.sum(axis=1) - p) & 1) == 0)
    return ok.reshape(y.shape[:-1])


# --------------------------------------------------------------------------
# Encode: the inverse map, for round trips
# --------------------------------------------------------------------------

class _Inverse:
    def __init__(self):
        t = tables.trellis()
        self.path = {}
        for s8 in range(64):
            for b1 in range(2):
                for b2 in range(16):
                    for b3 in range(2):
                        p1, p2, p3, _ = tables.walk(s8, b1, b2, b3)
                        self.path[(int(p1), int(p2), int(p3))] = (s8, b1, b2, b3)
        rt = tables.rank_table()
        rows = rt["rows"]
        self.half = [{int(v): i for i, v in enumerate(rows[:N_HALF])},
                     {int(v): i for i, v in enumerate(rows[N_HALF:])}]
        self.mid = {int(v): i for i, v in enumerate(rt["middle"])}
        V = tables.value_lists()
        self.rank = {(o, int(V[o, r])): r for o in range(4) for r in range(8)}
        del t


_inv = None


def encode(y, g: int):
    """Word for the lattice point y (block order) and gain bit g, or None if
    the point is outside the kept codebook."""
    global _inv
    if _inv is None:
        _inv = _Inverse()
    y = [int(v) for v in y]
    p = y[0] & 1
    pats, rhos = [], []
    for s in range(3):
        pat, rho = 0, 0
        for tt in range(8):
            v = y[8 * s + tt]
            c = ((v - p) >> 1) & 1
            o = p + 2 * c
            r = _inv.rank.get((o, v))
            if r is None:
                return None
            pat |= c << tt
            rho |= r << (4 * tt)
        pats.append(pat)
        rhos.append(rho)
    path = _inv.path.get(tuple(pats))
    if path is None:
        return None
    s8, b1, b2, b3 = path
    r = int(tables.cls_of(rhos[0]))
    i1 = _inv.half[r].get(rhos[0])
    i2 = _inv.mid.get(rhos[1])
    r3 = int(tables.cls_of(rhos[2]))
    i3 = _inv.half[r3].get(rhos[2])
    if i1 is None or i2 is None or i3 is None:
        return None
    delta = int(tables.cls_of(rhos[1]))
    if r3 != p ^ r ^ delta:
        return None
    return int(pack_fields(s8=s8, p=p, r=r, b1=b1, b2=b2, b3=b3, g=g,
                           i1=i1, i2=i2, i3=i3))
