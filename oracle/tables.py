"""Decoder tables of the Tetra codebook (oracle, test-only).

Paper passages followed:
* Sec. 3.2 and Fig. 2: in octad order the Golay code is a trellis with 64
  states at each cut, 2 prefixes x 16 branches x 2 suffixes = 4096 paths,
  one per codeword.  The state s8 after section 1 is stored in the word;
  s16 is returned by the branch read.
* Fig. 4: prefixes[2*s8 + b1], branches[16*s8 + b2] -> (pattern byte, s16),
  suffixes[2*s16 + b3]; 2,304 B of trellis tables.
* Sec. 3.3: coordinate j of a section lies in o_j + 4Z with o_j = p + 2*c_j;
  its rank is its position in that list counted outward from zero (o=0:
  0,+4,-4,+8,...; o=1: +1,-3,+5,...).  cost(rho) = sum_j (2*rho_j+1)^2;
  cls(rho) = #{j : rho_j in {1,2,5,6}} mod 2.  The table holds the 2,048
  cheapest rank vectors of class 0, then the 2,048 cheapest of class 1, four
  bits per rank in one 32-bit row.  The middle section reads the same rows
  through its own list of the 2,048 cheapest overall, class 0 first
  (N0 = 1240 rows), then class 1 (808 rows).
* Sec. 3.4: 32 floats hold 1/sqrt(16*m), the m = 0 entry is 0.
* Eq. 2: one gain bit g selects gain[g].

Readings (the paper is silent; each is listed with its pins in the design
notes):
* Trellis numbering: s8 numbers the 64 complementary pairs {P, P^0xFF} of
  section-1 pattern bytes in ascending order of min(P, P^0xFF);
  prefixes[2*s8 + b1] is the smaller byte when b1 = 0, its complement when
  b1 = 1.  s16 numbers the section-3 pairs the same way, suffixes likewise.
  branches[16*s8 + b2] is the b2-th of the 16 continuations (P2, s16) of s8
  in ascending order of P2, stored as P2 | s16 << 8.
* Value list for o = 2: at equal magnitude the positive value comes first
  (2, -2, 6, -6, ...), as in the o = 0 example.  Parity unpinned: the other
  order gives lattice points too.
* Ties of cost at the three 2,048 cuts are broken by the packed 32-bit row
  value, ascending; nibble j of a row is the rank of section coordinate j.
  N0 = 1240, m <= 26 and max|y| = 10 are reproduced under it; which tied
  vectors are kept is parity unpinned.
* gain = (4.3, 5.4) as float32: the paper defers the gain values to the
  encoder.  Parity unpinned (any pair can be loaded through the table blob).
"""

from functools import lru_cache

import numpy as np

from . import golay

N_ROWS_HALF = 2048
GAIN = np.array([4.3, 5.4], dtype=np.float32)


# --------------------------------------------------------------------------
# Trellis (Sec. 3.2, Fig. 2, Fig. 4)
# --------------------------------------------------------------------------

def _pair_rep(b: int) -> int:
    return min(b, b ^ 0xFF)


@lru_cache(maxsize=None)
def trellis() -> dict:
    secs = [golay.to_sections(c) for c in golay.codewords()]
    reps1 = sorted({_pair_rep(s[0]) for s in secs})
    reps3 = sorted({_pair_rep(s[2]) for s in secs})
    s8_of = {r: i for i, r in enumerate(reps1)}
    s16_of = {r: i for i, r in enumerate(reps3)}

    prefixes = np.zeros(2 * len(reps1), dtype=np.uint8)
    for s8, rep in enumerate(reps1):
        prefixes[2 * s8] = rep
        prefixes[2 * s8 + 1] = rep ^ 0xFF
    suffixes = np.zeros(2 * len(reps3), dtype=np.uint8)
    for s16, rep in enumerate(reps3):
        suffixes[2 * s16] = rep
        suffixes[2 * s16 + 1] = rep ^ 0xFF

    cont = {}          # s8 -> set of (P2, s16), gathered over both prefixes
    for p1, p2, p3 in secs:
        cont.setdefault(s8_of[_pair_rep(p1)], set()).add((p2, s16_of[_pair_rep(p3)]))
    branches = np.zeros(16 * len(reps1), dtype=np.uint16)
    nbranch = {}
    for s8, edges in cont.items():
        edges = sorted(edges)
        nbranch[s8] = len(edges)
        for b2, (p2, s16) in enumerate(edges[:16]):
            branches[16 * s8 + b2] = p2 | (s16 << 8)
    return {
        "prefixes": prefixes, "branches": branches, "suffixes": suffixes,
        "n_s8": len(reps1), "n_s16": len(reps3), "branches_per_state": nbranch,
    }


def walk(s8, b1, b2, b3):
    """Trellis walk of Fig. 4: returns the three pattern bytes and s16."""
    t = trellis()
    p1 = t["prefixes"][2 * s8 + b1]
    br = t["branches"][16 * s8 + b2]
    p2 = br & 0xFF
    s16 = br >> 8
    p3 = t["suffixes"][2 * s16 + b3]
    return p1, p2, p3, s16


# --------------------------------------------------------------------------
# Coordinate value lists (Sec. 3.3)
# --------------------------------------------------------------------------

@lru_cache(maxsize=None)
def value_lists() -> np.ndarray:
    """V[o, rho]: the rho-th value of o + 4Z counted outward from zero,
    positive first at equal magnitude.  Shape (4, 8), int."""
    V = np.zeros((4, 8), dtype=np.int64)
    for o in range(4):
        cands = [v for v in range(-64, 65) if (v - o) % 4 == 0]
        cands.sort(key=lambda v: (abs(v), v < 0))
        V[o] = cands[:8]
    return V


# --------------------------------------------------------------------------
# Rank table (Sec. 3.3, Fig. 4)
# --------------------------------------------------------------------------

def cost_of(packed: np.ndarray) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.int64)
    out = np.zeros(packed.shape, dtype=np.int64)
    for j in range(8):
        d = (packed >> (4 * j)) & 0xF
        out += (2 * d + 1) ** 2
    return out


def cls_of(packed: np.ndarray) -> np.ndarray:
    packed = np.asarray(packed, dtype=np.int64)
    out = np.zeros(packed.shape, dtype=np.int64)
    for j in range(8):
        d = (packed >> (4 * j)) & 0xF
        out += np.isin(d, (1, 2, 5, 6))
    return out & 1


@lru_cache(maxsize=None)
def _all_rank_vectors():
    """Every rho in {0..7}^8 as (packed u32, cost, cls)."""
    idx = np.arange(8 ** 8, dtype=np.int64)
    packed = np.zeros_like(idx)
    cost = np.zeros_like(idx)
    odd = np.zeros_like(idx)
    for j in range(8):
        d = (idx >> (3 * j)) & 7
        packed |= d << (4 * j)
        cost += (2 * d + 1) ** 2
        odd += (d == 1) | (d == 2) | (d == 5) | (d == 6)
    return packed, cost, odd & 1


def _cheapest(packed, cost, n):
    key = (cost << 32) | packed          # (cost, packed) ascending, all distinct
    part = np.partition(key, n - 1)[:n]
    part.sort()
    return (part & 0xFFFFFFFF).astype(np.uint32)


@lru_cache(maxsize=None)
def rank_table() -> dict:
    packed, cost, cls = _all_rank_vectors()
    half0 = _cheapest(packed[cls == 0], cost[cls == 0], N_ROWS_HALF)
    half1 = _cheapest(packed[cls == 1], cost[cls == 1], N_ROWS_HALF)
    overall = _cheapest(packed, cost, N_ROWS_HALF)
    ocls = cls_of(overall)
    middle = np.concatenate([overall[ocls == 0], overall[ocls == 1]])
    return {
        "rows": np.concatenate([half0, half1]).astype(np.uint32),
        "middle": middle.astype(np.uint32),
        "n0": int((ocls == 0).sum()),
    }


def mix(i2):
    """Physical row of middle-list entry i2, given that the middle list is
    the first n0 class-0 rows followed by the first 2048-n0 class-1 rows."""
    n0 = rank_table()["n0"]
    i2 = np.asarray(i2, dtype=np.int64)
    return np.where(i2 < n0, i2, N_ROWS_HALF + (i2 - n0))


# --------------------------------------------------------------------------
# Norm and gain tables (Sec. 3.4, Eq. 2)
# --------------------------------------------------------------------------

@lru_cache(maxsize=None)
def invnorm() -> np.ndarray:
    t = np.zeros(32, dtype=np.float32)
    for m in range(1, 32):
        t[m] = np.float32(1.0 / np.sqrt(16.0 * m))   # double, then RNE to f32
    return t


def gain() -> np.ndarray:
    return GAIN.copy()


# --------------------------------------------------------------------------
# Canonical table blob
# --------------------------------------------------------------------------

BLOB_BYTES = 16384 + 2048 + 128 + 128 + 128 + 8


def table_blob() -> bytes:
    """rows u32[4096] | branches u16[1024] | prefixes u8[128] |
    suffixes u8[128] | invnorm f32[32] | gain f32[2], little-endian."""
    t = trellis()
    parts = [
        rank_table()["rows"].astype("<u4").tobytes(),
        t["branches"].astype("<u2").tobytes(),
        t["prefixes"].astype("u1").tobytes(),
        t["suffixes"].astype("u1").tobytes(),
        invnorm().astype("<f4").tobytes(),
        gain().astype("<f4").tobytes(),
    ]
    blob = b"".join(parts)
    assert len(blob) == BLOB_BYTES
    return blob
