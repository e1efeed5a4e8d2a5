"""Extended binary Golay code G24 and the octad trio (oracle, test-only).

Paper passages followed:
* Sec. 3.1, Eq. 1: the lattice is built from a codeword c of the binary Golay
  code of length 24 (2**12 codewords among the 2**24 bit patterns).
* Sec. 3.2: three octads (weight-8 codewords) that share no position cover
  the 24 coordinates; the coordinates are read octad by octad, giving three
  sections of eight.

Readings (the paper names neither the construction nor the octads):
* G24 is the cyclic [23,12] code with generator polynomial
  g(x) = 1 + x^2 + x^4 + x^5 + x^6 + x^10 + x^11, extended by an overall
  parity bit at coordinate 23.  A codeword is an int whose bit i is
  coordinate i.
* Octad 1 is the octad whose sorted support is lexicographically smallest;
  octad 2 is the lexicographically smallest octad disjoint from it; octad 3
  is the complement of their union.  Block coordinate j = 8*s + t is the t-th
  smallest original coordinate of octad s+1.

Pins (tests): the weight enumerator 1/759/2576/759/1 of the extended Golay
code; the trio is three disjoint octads covering all 24 coordinates;
membership by polynomial division agrees with the enumerated set.
"""

from functools import lru_cache

GEN_POLY = (1 << 0) | (1 << 2) | (1 << 4) | (1 << 5) | (1 << 6) | (1 << 10) | (1 << 11)


def _parity(v: int) -> int:
    return bin(v).count("1") & 1


@lru_cache(maxsize=None)
def codewords() -> tuple:
    """All 4096 codewords of G24 as 24-bit ints, sorted ascending."""
    rows = [GEN_POLY << i for i in range(12)]          # x^i g(x), degree <= 22
    words = set()
    for m in range(1 << 12):
        c = 0
        for i in range(12):
            if (m >> i) & 1:
                c ^= rows[i]
        c |= _parity(c) << 23                            # overall parity bit
        words.add(c)
    return tuple(sorted(words))


def poly_mod(a: int, g: int = GEN_POLY) -> int:
    """Remainder of the GF(2) polynomial a modulo g."""
    dg = g.bit_length() - 1
    while a and a.bit_length() - 1 >= dg:
        a ^= g << (a.bit_length() - 1 - dg)
    return a


def is_codeword(c: int) -> bool:
    """Membership by definition of the extended cyclic code: the first 23
    coordinates form a multiple of g(x) and the overall weight is even.
    Written independently of ``codewords`` so each can check the other."""
    if c >> 24:
        return False
    return poly_mod(c & ((1 << 23) - 1)) == 0 and _parity(c) == 0


def support(c: int) -> tuple:
    return tuple(i for i in range(24) if (c >> i) & 1)


@lru_cache(maxsize=None)
def trio() -> tuple:
    """The three octads (as sorted supports) fixed by the reading above."""
    octads = sorted(support(c) for c in codewords() if bin(c).count("1") == 8)
    o1 = octads[0]
    m1 = sum(1 << i for i in o1)
    o2 = next(o for o in octads if not (sum(1 << i for i in o) & m1))
    rest = tuple(i for i in range(24) if i not in o1 and i not in o2)
    return (o1, o2, rest)


@lru_cache(maxsize=None)
def block_order() -> tuple:
    """perm[j] = original Golay coordinate of block coordinate j = 8*s + t."""
    o = trio()
    return tuple(o[s][t] for s in range(3) for t in range(8))


def to_sections(c: int) -> tuple:
    """Split a codeword into its three pattern bytes (Sec. 3.3): bit t of
    byte s is the codeword bit at block coordinate 8*s + t."""
    perm = block_order()
    out = []
    for s in range(3):
        b = 0
        for t in range(8):
            b |= ((c >> perm[8 * s + t]) & 1) << t
        out.append(b)
    return tuple(out)


def from_sections(p1: int, p2: int, p3: int) -> int:
    """Inverse of ``to_sections``."""
    perm = block_order()
    c = 0
    for s, b in enumerate((p1, p2, p3)):
        for t in range(8):
            c |= ((b >> t) & 1) << perm[8 * s + t]
    return c
