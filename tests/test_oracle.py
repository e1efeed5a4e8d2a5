"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the passage or the closed form it checks.  None of them
re-types the oracle's own formula: they use textbook facts (the Golay weight
enumerator, the Leech-lattice congruences), brute force over small sets,
printed constants (tests/golden/paper_constants.json), inverse maps and
invariants of the reconstruction.
"""

import json
import os
from collections import Counter

import numpy as np
import pytest

from oracle import codec, gemv, golay, int4, tables

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def paper():
    with open(os.path.join(GOLDEN, "paper_constants.json")) as f:
        return {k: v["value"] for k, v in json.load(f).items() if not k.startswith("_")}


# ---------------------------------------------------------------- Golay code

def test_golay_weight_enumerator(paper):
    cw = golay.codewords()
    assert len(cw) == paper["n_codewords"]
    hist = Counter(bin(c).count("1") for c in cw)
    assert {str(k): v for k, v in hist.items()} == paper["golay_weight_enumerator"]


def test_golay_membership_two_ways():
    cw = set(golay.codewords())
    assert all(golay.is_codeword(c) for c in cw)
    rng = np.random.default_rng(11)
    for v in rng.integers(0, 1 << 24, size=4000):
        assert golay.is_codeword(int(v)) == (int(v) in cw)
    # closure: sum of two codewords is a codeword (linearity)
    cwl = list(cw)
    for _ in range(500):
        a, b = rng.choice(len(cwl), 2)
        assert (cwl[a] ^ cwl[b]) in cw


def test_trio_is_three_disjoint_octads():
    o = golay.trio()
    masks = [sum(1 << i for i in s) for s in o]
    assert all(len(s) == 8 for s in o)
    assert masks[0] & masks[1] == 0 and masks[0] & masks[2] == 0 and masks[1] & masks[2] == 0
    assert masks[0] | masks[1] | masks[2] == (1 << 24) - 1
    assert all(golay.is_codeword(m) for m in masks)
    assert sorted(golay.block_order()) == list(range(24))


def test_section_projections(paper):
    secs = [golay.to_sections(c) for c in golay.codewords()]
    even = {b for b in range(256) if bin(b).count("1") % 2 == 0}
    for s in range(3):
        proj = {t[s] for t in secs}
        assert proj == even and len(proj) == paper["pattern_bytes_per_section"]
        # sub-code supported on section s alone: only 0x00 and 0xFF
        sub = {t[s] for t in secs if all(t[u] == 0 for u in range(3) if u != s)}
        assert sub == {0x00, 0xFF}


# ------------------------------------------------------------------ trellis

def test_trellis_counts(paper):
    t = tables.trellis()
    assert t["n_s8"] == paper["trellis_states_per_cut"] == t["n_s16"]
    assert set(t["branches_per_state"].values()) == {paper["trellis_fan"][1]}
    assert len(t["prefixes"]) == 2 * 64 and len(t["suffixes"]) == 2 * 64
    assert len(t["branches"]) == 16 * 64
    for s8 in range(64):
        br = t["branches"][16 * s8:16 * s8 + 16]
        p2 = br & 0xFF
        assert len(set(p2.tolist())) == 16
        assert len(set((br >> 8).tolist())) == 8          # 2 parallel branches
    # bytes of the trellis tables
    assert (t["prefixes"].nbytes + t["suffixes"].nbytes + t["branches"].nbytes
            == paper["trellis_table_bytes"])


def test_trellis_paths_are_a_bijection_onto_the_code(paper):
    cw = set(golay.codewords())
    seen = set()
    s16_of = {}
    for s8 in range(64):
        for b1 in range(2):
            for b2 in range(16):
                for b3 in range(2):
                    p1, p2, p3, s16 = tables.walk(s8, b1, b2, b3)
                    c = golay.from_sections(int(p1), int(p2), int(p3))
                    assert c in cw
                    seen.add(c)
                    # s16 is a function of (P1, P2)
                    assert s16_of.setdefault((int(p1), int(p2)), int(s16)) == int(s16)
    assert len(seen) == paper["n_codewords"] == 64 * 2 * 16 * 2


# ------------------------------------------------------------- value lists

def test_value_lists(paper):
    V = tables.value_lists()
    assert V[0, :4].tolist() == paper["value_list_o0_prefix"]
    assert V[1, :3].tolist() == paper["value_list_o1_prefix"]
    for o in range(4):
        assert np.all((V[o] - o) % 4 == 0)
        mags = np.abs(V[o])
        assert np.all(np.diff(mags) >= 0)                  # outward from zero
        assert len(set(V[o].tolist())) == 8
        # the 8 entries are exactly the 8 smallest-magnitude members of o+4Z
        allm = sorted(abs(v) for v in range(-40, 41) if (v - o) % 4 == 0)[:8]
        assert sorted(mags.tolist()) == allm


# --------------------------------------------------------------- rank table

def test_rank_table_shape_and_order(paper):
    rt = tables.rank_table()
    rows = rt["rows"]
    assert rows.dtype == np.uint32 and rows.nbytes == paper["rank_table_bytes"]
    assert len(rows) == paper["rank_rows"]
    cls = tables.cls_of(rows)
    assert np.all(cls[:2048] == 0) and np.all(cls[2048:] == 1)
    for half in (rows[:2048], rows[2048:]):
        c = tables.cost_of(half)
        assert np.all(np.diff(c) >= 0)
        assert len(set(half.tolist())) == 2048
    # closed form: (2r+1)^2 = 1 mod 8 and = 9 mod 16 exactly when r is in
    # {1,2,5,6}; so cost = 8 + 8*cls (mod 16)
    c = tables.cost_of(rows)
    assert np.all(c[:2048] % 16 == 8) and np.all(c[2048:] % 16 == 0)
    # no rank above 4 survives the cut (cost <= 96 < 81 + 7 + 9 + ...)
    nib = (rows[:, None].astype(np.int64) >> (4 * np.arange(8))) & 0xF
    assert nib.max() == 4


def test_rank_table_is_the_cheapest_by_brute_force():
    """Independent of the oracle's enumeration: every vector of {0..7}^8 that
    is strictly cheaper than a half's last row is in that half."""
    rt = tables.rank_table()
    rows = rt["rows"]
    # only ranks <= 4 can reach cost <= 96; enumerate {0..4}^8 directly
    import itertools
    for cls_target, half in ((0, rows[:2048]), (1, rows[2048:])):
        last = int(tables.cost_of(half[-1:])[0])
        hs = set(half.tolist())
        count_below = 0
        for r in itertools.product(range(5), repeat=8):
            cost = sum((2 * v + 1) ** 2 for v in r)
            cl = sum(v in (1, 2, 5, 6) for v in r) % 2
            if cl == cls_target and cost < last:
                count_below += 1
                assert sum(v << (4 * j) for j, v in enumerate(r)) in hs
        assert count_below < 2048


def test_middle_list(paper):
    rt = tables.rank_table()
    assert rt["n0"] == paper["n0_middle_class0"]
    assert 2048 - rt["n0"] == paper["n1_middle_class1"]
    mid = rt["middle"]
    # class 0 first, then class 1; the middle list is read through mix()
    assert np.all(tables.cls_of(mid[:1240]) == 0) and np.all(tables.cls_of(mid[1240:]) == 1)
    assert np.array_equal(rt["rows"][tables.mix(np.arange(2048))], mid)
    # the 2048 cheapest overall: nothing outside is strictly cheaper than the
    # dearest member
    dear = tables.cost_of(mid).max()
    rows = rt["rows"]
    outside = np.setdiff1d(rows, mid)
    assert tables.cost_of(outside).min() >= dear


def test_class_gives_k_parity_for_every_pattern():
    """Sec. 3.3: cls(rho) equals the parity of sum_j k_j for every p and every
    admissible pattern byte (brute force over 2 x 128 x 4096)."""
    V = tables.value_lists()
    rows = tables.rank_table()["rows"].astype(np.int64)
    nib = (rows[:, None] >> (4 * np.arange(8))) & 0xF            # [4096, 8]
    cls = tables.cls_of(rows)
    for p in (0, 1):
        for pat in range(256):
            if bin(pat).count("1") % 2:
                continue
            c = (pat >> np.arange(8)) & 1
            o = p + 2 * c
            vals = V[o[None, :], nib]                              # [4096, 8]
            k = (vals - o[None, :]) // 4
            assert np.all((k.sum(axis=1) & 1) == cls)


def test_table_blob_size(paper):
    assert tables.BLOB_BYTES - 8 == paper["total_table_bytes"]
    assert len(tables.table_blob()) == tables.BLOB_BYTES


# ----------------------------------------------------------- norms and gain

def test_invnorm_table(paper):
    t = tables.invnorm()
    assert t.dtype == np.float32 and len(t) == paper["norm_table_floats"]
    assert t[0] == 0.0
    m = np.arange(1, 32)
    # within half an ulp of the exact value (RNE of the double result)
    exact = 1.0 / np.sqrt(16.0 * m)
    ulp = np.spacing(t[1:].astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(t[1:].astype(np.float64) - exact) <= 0.5 * ulp)


# ---------------------------------------------------------------- decoding

def _section_max_sq():
    """max over kept rows of the squared norm of one section, for each p,
    pattern byte and row list (half 0, half 1, middle class 0/1)."""
    V = tables.value_lists()
    rt = tables.rank_table()
    rows = rt["rows"].astype(np.int64)
    lists = {("h", 0): rows[:2048], ("h", 1): rows[2048:],
             ("m", 0): rows[:1240], ("m", 1): rows[2048:2048 + 808]}
    out, vmax = {}, 0
    for key, lst in lists.items():
        nib = (lst[:, None] >> (4 * np.arange(8))) & 0xF
        for p in (0, 1):
            for pat in range(256):
                if bin(pat).count("1") % 2:
                    continue
                c = (pat >> np.arange(8)) & 1
                vals = V[(p + 2 * c)[None, :], nib]
                out[(p, pat) + key] = int((vals ** 2).sum(axis=1).max())
                vmax = max(vmax, int(np.abs(vals).max()))
    return out, vmax


def test_shell_and_coordinate_bounds(paper):
    """Sec. 3.4: every codeword with both parities and every allowed row in
    each section gives m <= 26 and max|y_j| = 10 (exact, since the sections
    are independent once the path, p, r and delta are fixed)."""
    smax, vmax = _section_max_sq()
    best = 0
    for c in golay.codewords():
        p1, p2, p3 = golay.to_sections(c)
        for p in (0, 1):
            for r in (0, 1):
                for d in (0, 1):
                    tot = (smax[(p, p1, "h", r)] + smax[(p, p2, "m", d)]
                           + smax[(p, p3, "h", p ^ r ^ d)])
                    best = max(best, tot)
    assert best % 16 == 0
    assert best // 16 == paper["max_shell_m"]
    assert vmax == paper["max_abs_coordinate"]


@pytest.fixture(scope="module")
def random_words():
    rng = np.random.default_rng(20260901)
    return rng.integers(0, 1 << 48, size=300_000, dtype=np.uint64)


def test_random_words_decode_into_leech(random_words):
    y, m, s = codec.decode(random_words)
    y = y.astype(np.int64)
    assert codec.in_leech(y).all()
    p = y[:, 0] & 1
    # textbook congruences of the integral Leech lattice (norm 16m, m != 1)
    assert np.all(y.sum(axis=1) % 8 == (4 * p) % 8)
    sq = (y * y).sum(axis=1)
    assert np.all(sq % 16 == 0)
    assert np.all((sq == 0) | (sq >= 32))
    assert m.max() <= 26 and np.abs(y).max() <= 10


def test_membership_rejects_non_lattice_points(random_words):
    y, _, _ = codec.decode(random_words[:2000])
    y = y.astype(np.int64)
    bad = y.copy()
    bad[:, 3] += 2                      # breaks the Golay word or the k-parity
    assert not codec.in_leech(bad).any()
    bad = y.copy()
    bad[:, 5] += 4                      # same pattern, k-parity flipped
    bad[:, 7] += 0
    assert not codec.in_leech(bad).any()
    bad = y.copy()
    bad[:, 0] += 1                      # mixed coordinate parity
    assert not codec.in_leech(bad).any()


def test_origin_word():
    y, m, s = codec.decode(np.zeros(1, dtype=np.uint64))
    assert not y.any() and m[0] == 0 and s[0] == 0.0


def test_every_word_is_legal_and_decode_is_injective(random_words):
    y, _, s = codec.decode(random_words[:100_000])
    g = codec.fields(random_words[:100_000])["g"]
    keys = {(bytes(yy.tobytes()), int(gg)) for yy, gg in zip(y, g)}
    uniq = len(set(random_words[:100_000].tolist()))
    assert len(keys) == uniq


def test_encode_decode_round_trip(random_words):
    w = random_words[:3000]
    y, _, _ = codec.decode(w)
    g = codec.fields(w)["g"]
    for wi, yi, gi in zip(w, y, g):
        assert codec.encode(yi, int(gi)) == int(wi)


def test_encode_rejects_points_outside_the_codebook():
    # (12, 0, ..., 0) + lattice structure: rank 5 of o=0 is never kept
    y = np.zeros(24, dtype=np.int64)
    y[0], y[1] = 12, 4                  # a lattice point? not needed: rank 5 missing
    assert codec.encode(y, 0) is None


# ----------------------------------------------- planted mistakes (CPU only)

def _caught(words):
    """True when the planted mistake shows: the decoder's own norm check
    fires or some decoded point leaves the lattice."""
    try:
        y, _, _ = codec.decode(words)
    except AssertionError:
        return True
    return not codec.in_leech(y.astype(np.int64)).all()


def test_planted_mistake_dropping_delta_is_caught(monkeypatch, random_words):
    """Dropping delta from Eq. 3 breaks the k-parity of some points."""
    monkeypatch.setattr(codec.tables, "cls_of", lambda v: np.zeros(np.shape(v), np.int64))
    assert _caught(random_words[:20000])


def test_planted_mistake_wrong_value_list_is_caught(monkeypatch, random_words):
    V = tables.value_lists().copy()
    V[1, [0, 1]] = V[1, [1, 0]]          # o = 1 list read as -3, +1, +5, ...
    monkeypatch.setattr(codec.tables, "value_lists", lambda: V)
    assert _caught(random_words[:20000])


def test_planted_mistake_wrong_state_link_is_caught(monkeypatch, random_words):
    """A branch entry that names the wrong s16 sends the suffix read to the
    wrong pair of pattern bytes: the words leave the Golay code."""
    orig = tables.trellis()
    t = dict(orig)
    br = orig["branches"].astype(np.int64)
    t["branches"] = ((br & 0xFF) | ((((br >> 8) + 1) % 64) << 8)).astype(np.uint16)
    monkeypatch.setattr(codec.tables, "trellis", lambda: t)
    assert _caught(random_words[:20000])


def test_planted_mistake_transposed_middle_byte_is_caught(monkeypatch, random_words):
    """Reading the middle pattern byte with its bit order reversed."""
    orig = tables.trellis()
    t = dict(orig)
    br = orig["branches"].astype(np.int64)
    rev = np.array([int(f"{b:08b}"[::-1], 2) for b in range(256)])
    t["branches"] = (rev[br & 0xFF] | (br & 0xFF00)).astype(np.uint16)
    monkeypatch.setattr(codec.tables, "trellis", lambda: t)
    assert _caught(random_words[:20000])


# --------------------------------------------------------------------- GEMV

def _matrix(M, K, seed):
    rng = np.random.default_rng(seed)
    nblk, T = gemv.split_k(K)
    words = rng.integers(0, 1 << 48, size=(M, nblk), dtype=np.uint64)
    sig = (rng.uniform(0.5, 2.0, M) * 1e-2).astype(np.float16)
    tail = (rng.standard_normal((M, T)) * sig[:, None].astype(np.float32)).astype(np.float16)
    return words, sig, tail


def test_dequant_block_norm_is_gain_times_sigma():
    """Eq. 2: the reconstructed block has norm gain[g] * sigma_row."""
    words, sig, tail = _matrix(64, 24 * 20 + 8, 3)
    w = gemv.dequant(words, sig, tail)[:, :480].reshape(64, 20, 24).astype(np.float64)
    g = codec.fields(words)["g"]
    _, m, _ = codec.decode(words)
    norms = np.sqrt((w * w).sum(axis=2))
    want = tables.gain()[g].astype(np.float64) * sig.astype(np.float64)[:, None]
    nz = m > 0
    assert np.allclose(norms[nz], want[nz], rtol=2e-6)
    assert np.all(norms[~nz] == 0)


def test_gemv_unit_vectors_and_tail():
    M, K = 16, 24 * 5 + 16
    words, sig, tail = _matrix(M, K, 5)
    W = gemv.dequant(words, sig, tail).astype(np.float64)
    for k in (0, 7, 23, 24, 119, 120, 135):
        x = np.zeros((1, K), np.float16)
        x[0, k] = 1.0
        y, _ = gemv.gemv_f64(words, sig, tail, x)
        assert np.allclose(y[0], W[:, k], rtol=1e-6, atol=0)
    # all-zero words: only the tail term survives
    x = np.random.default_rng(1).standard_normal((2, K)).astype(np.float16)
    y, _ = gemv.gemv_f64(np.zeros_like(words), sig, tail, x)
    want = x[:, 120:].astype(np.float64) @ tail.astype(np.float64).T
    assert np.allclose(y, want, rtol=1e-12, atol=1e-12)


def test_gemv_rows_subset_matches_full():
    words, sig, tail = _matrix(40, 24 * 9 + 8, 9)
    x = np.random.default_rng(2).standard_normal((3, 24 * 9 + 8)).astype(np.float16)
    y, n = gemv.gemv_f64(words, sig, tail, x)
    ys, ns = gemv.gemv_f64(words, sig, tail, x, rows=[3, 17, 39])
    assert np.allclose(ys, y[:, [3, 17, 39]], rtol=1e-13) and np.allclose(ns, n[:, [3, 17, 39]])


# --------------------------------------------------------------------- int4

def test_int4_affine_pins():
    rng = np.random.default_rng(4)
    M, K = 3, 256
    so = rng.uniform(0.1, 1.0, (M, K // 128, 2)).astype(np.float16)
    q = np.zeros((M, K // 2), np.uint8)
    w = int4.dequant_affine(q, so, 128)
    assert np.array_equal(w[:, 0], so[:, 0, 1].astype(np.float32))
    q[1, 70] = 0x30                       # element 141 (odd -> high nibble) = 3
    w2 = int4.dequant_affine(q, so, 128)
    diff = np.argwhere(w2 != w)
    assert diff.tolist() == [[1, 141]]
    assert np.isclose(w2[1, 141] - w[1, 141], 3 * float(so[1, 1, 0]), rtol=1e-3)


def test_head4_groups_of_64_pins():
    """The output head of Sec. 4.4 uses groups of 64: constant nibbles reduce
    the product to per-group sums of x, and a one-hot x on either side of a
    group boundary picks the weight of its own group."""
    rng = np.random.default_rng(9)
    rows, dim = 4, 256
    so = rng.uniform(0.1, 1.0, (rows, dim // 64, 2)).astype(np.float16)
    x = rng.standard_normal((1, dim)).astype(np.float16)
    c = 11
    q = np.full((rows, dim // 2), c | c << 4, np.uint8)
    y, _ = int4.int4_gemv_f64(q, so, x, group=64)
    sx = x.astype(np.float64).reshape(dim // 64, 64).sum(axis=1)          # per-group sums
    s64 = so.astype(np.float32).astype(np.float64)
    want = ((s64[..., 0] * c + s64[..., 1]) * sx).sum(axis=1)
    assert np.allclose(y[0], want, rtol=1e-6)
    q = rng.integers(0, 256, size=(rows, dim // 2), dtype=np.uint8)
    for k in (63, 64, 127, 128):
        e = np.zeros((1, dim), np.float16)
        e[0, k] = 1.0
        y, _ = int4.int4_gemv_f64(q, so, e, group=64)
        nib = (q[:, k // 2] >> (4 * (k % 2))) & 0xF
        want = (so[:, k // 64, 0].astype(np.float32) * nib).astype(np.float32) + so[:, k // 64, 1].astype(np.float32)
        assert np.array_equal(y[0].astype(np.float32), want.astype(np.float32)), k


# ----------------------------------------------------------------- rotation

from oracle import rotation  # noqa: E402


@pytest.mark.parametrize("n", [1, 2, 4, 8, 16, 64])
def test_hadamard_is_sylvester_and_orthogonal(n):
    """H_n: entries +-1, H H^T = n I, and the Sylvester recursion."""
    from scipy.linalg import hadamard
    h = hadamard(n)
    assert set(np.unique(h).tolist()) <= {-1, 1}
    assert np.array_equal(h @ h.T, n * np.eye(n, dtype=h.dtype))
    if n > 1:
        q = hadamard(n // 2)
        assert np.array_equal(h, np.block([[q, q], [q, -q]]))
    # entry (i, m) is (-1)^popcount(i & m) (the Walsh-Hadamard form)
    for i in range(n):
        for m in range(n):
            assert h[i, m] == (-1) ** bin(i & m).count("1")


def test_rotation_pins():
    """Norm preservation per block, involution of the unsigned transform,
    the sign convention, and a one-hot column."""
    rng = np.random.default_rng(21)
    n, K = 64, 256
    x = rng.standard_normal((2, K)).astype(np.float16)
    bits = rng.integers(0, 256, K // 8, dtype=np.uint8)
    y = rotation.rotate_f64(x, bits, n)
    xb = x.astype(np.float64).reshape(2, K // n, n)
    assert np.allclose(np.linalg.norm(y.reshape(2, K // n, n), axis=-1), np.linalg.norm(xb, axis=-1), rtol=1e-12)
    zero = np.zeros(K // 8, np.uint8)
    twice = rotation.rotate_f64(rotation.rotate_f64(x, zero, n).astype(np.float64), zero, n)
    assert np.allclose(twice, x.astype(np.float64), atol=1e-3)      # the inner result was rounded to fp16
    # sign bit k negates element k before the transform
    one = np.zeros((1, K), np.float16)
    one[0, 5] = 1.0
    b5 = np.zeros(K // 8, np.uint8)
    b5[0] = 1 << 5
    assert np.allclose(rotation.rotate_f64(one, b5, n), -rotation.rotate_f64(one, zero, n))
    full = rotation.rotate_f64(one, zero, n)[0]
    want = np.array([(-1) ** bin(i & 5).count("1") for i in range(n)]) / np.sqrt(n)
    assert np.allclose(full[:n], want, rtol=1e-15)
    assert not full[n:].any()                                       # blocks do not mix


# ----------------------------------------------------------------- encoder

from oracle import encoder  # noqa: E402


def _block_of(word):
    """A block pointing exactly at the decoded point of `word`, with norm
    gain[g] (sigma = 1), and that point's radius."""
    y = codec.decode(np.array([word], dtype=np.uint64))[0][0].astype(np.int64)
    g = int(codec.fields(np.array([word], dtype=np.uint64))["g"][0])
    ny = float(np.sqrt((y * y).sum()))
    return (y * (float(tables.gain()[g]) / ny)).astype(np.float32), ny


def test_encoder_returns_the_word_at_its_own_radius():
    """At a trial radius equal to ||y|| the targets are y itself (on the
    2^-16 grid), every other kept point scores strictly lower, and the gain
    nearest to ||w|| = gain[g] is g: the search must give back the word,
    every field of every section included (both row halves, the middle list
    on both sides of N0, all trellis edges)."""
    rng = np.random.default_rng(2024)
    words = [int(v) for v in rng.integers(0, 1 << 48, size=6, dtype=np.uint64)]
    # a word with delta = 1 (middle index past N0) and one with delta = 0
    f = codec.fields(np.array(words, dtype=np.uint64))
    assert (f["i2"] >= tables.rank_table()["n0"]).any() and (f["i2"] < tables.rank_table()["n0"]).any()
    for wd in words:
        w, ny = _block_of(wd)
        assert encoder.encode_block(w, 1.0, [ny]) == wd
        # a second, worse radius does not displace the exact direction
        assert encoder.encode_block(w, 1.0, [ny, 0.5 * ny]) == wd


def test_encoder_search_beats_every_single_field_change():
    """The search result scores at least as high as every word that differs
    from it in one field: each row index over its whole list (a brute force
    of each section given the others), each trellis edge and state, p and
    r; and at least as high as 20,000 random words."""
    rng = np.random.default_rng(99)
    w = rng.standard_normal(24).astype(np.float32)
    T = encoder.targets(w, 14.0)
    best, f, y = encoder.nearest_point(T)
    assert encoder.score(T, y) == best
    word = int(codec.pack_fields(g=0, **f))
    assert np.array_equal(codec.decode(np.array([word], dtype=np.uint64))[0][0], y)
    sweeps = {"i1": 2048, "i2": 2048, "i3": 2048, "s8": 64, "b1": 2, "b2": 16, "b3": 2, "p": 2, "r": 2}
    for name, n in sweeps.items():
        ff = dict(f, g=0)
        ff[name] = np.arange(n)
        ff = {k: np.broadcast_to(np.asarray(v), (n,)) for k, v in ff.items()}
        ys = codec.decode(codec.pack_fields(**ff))[0].astype(np.int64)
        scores = (2 * T[None] * ys - encoder.SCALE * ys * ys).sum(axis=1)
        assert scores.max() <= best, name
        assert scores[f[name]] == best, name
    ys = codec.decode(rng.integers(0, 1 << 48, size=20000, dtype=np.uint64))[0].astype(np.int64)
    assert ((2 * T[None] * ys - encoder.SCALE * ys * ys).sum(axis=1) <= best).all()


def test_encoder_degenerate_blocks_and_gain_rule():
    """Zero and non-finite blocks give the word 0; a block along a decoded
    point but longer than both gains takes the larger gain, shorter than
    both the smaller one."""
    assert encoder.encode_block(np.zeros(24, np.float32), 1.0, [14.0, 17.0]) == 0
    bad = np.zeros(24, np.float32)
    bad[3] = np.nan
    assert encoder.encode_block(bad, 1.0, [14.0, 17.0]) == 0
    bad[3] = np.inf
    assert encoder.encode_block(bad, 1.0, [14.0, 17.0]) == 0
    rng = np.random.default_rng(5)
    wd = int(rng.integers(0, 1 << 48, dtype=np.uint64))
    w, ny = _block_of(wd)
    g = [int(codec.fields(np.array([encoder.encode_block(w * s, 1.0, [ny])], np.uint64))["g"][0])
         for s in (0.5, 10.0)]
    assert g == [0, 1]


def test_retention_formula():
    """0.5 log2(1 / D) bits of the Gaussian limit over the 2 bits spent:
    D = 2^-4 is a rate of 2 bits, retention 1; D = 1/4 gives 1/2."""
    assert encoder.retention(2.0 ** -4) == pytest.approx(1.0)
    assert encoder.retention(0.25) == pytest.approx(0.5)


def test_encoder_is_nearest_to_the_scaled_direction_in_float64():
    """Sec. 3.1, Eq. 2: at a trial radius a the search keeps the point y
    nearest to t = a w / ||w||.  The oracle scores on a grid of 2^-16:
    with T_j = 2^16 t_j + e_j and |e_j| <= 1/2, its score is
    S(y) = 2^16 (||t||^2 - ||t - y||^2) + 2 e.y, so for the result y* and any
    kept point y,  ||t - y*||^2 <= ||t - y||^2 + ||y* - y||_1 / 2^16.
    Here that bound is checked with distances computed directly in float64
    (not through S) against every word one field away from y* and 20,000
    random words, for seeded Gaussian blocks at both trial radii."""
    rng = np.random.default_rng(314)
    sweeps = {"i1": 2048, "i2": 2048, "i3": 2048, "s8": 64, "b1": 2, "b2": 16, "b3": 2, "p": 2, "r": 2}
    rand = codec.decode(rng.integers(0, 1 << 48, size=20000, dtype=np.uint64))[0].astype(np.float64)
    for _ in range(3):
        w = rng.standard_normal(24).astype(np.float32)
        for a in (13.0, 15.0):
            t = a * w.astype(np.float64) / np.sqrt((w.astype(np.float64) ** 2).sum())
            _, f, y = encoder.nearest_point(encoder.targets(w, a))
            ys = [rand]
            for name, n in sweeps.items():
                ff = dict(f, g=0)
                ff[name] = np.arange(n)
                ff = {k: np.broadcast_to(np.asarray(v), (n,)) for k, v in ff.items()}
                ys.append(codec.decode(codec.pack_fields(**ff))[0].astype(np.float64))
            ys = np.concatenate(ys)
            ystar = y.astype(np.float64)
            d_star = ((t - ystar) ** 2).sum()
            d = ((t[None] - ys) ** 2).sum(axis=1)
            slack = np.abs(ys - ystar[None]).sum(axis=1) / 2.0 ** 16 + 1e-9
            assert (d_star <= d + slack).all()
            # the grid term is rarely needed: almost every listed point is plainly farther
            assert (d_star <= d + 1e-9).mean() > 0.999


def test_reconstruct_is_the_shape_gain_block_and_matches_dequant():
    """Eq. 2 for the encoder's reconstruction: a nonzero word gives a block
    along its lattice point y with Euclidean norm gain[g] * sigma; the zero
    point gives zeros; and it equals the dequantised weights
    fl32(fl32(y s_blk) sigma) within their four fp32 roundings."""
    rng = np.random.default_rng(2718)
    words = rng.integers(0, 1 << 48, size=4000, dtype=np.uint64)
    words[:4] = 0                                              # the origin, g = 0
    sig16 = (rng.uniform(0.5, 2.0, words.size) * 1e-2).astype(np.float16)
    rec = encoder.reconstruct(words, sig16.astype(np.float64))
    y = codec.decode(words)[0].astype(np.float64)
    g = codec.fields(words)["g"]
    ny = np.sqrt((y * y).sum(axis=1))
    nz = ny > 0
    assert not nz[:4].any() and np.all(rec[~nz] == 0)
    want = tables.gain().astype(np.float64)[g] * sig16.astype(np.float64)
    assert np.allclose(np.sqrt((rec * rec).sum(axis=1))[nz], want[nz], rtol=1e-12, atol=0)
    # along y: rec = c * y with one c per block
    c = (rec * y).sum(axis=1)[nz] / (ny[nz] ** 2)
    assert np.allclose(rec[nz], c[:, None] * y[nz], rtol=1e-12, atol=1e-300)
    dq = gemv.dequant(words.reshape(-1, 1), sig16).astype(np.float64)
    assert np.allclose(dq[nz], rec[nz], rtol=4 * 2.0 ** -24, atol=0)
