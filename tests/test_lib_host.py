"""Host-side checks of libtetra.so (no GPU needed).

* the library loads and exports every function that include/tetra.h declares;
* the library's own table builder (C++) gives byte for byte the oracle's
  tables (the two are written independently from the same conventions);
* pack/unpack round trips and the documented chunk layout;
* argument validation returns the documented status codes before any launch.
"""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_35465_amd as tt
from oracle import tables as otables

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "tetra.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tetra_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert len(names) >= 8
    lib = tt.library()
    for n in names:
        assert hasattr(lib, n), n
        assert isinstance(getattr(lib, n), ctypes._CFuncPtr)
    assert set(names) == set(tt.EXPORTED)


def test_tables_match_oracle_bytes():
    blob = tt.get_tables()
    assert len(blob) == tt.TABLE_BLOB_BYTES == otables.BLOB_BYTES
    assert blob == otables.table_blob()


def test_status_strings():
    for s in (tt.OK, tt.EINVAL, tt.EALIGN, tt.EDEVICE, tt.EUNSUPPORTED, tt.EBUSY):
        assert tt.status_string(s)
    assert tt.status_string(12345) == "unknown status"


@pytest.mark.parametrize("M,K", [(1, 24), (64, 1536), (65, 24 * 7 + 8), (130, 2560), (17, 48)])
def test_pack_unpack_round_trip(M, K):
    rng = np.random.default_rng(M * 1000 + K)
    words = rng.integers(0, 1 << 48, size=(M, K // 24), dtype=np.uint64)
    tail = rng.standard_normal((M, K % 24)).astype(np.float16)
    blob = tt.pack_rows(words, tail, M, K)
    assert blob.nbytes == tt.codes_bytes(M, K)
    w2, t2 = tt.unpack_rows(blob, M, K)
    assert np.array_equal(w2, words)
    assert np.array_equal(t2.view(np.uint16), tail.view(np.uint16))


def _device_word(w: int):
    """The recoding documented in include/tetra.h, written out again here."""
    f = {k: (w >> lsb) & ((1 << n) - 1) for k, (lsb, n) in {
        "s8": (0, 6), "p": (6, 1), "r": (7, 1), "b1": (8, 1), "b2": (9, 4), "b3": (13, 1),
        "g": (14, 1), "i1": (15, 11), "i2": (26, 11), "i3": (37, 11)}.items()}

    def phys(cls, i):
        return 2048 + i if cls else (i + 808) % 2048

    delta = int(f["i2"] >= 1240)
    r3 = f["p"] ^ f["r"] ^ delta
    path = f["s8"] | f["b1"] << 6 | f["b2"] << 7 | f["b3"] << 11
    phys1 = phys(f["r"], f["i1"])
    u3 = phys(r3, f["i3"]) ^ (delta << 11)
    lo = path | f["g"] << 12 | phys1 << 13 | (f["i2"] & 0x7F) << 25
    hi = (f["i2"] >> 7) | u3 << 4
    return lo, hi


def _stored_word(blob, nblk, tile, r, b):
    """(lo32, hi16) of row r, block column b of a tile, by the layout that
    include/tetra.h documents (groups of four columns, then single columns)."""
    base = tile * nblk * 384
    ng = nblk // 4
    if b < 4 * ng:
        g, k = divmod(b, 4)
        lo_at = base + g * 1536 + 16 * r + 4 * k
        hi_at = base + g * 1536 + 1024 + 8 * r + 2 * k
    else:
        s, q = nblk - 4 * ng, b - 4 * ng
        run = base + ng * 1536
        lo_at = run + 4 * s * r + 4 * q
        hi_at = run + 256 * s + 2 * min(s, 2) * r + 2 * q if q < 2 else run + 1024 + 2 * r
    lo = int(blob[lo_at:lo_at + 4].view(np.uint32)[0])
    hi = int(blob[hi_at:hi_at + 2].view(np.uint16)[0])
    return lo, hi


@pytest.mark.parametrize("nblk,T", [(3, 16), (9, 6), (8, 0), (6, 2), (7, 10), (2, 0), (1, 4)])
def test_pack_layout_is_the_documented_chunking(nblk, T):
    M, K = 70, 24 * nblk + T
    rng = np.random.default_rng(3 + nblk)
    words = rng.integers(0, 1 << 48, size=(M, nblk), dtype=np.uint64)
    words[0, 0] = 0
    words[1, 0] = (1 << 48) - 1
    tail = rng.standard_normal((M, T)).astype(np.float16) if T else None
    blob = tt.pack_rows(words, tail, M, K)
    tiles = 2
    for row in (0, 1, 5, 63, 64, 69):
        tile, r = divmod(row, 64)
        for b in range(nblk):
            assert _stored_word(blob, nblk, tile, r, b) == _device_word(int(words[row, b]))
    # padded rows of the last tile hold the recoded zero word
    for r in (6, 40, 63):
        for b in range(nblk):
            assert _stored_word(blob, nblk, 1, r, b) == _device_word(0)
    tail_off = (tiles * nblk * 384 + 15) // 16 * 16
    assert tt.tail_offset(M, K) == tail_off
    assert tt.codes_bytes(M, K) == tail_off + 2 * M * T
    if T:
        assert np.array_equal(blob[tail_off:].view(np.uint16).reshape(M, T), tail.view(np.uint16))


def test_recoding_is_one_to_one():
    rng = np.random.default_rng(8)
    words = rng.integers(0, 1 << 48, size=(64, 41), dtype=np.uint64)
    # adversarial words: every field at its extremes, and delta on both sides
    words[0, :4] = [0, (1 << 48) - 1, 1239 << 26, 1240 << 26]
    blob = tt.pack_rows(words, None, 64, 24 * 41)
    dev = np.array([[_stored_word(blob, 41, 0, r, b) for b in range(41)] for r in range(64)],
                   dtype=np.uint64)
    packed = dev[..., 0] | dev[..., 1] << np.uint64(32)
    assert np.all(packed < (1 << 48))
    assert len(set(packed.ravel().tolist())) == len(set(words.ravel().tolist()))
    for r in range(64):
        for b in range(41):
            assert tuple(int(v) for v in dev[r, b]) == _device_word(int(words[r, b]))


def test_codes_bytes_and_bits_per_weight():
    assert tt.codes_bytes(0, 24) == 0 and tt.codes_bytes(4, 23) == 0 and tt.codes_bytes(4, 25) == 0
    # 48 bits per block + 16 per tail weight; + 16 per row for the fp16 scale
    M, K = 5120, 17408
    n = tt.codes_bytes(M, K)
    assert n == (M // 64) * (K // 24) * 384 + M * (K % 24) * 2
    bw = (n + 2 * M) * 8 / (M * K)
    assert 2.0 < bw < 2.2


def test_row_stride_is_the_tile_stride_per_row():
    """48 bits per block and row; a tile of TETRA_ROW_TILE rows spans
    TETRA_ROW_TILE row strides, so tile t starts at t * 64 * row_stride."""
    for K in (24, 48, 1536, 2560, 5120, 17408, 24 * 7 + 8):
        assert tt.row_stride(K) == 6 * (K // 24)
        M = 3 * tt.ROW_TILE + 5
        assert tt.tail_offset(M, K) == ((M + 63) // 64) * tt.ROW_TILE * tt.row_stride(K)
    rng = np.random.default_rng(1)
    M, K = 130, 24 * 9 + 8
    words = rng.integers(0, 1 << 48, size=(M, K // 24), dtype=np.uint64)
    blob = tt.pack_rows(words, np.zeros((M, 8), np.float16), M, K)
    t = 1                                    # changing tile 1's rows changes only its bytes
    words2 = words.copy()
    words2[64:128] ^= np.uint64(0xFFFF_FFFF_FFFF)
    blob2 = tt.pack_rows(words2, np.zeros((M, 8), np.float16), M, K)
    diff = np.flatnonzero(blob != blob2)
    start = t * tt.ROW_TILE * tt.row_stride(K)
    assert diff.min() >= start and diff.max() < start + tt.ROW_TILE * tt.row_stride(K)
    assert tt.row_stride(23) == 0 and tt.row_stride(25) == 0


def test_pack_rejects_bad_input():
    words = np.zeros((2, 1), np.uint64)
    words[1, 0] = 1 << 48
    with pytest.raises(tt.TetraError) as e:
        tt.pack_rows(words, None, 2, 24)
    assert e.value.status == tt.EINVAL
    lib = tt.library()
    assert lib.tetra_pack_rows(None, None, 2, 24, None, 0) == tt.EINVAL
    buf = np.zeros(10, np.uint8)
    ok = np.zeros((2, 1), np.uint64)
    assert lib.tetra_pack_rows(ok.ctypes.data, None, 2, 24, buf.ctypes.data, 10) == tt.EINVAL
    # a tail is required when K % 24 != 0
    big = np.zeros(tt.codes_bytes(2, 40), np.uint8)
    w1 = np.zeros((2, 1), np.uint64)
    assert lib.tetra_pack_rows(w1.ctypes.data, None, 2, 40, big.ctypes.data, big.nbytes) == tt.EINVAL


def test_launch_entry_points_validate_before_touching_the_device():
    lib = tt.library()
    fake = 0x1000                   # never dereferenced: validation fails first
    assert lib.tetra_gemv(None, fake, fake, fake, 64, 48, 1, None) == tt.EINVAL
    assert lib.tetra_gemv(fake, fake, fake, fake, 0, 48, 1, None) == tt.EINVAL
    assert lib.tetra_gemv(fake, fake, fake, fake, 64, 23, 1, None) == tt.EINVAL
    assert lib.tetra_gemv(fake, fake, fake, fake, 64, 48, 0, None) == tt.EINVAL
    assert lib.tetra_gemv(fake, fake, fake, fake, 64, 48, 9, None) == tt.EINVAL
    assert lib.tetra_gemv(fake + 4, fake, fake, fake, 64, 48, 1, None) == tt.EALIGN
    assert lib.tetra_gemv(fake, fake, fake + 2, fake, 64, 48, 1, None) == tt.EALIGN
    assert lib.tetra_decode(None, 10, fake, None, None) == tt.EINVAL
    assert lib.tetra_decode(fake, 0, fake, None, None) == tt.EINVAL
    assert lib.tetra_decode(fake + 1, 4, fake, None, None) == tt.EALIGN
    assert lib.tetra_dequant(fake, None, 64, 48, fake, None) == tt.EINVAL
    assert lib.tetra_dequant(fake + 8, fake, 64, 48, fake, None) == tt.EALIGN


def test_grouped_validation():
    lib = tt.library()
    fake = 0x1000
    good = tt.Problem(fake, fake, fake, fake, 64, 48)
    bad = tt.Problem(fake, fake, fake, fake, 64, 23)
    arr = (tt.Problem * (tt.MAX_GROUP + 1))(*([good] * (tt.MAX_GROUP + 1)))
    p = ctypes.cast(arr, ctypes.c_void_p)
    assert lib.tetra_gemv_grouped(None, 1, 1, None) == tt.EINVAL
    assert lib.tetra_gemv_grouped(p, 0, 1, None) == tt.EINVAL
    assert lib.tetra_gemv_grouped(p, tt.MAX_GROUP + 1, 1, None) == tt.EINVAL
    assert lib.tetra_gemv_grouped(p, 2, 0, None) == tt.EINVAL
    arr2 = (tt.Problem * 2)(good, bad)
    assert lib.tetra_gemv_grouped(ctypes.cast(arr2, ctypes.c_void_p), 2, 1, None) == tt.EINVAL
    mis = tt.Problem(fake + 8, fake, fake, fake, 64, 48)
    arr3 = (tt.Problem * 2)(good, mis)
    assert lib.tetra_gemv_grouped(ctypes.cast(arr3, ctypes.c_void_p), 2, 1, None) == tt.EALIGN


def test_int4_head4_and_emb4_validation():
    lib = tt.library()
    fake = 0x1000
    assert lib.tetra_int4_gemv(None, fake, fake, fake, 64, 128, 1, None) == tt.EINVAL
    assert lib.tetra_int4_gemv(fake, fake, fake, fake, 64, 100, 1, None) == tt.EINVAL   # K % 128
    assert lib.tetra_int4_gemv(fake, fake, fake, fake, 0, 128, 1, None) == tt.EINVAL
    assert lib.tetra_int4_gemv(fake, fake, fake, fake, 64, 128, 9, None) == tt.EINVAL
    assert lib.tetra_int4_gemv(fake + 4, fake, fake, fake, 64, 128, 1, None) == tt.EALIGN
    assert lib.tetra_int4_gemv(fake, fake, fake + 8, fake, 64, 128, 1, None) == tt.EALIGN
    assert lib.tetra_head4_gemv(None, fake, fake, fake, 64, 64, 1, None) == tt.EINVAL
    assert lib.tetra_head4_gemv(fake, fake, fake, fake, 64, 96, 1, None) == tt.EINVAL    # dim % 64
    assert lib.tetra_head4_gemv(fake, fake, fake, fake, 0, 64, 1, None) == tt.EINVAL
    assert lib.tetra_head4_gemv(fake, fake, fake, fake, 64, 64, 0, None) == tt.EINVAL
    assert lib.tetra_head4_gemv(fake, fake + 2, fake, fake, 64, 64, 1, None) == tt.EALIGN
    assert lib.tetra_head4_gemv(fake, fake, fake + 4, fake, 64, 64, 1, None) == tt.EALIGN
    assert lib.tetra_gemm(None, fake, fake, fake, 64, 96, 16, fake, 1 << 20, None) == tt.EINVAL
    assert lib.tetra_gemm(fake, fake, fake, fake, 64, 100, 16, fake, 1 << 20, None) == tt.EINVAL   # K % 8
    assert lib.tetra_gemm(fake, fake, fake, fake, 64, 96, 0, fake, 1 << 20, None) == tt.EINVAL
    assert lib.tetra_gemm(fake, fake, fake, fake, 0, 96, 16, fake, 1 << 20, None) == tt.EINVAL
    assert lib.tetra_gemm(fake + 8, fake, fake, fake, 64, 96, 16, fake, 1 << 20, None) == tt.EALIGN
    assert lib.tetra_gemm(fake, fake, fake + 8, fake, 64, 96, 16, fake, 1 << 20, None) == tt.EALIGN
    assert lib.tetra_gemm(fake, fake, fake, fake, 64, 96, 16, None, 1 << 20, None) == tt.EINVAL    # no workspace
    assert lib.tetra_gemm(fake, fake, fake, fake, 64, 96, 16, fake + 16, 1 << 20, None) == tt.EALIGN
    assert lib.tetra_rotate(None, fake, fake, 1024, 256, 1, None) == tt.EINVAL
    assert lib.tetra_rotate(fake, fake, fake, 1024, 96, 1, None) == tt.EINVAL       # n not a power of two
    assert lib.tetra_rotate(fake, fake, fake, 1024, 2, 1, None) == tt.EINVAL        # n < 4
    assert lib.tetra_rotate(fake, fake, fake, 8192, 8192, 1, None) == tt.EINVAL     # n > 4096
    assert lib.tetra_rotate(fake, fake, fake, 1000, 256, 1, None) == tt.EINVAL      # n does not divide K
    assert lib.tetra_rotate(fake, fake, fake, 1024, 256, 0, None) == tt.EINVAL
    assert lib.tetra_rotate(fake + 4, fake, fake, 1024, 256, 1, None) == tt.EALIGN
    assert lib.tetra_rotate(fake, fake, fake + 2, 1024, 256, 1, None) == tt.EALIGN
    assert lib.tetra_emb4_gather(None, fake, 10, 128, fake, 1, fake, None) == tt.EINVAL
    assert lib.tetra_emb4_gather(fake, fake, 10, 96, fake, 1, fake, None) == tt.EINVAL    # dim % 64
    assert lib.tetra_emb4_gather(fake, fake, 0, 128, fake, 1, fake, None) == tt.EINVAL
    assert lib.tetra_emb4_gather(fake, fake, 10, 128, fake, 0, fake, None) == tt.EINVAL
    assert lib.tetra_emb4_gather(fake, fake, 10, 128, fake + 2, 1, fake, None) == tt.EALIGN
    assert lib.tetra_encode(None, fake, 4, 14.0, 17.0, fake, None) == tt.EINVAL
    assert lib.tetra_encode(fake, fake, 0, 14.0, 17.0, fake, None) == tt.EINVAL
    assert lib.tetra_encode(fake, fake, 4, 0.0, 17.0, fake, None) == tt.EINVAL          # radius <= 0
    assert lib.tetra_encode(fake, fake, 4, 14.0, 25.5, fake, None) == tt.EINVAL         # radius > 25
    assert lib.tetra_encode(fake, fake, 4, float("nan"), 17.0, fake, None) == tt.EINVAL
    assert lib.tetra_encode(fake + 2, fake, 4, 14.0, 17.0, fake, None) == tt.EALIGN
    assert lib.tetra_encode(fake, fake, 4, 14.0, 17.0, fake + 1, None) == tt.EALIGN



def test_kernel_hash_ignores_comments_only():
    """The traffic record's source hash covers code, not comments: stripping
    comments keeps every code line and drops comment-only text."""
    import bench
    src = 'int a = 1; // one\n/* block\n comment */ int b = 2;\n  \nasm("s // t"); // x\n'
    assert bench._code_only(src) == 'int a = 1;\n int b = 2;\nasm("s // t");'
    assert bench._code_only(src) != bench._code_only(src.replace("2;", "3;"))
