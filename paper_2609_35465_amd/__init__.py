"""Python binding of libtetra.so (the MI355X Tetra decode-GEMV library).

Argument marshalling only: every step of the decode and the product runs in
the library's HIP kernels.  Device buffers are torch tensors on a ROCm
device (torch is used for memory and streams only); host-side helpers take
numpy arrays.  The first call loads libtetra.so, built in-tree by
``paper_2609_35465_amd.build``; a missing library raises ImportError.
"""

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtetra.so")

OK, EINVAL, EALIGN, EDEVICE, EUNSUPPORTED, EBUSY, ETIMEOUT = 0, -1, -2, -3, -4, -5, -6
ROW_TILE = 64
TABLE_BLOB_BYTES = 18824
MAX_BATCH = 8
MAX_GROUP = 32
MAX_PHASES = 16
ENCODE_MAX_RADIUS = 25.0
ENCODE_RADII = (13.0, 15.0)        # trial radii of the encoder: the best integer pair on Gaussian blocks

_vp, _sz, _int = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int

# name: (restype, argtypes)
_SIGNATURES = {
    "tetra_status_string": (ctypes.c_char_p, [_int]),
    "tetra_get_tables": (_int, [_vp, _sz]),
    "tetra_codes_bytes": (_sz, [_int, _int]),
    "tetra_row_stride": (_sz, [_int]),
    "tetra_tail_offset": (_sz, [_int, _int]),
    "tetra_pack_rows": (_int, [_vp, _vp, _int, _int, _vp, _sz]),
    "tetra_unpack_rows": (_int, [_vp, _sz, _int, _int, _vp, _vp]),
    "tetra_gemv": (_int, [_vp, _vp, _vp, _vp, _int, _int, _int, _vp]),
    "tetra_gemv_grouped": (_int, [_vp, _int, _int, _vp]),
    "tetra_gemv_chain": (_int, [_vp, _int, _vp, _int, _int, _vp, _vp]),
    "tetra_set_chain_wait_limit": (ctypes.c_uint32, [ctypes.c_uint32]),
    "tetra_decode": (_int, [_vp, _sz, _vp, _vp, _vp]),
    "tetra_dequant": (_int, [_vp, _vp, _int, _int, _vp, _vp]),
    "tetra_int4_gemv": (_int, [_vp, _vp, _vp, _vp, _int, _int, _int, _vp]),
    "tetra_head4_gemv": (_int, [_vp, _vp, _vp, _vp, _int, _int, _int, _vp]),
    "tetra_rotate": (_int, [_vp, _vp, _vp, _int, _int, _int, _vp]),
    "tetra_gemm": (_int, [_vp, _vp, _vp, _vp, _int, _int, _int, _vp, _sz, _vp]),
    "tetra_gemm_workspace_bytes": (_sz, []),
    "tetra_gemm_noalloc": (_int, [_vp, _vp, _vp, _vp, _int, _int, _int, _vp]),
    "tetra_release_stream": (_int, [_vp]),
    "tetra_emb4_gather": (_int, [_vp, _vp, _int, _int, _vp, _int, _vp, _vp]),
    "tetra_encode": (_int, [_vp, _vp, _sz, ctypes.c_double, ctypes.c_double, _vp, _vp]),
}
EXPORTED = tuple(_SIGNATURES)

_lib = None


def library():
    """The loaded ctypes library (loaded on first use; raises if it is
    missing, so no call can silently fall back to another implementation)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_2609_35465_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(lib, name)
            f.restype, f.argtypes = res, args
        _lib = lib
    return _lib


def _call(name, *args):
    return getattr(library(), name)(*args)


class TetraError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


def status_string(status: int) -> str:
    return _call("tetra_status_string", status).decode()


def _check(status, what):
    if status != OK:
        raise TetraError(status, what)


# ------------------------------------------------------------------ host side

def get_tables() -> bytes:
    buf = ctypes.create_string_buffer(TABLE_BLOB_BYTES)
    _check(_call("tetra_get_tables", buf, TABLE_BLOB_BYTES), "tetra_get_tables")
    return buf.raw


def codes_bytes(M: int, K: int) -> int:
    return int(_call("tetra_codes_bytes", M, K))


def row_stride(K: int) -> int:
    return int(_call("tetra_row_stride", K))


def tail_offset(M: int, K: int) -> int:
    return int(_call("tetra_tail_offset", M, K))


def pack_rows(words: np.ndarray, tail: np.ndarray, M: int, K: int) -> np.ndarray:
    """Device code blob (as a host uint8 array) of canonical words
    uint64 [M, K//24] and fp16 tail [M, K%24]."""
    words = np.ascontiguousarray(words, dtype=np.uint64)
    n = codes_bytes(M, K)
    if n == 0:
        raise TetraError(EINVAL, "tetra_codes_bytes")
    out = np.zeros(n, dtype=np.uint8)
    tptr = None
    if K % 24:
        tail = np.ascontiguousarray(tail, dtype=np.float16)
        tptr = tail.ctypes.data
    _check(_call("tetra_pack_rows", words.ctypes.data, tptr, M, K, out.ctypes.data, n), "tetra_pack_rows")
    return out


def unpack_rows(codes: np.ndarray, M: int, K: int):
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    words = np.zeros((M, K // 24), dtype=np.uint64)
    tail = np.zeros((M, K % 24), dtype=np.float16)
    _check(_call("tetra_unpack_rows", codes.ctypes.data, codes.nbytes, M, K, words.ctypes.data,
                       tail.ctypes.data if K % 24 else None), "tetra_unpack_rows")
    return words, tail


# ---------------------------------------------------------------- device side

def _stream(stream):
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


def gemv(codes, row_scales, x, y, M: int, K: int, batch: int = 1, stream=None):
    """y[batch, M] = W x for a packed Tetra matrix (all device tensors)."""
    _check(_call("tetra_gemv", _ptr(codes), _ptr(row_scales), _ptr(x), _ptr(y), M, K, batch,
                     _stream(stream)), "tetra_gemv")


def gemm_workspace_bytes() -> int:
    """Workspace bytes at which tetra_gemm uses the whole current device."""
    return int(_call("tetra_gemm_workspace_bytes"))


def gemm_workspace():
    """A zero-filled workspace for tetra_gemm on the current device (a torch
    uint8 tensor; torch allocates it, 256-byte aligned)."""
    import torch
    n = gemm_workspace_bytes()
    if n == 0:
        raise TetraError(EDEVICE, "tetra_gemm_workspace_bytes")
    return torch.zeros(n, dtype=torch.uint8, device="cuda")


def gemm_noalloc(codes, row_scales, x, y, M: int, K: int, N: int, stream=None):
    """tetra_gemm on the library's static per-device scratch (no workspace,
    nothing allocated); calls overlapping on one device race."""
    _check(_call("tetra_gemm_noalloc", _ptr(codes), _ptr(row_scales), _ptr(x), _ptr(y), M, K, N, _stream(stream)),
           "tetra_gemm_noalloc")


def gemm(codes, row_scales, x, y, M: int, K: int, N: int, workspace, stream=None):
    """y[N, M] = W x for N activation rows (a prompt), on the matrix cores;
    workspace from gemm_workspace() (one per stream that runs products at
    the same time as others)."""
    _check(_call("tetra_gemm", _ptr(codes), _ptr(row_scales), _ptr(x), _ptr(y), M, K, N, _ptr(workspace),
                 int(workspace.numel() * workspace.element_size()), _stream(stream)), "tetra_gemm")


def release_stream(stream=None):
    """Gives back the GEMV workspace slot that the stream holds on the current device."""
    _check(_call("tetra_release_stream", _stream(stream)), "tetra_release_stream")


def encode(w, sigma, n: int, words_out, radii=None, stream=None):
    """Canonical words [n][6 bytes] of n blocks w [n, 24] (float32, block
    order) with per-block scales sigma [n] (float32): the nearest kept point
    at two trial radii, then the gain bit."""
    r0, r1 = ENCODE_RADII if radii is None else radii
    _check(_call("tetra_encode", _ptr(w), _ptr(sigma), n, float(r0), float(r1), _ptr(words_out), _stream(stream)),
           "tetra_encode")


class Problem(ctypes.Structure):
    """tetra_gemv_problem"""
    _fields_ = [("codes", ctypes.c_void_p), ("row_scales", ctypes.c_void_p),
                ("x", ctypes.c_void_p), ("y", ctypes.c_void_p),
                ("M", ctypes.c_int), ("K", ctypes.c_int)]


def make_problems(items):
    """items: [(codes, row_scales, x, y, M, K)] of device tensors -> C array."""
    arr = (Problem * len(items))()
    for i, (c, s, x, y, M, K) in enumerate(items):
        arr[i] = Problem(_ptr(c), _ptr(s), _ptr(x), _ptr(y), M, K)
    return arr


def gemv_grouped(problems, batch: int = 1, stream=None):
    """Several products in one launch; problems from make_problems()."""
    _check(_call("tetra_gemv_grouped", ctypes.cast(problems, ctypes.c_void_p), len(problems),
                 batch, _stream(stream)), "tetra_gemv_grouped")


def gemv_chain(problems, phase_counts, batch: int = 1, status=None, stream=None):
    """Phases of products in order in one launch (problems from
    make_problems(), in phase order; phase k holds phase_counts[k] of them);
    status: an optional device int32 tensor that receives the launch's status."""
    counts = (ctypes.c_int * len(phase_counts))(*[int(c) for c in phase_counts])
    _check(_call("tetra_gemv_chain", ctypes.cast(problems, ctypes.c_void_p), len(problems),
                 ctypes.cast(counts, ctypes.c_void_p), len(phase_counts), batch, _ptr(status), _stream(stream)),
           "tetra_gemv_chain")


def set_chain_wait_limit(polls: int) -> int:
    """Test hook: polls before a chain barrier wait gives up (0: default)."""
    return int(_call("tetra_set_chain_wait_limit", int(polls)))


def decode(words_bytes, n: int, y_out, scale_out=None, stream=None):
    """words_bytes: device uint8 [n*6]; y_out int8 [n, 24]; scale_out f32 [n]."""
    _check(_call("tetra_decode", _ptr(words_bytes), n, _ptr(y_out), _ptr(scale_out),
                       _stream(stream)), "tetra_decode")


def dequant(codes, row_scales, M: int, K: int, w_out, stream=None):
    _check(_call("tetra_dequant", _ptr(codes), _ptr(row_scales), M, K, _ptr(w_out),
                        _stream(stream)), "tetra_dequant")


def int4_gemv(q, scale_off, x, y, M: int, K: int, batch: int = 1, stream=None):
    """y[batch, M] for an int4 projection: q uint8 [M, K/2], scale_off fp16
    [M, K/128, 2], x fp16 [batch, K] (all device tensors)."""
    _check(_call("tetra_int4_gemv", _ptr(q), _ptr(scale_off), _ptr(x), _ptr(y), M, K, batch,
                 _stream(stream)), "tetra_int4_gemv")


def head4_gemv(q, scale_off, x, y, rows: int, dim: int, batch: int = 1, stream=None):
    """y[batch, rows] for the 4-bit output head: q uint8 [rows, dim/2],
    scale_off fp16 [rows, dim/64, 2], x fp16 [batch, dim] (device tensors)."""
    _check(_call("tetra_head4_gemv", _ptr(q), _ptr(scale_off), _ptr(x), _ptr(y), rows, dim, batch,
                 _stream(stream)), "tetra_head4_gemv")


def rotate(x, sign_bits, out, K: int, n: int, rows: int = 1, stream=None):
    """out[rows, K] fp16 = blockwise randomized Hadamard transform of x
    (blocks of n) with the signs in sign_bits (uint8 [ceil(K/8)]); out may be x."""
    _check(_call("tetra_rotate", _ptr(x), _ptr(sign_bits), _ptr(out), K, n, rows, _stream(stream)),
           "tetra_rotate")


def emb4_gather(q, scale_off, rows: int, dim: int, tokens, out, stream=None):
    """out[n, dim] fp32 = rows tokens[n] (int32 device tensor) of a 4-bit
    embedding table q uint8 [rows, dim/2], scale_off fp16 [rows, dim/64, 2]."""
    _check(_call("tetra_emb4_gather", _ptr(q), _ptr(scale_off), rows, dim, _ptr(tokens),
                 int(tokens.numel()), _ptr(out), _stream(stream)), "tetra_emb4_gather")
