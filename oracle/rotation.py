"""Online activation rotation (oracle, test-only).

Paper passages followed:
* Sec. 3.1: the encoder rotates its input in the manner of the randomized
  Hadamard incoherence processing it cites, so the served model must apply
  the same rotation to the activations.
* Sec. 5.1 (the rest of a served model): a small kernel rotates the
  activations online, once per group of projections that share a rotation.

The paper names no construction.  Reading taken: a randomized Hadamard
transform applied block by block.  For each block of n = 2^k consecutive
elements (n divides K),
    out[b, j0 + i] = (1 / sqrt(n)) * sum_m H_n[i, m] * s[j0 + m] * x[b, j0 + m]
with H_n the Sylvester Hadamard matrix (entries +-1) and s in {+1, -1} the
random signs, drawn by the caller and passed in (bit k of byte k // 8 set
means s[k] = -1).  The GPU computes in fp32 and rounds the result to fp16.

Definition used as the parity target: the dense product above in float64,
with scipy.linalg.hadamard as the matrix (a library primitive).

Pins (tests): H_n has entries +-1 and H_n H_n^T = n I; it satisfies the
Sylvester recursion H_2n = [[H_n, H_n], [H_n, -H_n]] (brute force over
small n); the rotation preserves the Euclidean norm of every block; two
applications of the unsigned transform give the input back; a one-hot input
gives one column of H_n / sqrt(n).
"""

import numpy as np
from scipy.linalg import hadamard


def signs_from_bits(bits: np.ndarray, K: int) -> np.ndarray:
    """float64 [K] of +-1 from the packed sign bits (bit k of byte k // 8)."""
    b = np.unpackbits(np.asarray(bits, np.uint8), bitorder="little")[:K]
    return 1.0 - 2.0 * b.astype(np.float64)


def rotate_f64(x_f16: np.ndarray, sign_bits: np.ndarray, n: int) -> np.ndarray:
    """float64 [batch, K]: the blockwise randomized Hadamard transform."""
    x = np.atleast_2d(np.asarray(x_f16, np.float16)).astype(np.float64)
    batch, K = x.shape
    assert K % n == 0 and n & (n - 1) == 0
    s = signs_from_bits(sign_bits, K)
    h = hadamard(n).astype(np.float64) / np.sqrt(n)
    xs = (x * s).reshape(batch, K // n, n)
    return np.einsum("im,btm->bti", h, xs).reshape(batch, K)
