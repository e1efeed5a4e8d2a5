"""CPU oracle for the Tetra decode and the fused decode-GEMV.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP library and
its Python binding) imports, links or runs this package. Only the tests, the
smoke check and the CPU-baseline leg of the benchmark use it.

The oracle is written from the paper ("Tetra: Serving Leech-Lattice Quantized
LLMs at 2.7 Bits per Parameter") and shares no code, table or constant
generator with the HIP path. It is deliberately plain and slow:

* ``golay``  - the extended binary Golay code and the octad trio (Sec. 3.1,
  Eq. 1; Sec. 3.2).
* ``tables`` - the trellis tables, the coordinate value lists, the rank table,
  the middle-section list, the norm and gain tables (Sec. 3.2-3.4, Fig. 4).
* ``codec``  - the decode of a 48-bit word into a point of the Leech lattice
  and its block scale (Sec. 3.3-3.4, Eq. 2, Eq. 3, Fig. 4), the inverse map
  used for round trips, and an independent lattice membership test (Eq. 1).
* ``gemv``   - dequantised weights and the float64 matrix-vector product
  (Eq. 2; Sec. 4.1 for the unquantised row tail; Sec. 5.1 for the product).
* ``int4``   - the secondary int4 projection record and the 4-bit embedding
  row gather (Sec. 4.3, Sec. 4.4).

Parity status of every function is stated in its module header.
"""

from . import golay, tables, codec, gemv, int4  # noqa: F401
