// Device-resident decoder tables.  Their contents are built on the host at
// build time (gen_tables.cpp writes the initialisers of tables_data.inc), so
// they are part of the code object: no call uploads, allocates or waits for
// anything to make them available on a device.
// Included once, by tetra.hip (the library is a single HIP translation unit,
// so the __device__ symbols below have one definition).
#pragma once

#include <hip/hip_runtime.h>

#include "table_layout.h"
#include "tables_data.inc"

namespace tetra_dev {

__device__ const CanonicalTables g_canonical = TETRA_CANONICAL_TABLES_INIT;
__device__ const PackedTables g_packed = TETRA_PACKED_TABLES_INIT;

}  // namespace tetra_dev
