// Host-side construction of the Tetra decoder tables.
//
// Built once per process from the definitions of the paper: the extended
// Golay code (Sec. 3.1), the octad trio and its trellis (Sec. 3.2, Fig. 2),
// the rank table and the middle-section list (Sec. 3.3), the norm table
// (Sec. 3.4) and the gain table (Eq. 2).  Conventions where the paper is
// silent are fixed in the comments of tables.cpp.
#pragma once

#include <cstdint>
#include <vector>

namespace tetra {

constexpr int kHalfRows = 2048;       // rows per class in the rank table
constexpr int kMidClass0 = 1240;      // class-0 rows at the head of the middle list
constexpr int kPaths = 4096;          // trellis paths = Golay codewords

struct HostTables {
    // canonical tables (Fig. 4)
    uint32_t rows[2 * kHalfRows];     // rank vectors, nibble j = coordinate j
    uint16_t branches[1024];          // P2 | s16 << 8, index 16*s8 + b2
    uint8_t prefixes[128];            // index 2*s8 + b1
    uint8_t suffixes[128];            // index 2*s16 + b3
    float invnorm[32];                // 1/sqrt(16 m), invnorm[0] = 0
    float gain[2];
    // derived: the three pattern bytes of every trellis path,
    // path index = s8 | b1 << 6 | b2 << 7 | b3 << 11
    uint32_t path_bytes[kPaths];      // P1 | P2 << 8 | P3 << 16
    int n_mid_class0;                 // recomputed; must equal kMidClass0
};

// Builds (once) and returns the tables; thread-safe.
const HostTables& host_tables();

// Serialises the canonical tables: rows | branches | prefixes | suffixes |
// invnorm | gain, little-endian, 18,824 bytes.
std::vector<uint8_t> canonical_blob();

}  // namespace tetra
