// Layout of the decoder tables the kernels read, and their construction
// from the host tables (tables.h).  Plain C++: the table generator that runs
// at build time (gen_tables.cpp) and the HIP library share it.
#pragma once

#include <cstddef>
#include <cstdint>
#include <cstring>

#include "tables.h"
#include "word_format.h"

namespace tetra_dev {


// Canonical tables, used by the bulk decode of canonical words.
struct CanonicalTables {
    uint32_t path_bytes[4096];    // P1 | P2 << 8 | P3 << 16 at s8 | b1 << 6 | b2 << 7 | b3 << 11
    uint32_t rows[4096];          // rank rows, canonical order (class 0 then class 1)
    float invnorm[32];
    float gain[2];
    uint32_t pad[2];
};

// Tables of the packed-matrix kernels (GEMV, dequant), staged into LDS at
// byte 0 of the workgroup's allocation.
//  * path_e[path]: the 24 codeword bits of a trellis path; coordinate
//    j = 4w + i of the block sits at bit 8i + 7 - w, so that
//    (E << w) & 0x80808080 holds the signs of coordinates 4w..4w+3 in the
//    sign bits of four bytes;
//  * rows_f8[phys]: the rank row at physical position phys (word_format.h)
//    as eight fp8 (e4m3) bytes of its signed values U = (-1)^rho (2 rho + 1),
//    byte t = coordinate t of the section (exact: |U| <= 9);
//  * scale: fl32(gain[g] * invnorm[m]) at byte kScaleOff + 1024 g + 4 m.
//    The gap lets the kernels form the address straight from the bits of a
//    norm accumulated on top of 2^23 + 4096 g.
constexpr uint32_t kPathOff = 0;
constexpr uint32_t kRowsOff = 16384;
constexpr uint32_t kScaleOff = 49152;
constexpr uint32_t kScaleGStride = 1024;
//  * cost[phys]: sum over the row's eight coordinates of U^2 = (2 rho + 1)^2,
//    the part of the block norm 16 m that does not depend on the codeword or
//    on p (at most 96, one byte).
constexpr uint32_t kCostOff = kScaleOff + kScaleGStride + 32 * 4;           // 50,304
constexpr size_t kPackedTableBytes = kCostOff + 4096;                         // 54,400 B

struct PackedTables {
    uint32_t path_e[4096];
    uint32_t rows_f8[4096][2];
    float scale[kScaleGStride / 4 + 32];   // [256 g + m]; entries 32..255 unused
    uint8_t cost[4096];
};
static_assert(sizeof(PackedTables) == kPackedTableBytes, "packed table layout");
static_assert(offsetof(PackedTables, rows_f8) == kRowsOff && offsetof(PackedTables, scale) == kScaleOff &&
                  offsetof(PackedTables, cost) == kCostOff,
              "packed table offsets");
static_assert(kPackedTableBytes % 16 == 0, "tables are staged in 16-byte words");


// fp8 e4m3 bits of an odd integer |v| <= 15 (exact in e4m3)
inline uint8_t fp8_of_small_odd(int v) {
    const uint8_t sign = v < 0 ? 0x80 : 0;
    const unsigned a = static_cast<unsigned>(v < 0 ? -v : v);
    const int e = 31 - __builtin_clz(a);
    const unsigned mant = ((a << 3) >> e) & 7u;
    return static_cast<uint8_t>(sign | (e + 7) << 3 | mant);
}

inline void build_canonical(const tetra::HostTables& T, CanonicalTables* h) {
    std::memset(h, 0, sizeof(*h));
    std::memcpy(h->path_bytes, T.path_bytes, sizeof(h->path_bytes));
    std::memcpy(h->rows, T.rows, sizeof(h->rows));
    std::memcpy(h->invnorm, T.invnorm, sizeof(h->invnorm));
    std::memcpy(h->gain, T.gain, sizeof(h->gain));
}

inline void build_packed(const tetra::HostTables& T, PackedTables* h) {
    std::memset(h, 0, sizeof(*h));
    for (uint32_t path = 0; path < 4096; ++path) {
        const uint32_t pb = T.path_bytes[path];   // bit 8s + t = codeword bit of coordinate 8s + t
        uint32_t e = 0;
        for (int j = 0; j < 24; ++j) {
            const int w = j >> 2, i = j & 3;
            e |= (pb >> j & 1u) << (8 * i + 7 - w);
        }
        h->path_e[path] = e;
    }
    for (uint32_t phys = 0; phys < 4096; ++phys) {
        const uint32_t cls = phys >= 2048u ? 1u : 0u;
        const uint32_t row = T.rows[cls * 2048u + tetra::half_index(phys)];
        int cost = 0;
        for (int t = 0; t < 8; ++t) {
            const int rho = static_cast<int>(row >> (4 * t) & 15u);
            const int u = (rho & 1 ? -1 : 1) * (2 * rho + 1);
            h->rows_f8[phys][t >> 2] |= static_cast<uint32_t>(fp8_of_small_odd(u)) << (8 * (t & 3));
            cost += u * u;
        }
        h->cost[phys] = static_cast<uint8_t>(cost);
    }
    for (int g = 0; g < 2; ++g)
        for (int m = 0; m < 32; ++m) h->scale[g * (kScaleGStride / 4) + m] = T.gain[g] * T.invnorm[m];
}

}  // namespace tetra_dev
