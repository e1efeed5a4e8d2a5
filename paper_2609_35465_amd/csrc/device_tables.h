// Device-resident decoder tables and their per-device upload.
// Included once, by tetra.hip (the library is a single HIP translation unit,
// so the __device__ symbols below have one definition).
#pragma once

#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <vector>

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

// Tables of the packed-matrix kernels (GEMV, dequant), staged into LDS.
//  * rows_f16[phys][k]: the rank row at physical position phys (see
//    word_format.h), as the fp16 pair (U_2k, U_2k+1) of its signed values
//    U = (-1)^rho (2 rho + 1);
//  * path_e[path]: the 24 codeword bits of a path, coordinates 2j and 2j+1
//    at bits 15-j and 31-j, so (E << j) & 0x80008000 is the fp16 sign mask
//    of coordinate pair j;
//  * scale[p << 6 | g << 5 | m] = (2p - 1) * fl32(gain[g] * invnorm[m]).
struct PackedTables {
    uint32_t rows_f16[4096][4];
    uint32_t path_e[4096];
    float scale[128];
};

constexpr size_t kPackedTableBytes = sizeof(PackedTables);   // 82,432 B

__device__ CanonicalTables g_canonical;
__device__ PackedTables g_packed;

inline uint16_t fp16_of_small_int(int v) {
    if (v == 0) return 0;
    const uint16_t sign = v < 0 ? 0x8000 : 0;
    const unsigned a = static_cast<unsigned>(v < 0 ? -v : v);
    const int e = 31 - __builtin_clz(a);
    const unsigned mant = (a << (10 - e)) & 0x3FFu;
    return static_cast<uint16_t>(sign | (e + 15) << 10 | mant);
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
    for (uint32_t phys = 0; phys < 4096; ++phys) {
        const uint32_t cls = phys >= 2048u ? 1u : 0u;
        const uint32_t row = T.rows[cls * 2048u + tetra::half_index(phys)];
        for (int k = 0; k < 4; ++k) {
            uint32_t pair = 0;
            for (int h2 = 0; h2 < 2; ++h2) {
                const int rho = static_cast<int>(row >> (4 * (2 * k + h2)) & 15u);
                const int u = (rho & 1 ? -1 : 1) * (2 * rho + 1);
                pair |= static_cast<uint32_t>(fp16_of_small_int(u)) << (16 * h2);
            }
            h->rows_f16[phys][k] = pair;
        }
    }
    for (int path = 0; path < 4096; ++path) {
        const uint32_t pb = T.path_bytes[path];
        uint32_t e = 0;
        for (int t = 0; t < 24; ++t) {
            const uint32_t c = pb >> t & 1u;      // byte s, bit tt = block coordinate 8s + tt
            const int j = t >> 1;
            e |= c << ((t & 1) ? 31 - j : 15 - j);
        }
        h->path_e[path] = e;
    }
    for (int p = 0; p < 2; ++p)
        for (int g = 0; g < 2; ++g)
            for (int m = 0; m < 32; ++m) {
                const float s = T.gain[g] * T.invnorm[m];
                h->scale[p << 6 | g << 5 | m] = p ? s : -s;
            }
}

}  // namespace tetra_dev
