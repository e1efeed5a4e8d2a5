// Device word format of the packed code blob (host and device).
//
// The paper's loader only reorders the bits of each 48-bit word (Sec. 5.1).
// This library's loader applies a bijective recoding that keeps every word
// at 48 bits but puts the decoder's table addresses next to each other:
//
//   path  (12) = s8 | b1 << 6 | b2 << 7 | b3 << 11   trellis path index
//   g     (1)
//   phys1 (12) = physical rank row of section 1       (class r, index i1)
//   i2    (11) = middle-list index, unchanged
//   u3    (12) = (p ^ r) << 11 | i3'                  section-3 row without delta
//
//   lo = path | g << 12 | phys1 << 13 | (i2 & 0x7F) << 25
//   hi = i2 >> 7 | u3 << 4
//
// Physical row order of the rank table: class-0 row i sits at
// (i + 808) mod 2048 and class-1 row i at 2048 + i.  The middle list
// (first 1240 class-0 rows, then the class-1 rows) is then the contiguous
// range 808 + i2, and delta = [i2 >= 1240] is bit 11 of 808 + i2.  With
// r3 = p ^ r ^ delta (Eq. 3), section 3's physical row is u3 ^ delta << 11,
// and p = bit 11 of phys1 ^ bit 11 of u3.
#pragma once

#include <cstdint>

namespace tetra {

constexpr uint32_t kMidOffset = 808;      // 2048 - 1240
constexpr uint32_t kMidClass0Rows = 1240;

struct CanonicalFields {
    uint32_t s8, p, r, b1, b2, b3, g, i1, i2, i3;
};

__host__ __device__ inline CanonicalFields canonical_fields(uint64_t w) {
    CanonicalFields f;
    f.s8 = static_cast<uint32_t>(w & 63u);
    f.p = static_cast<uint32_t>(w >> 6 & 1u);
    f.r = static_cast<uint32_t>(w >> 7 & 1u);
    f.b1 = static_cast<uint32_t>(w >> 8 & 1u);
    f.b2 = static_cast<uint32_t>(w >> 9 & 15u);
    f.b3 = static_cast<uint32_t>(w >> 13 & 1u);
    f.g = static_cast<uint32_t>(w >> 14 & 1u);
    f.i1 = static_cast<uint32_t>(w >> 15 & 2047u);
    f.i2 = static_cast<uint32_t>(w >> 26 & 2047u);
    f.i3 = static_cast<uint32_t>(w >> 37 & 2047u);
    return f;
}

__host__ __device__ inline uint64_t canonical_word(const CanonicalFields& f) {
    return static_cast<uint64_t>(f.s8) | static_cast<uint64_t>(f.p) << 6 |
           static_cast<uint64_t>(f.r) << 7 | static_cast<uint64_t>(f.b1) << 8 |
           static_cast<uint64_t>(f.b2) << 9 | static_cast<uint64_t>(f.b3) << 13 |
           static_cast<uint64_t>(f.g) << 14 | static_cast<uint64_t>(f.i1) << 15 |
           static_cast<uint64_t>(f.i2) << 26 | static_cast<uint64_t>(f.i3) << 37;
}

// physical row of class `cls`, index i
__host__ __device__ inline uint32_t phys_row(uint32_t cls, uint32_t i) {
    return cls ? 2048u + i : (i + kMidOffset) & 2047u;
}

__host__ __device__ inline uint32_t half_index(uint32_t phys) {
    return phys >= 2048u ? phys - 2048u : (phys + 2048u - kMidOffset) & 2047u;
}

struct DeviceWord {
    uint32_t lo, hi;   // hi uses its low 16 bits
};

__host__ __device__ inline DeviceWord device_word(uint64_t canonical) {
    const CanonicalFields f = canonical_fields(canonical);
    const uint32_t path = f.s8 | f.b1 << 6 | f.b2 << 7 | f.b3 << 11;
    const uint32_t delta = f.i2 >= kMidClass0Rows ? 1u : 0u;
    const uint32_t r3 = f.p ^ f.r ^ delta;
    const uint32_t phys1 = phys_row(f.r, f.i1);
    const uint32_t u3 = phys_row(r3, f.i3) ^ delta << 11;
    DeviceWord d;
    d.lo = path | f.g << 12 | phys1 << 13 | (f.i2 & 0x7Fu) << 25;
    d.hi = (f.i2 >> 7) | u3 << 4;
    return d;
}

__host__ __device__ inline uint64_t canonical_from_device(DeviceWord d) {
    CanonicalFields f;
    const uint32_t path = d.lo & 0xFFFu;
    f.s8 = path & 63u;
    f.b1 = path >> 6 & 1u;
    f.b2 = path >> 7 & 15u;
    f.b3 = path >> 11 & 1u;
    f.g = d.lo >> 12 & 1u;
    const uint32_t phys1 = d.lo >> 13 & 0xFFFu;
    f.i2 = (d.lo >> 25 & 0x7Fu) | (d.hi & 0xFu) << 7;
    const uint32_t u3 = d.hi >> 4 & 0xFFFu;
    const uint32_t delta = f.i2 >= kMidClass0Rows ? 1u : 0u;
    f.r = phys1 >> 11;
    f.i1 = half_index(phys1);
    f.p = (u3 >> 11) ^ f.r;
    const uint32_t phys3 = u3 ^ delta << 11;
    f.i3 = half_index(phys3);
    return canonical_word(f);
}

// Placement of the words of one 64-row tile (tiles are nblk * 384 bytes).
// Block columns go in groups of four: group g is a 1536-byte run holding, for
// lane (row in tile) r, the 32-bit parts of columns 4g..4g+3 at 16r and
// their 16-bit parts at 1024 + 8r, so a lane reads a group with one 16-byte
// and one 8-byte load.  The s = nblk mod 4 trailing columns follow as one
// run of 384 s bytes, laid out so that a lane reads them with whole loads and
// no bit assembly: the 32-bit parts of lane r at 4 s r (columns in order);
// the 16-bit parts of the first two columns at 256 s + 2 min(s, 2) r, and
// that of a third column at 1024 + 2r.
constexpr int kGroupCols = 4;
constexpr int kGroupBytes = 1536;
constexpr int kColBytes = 384;

struct WordLoc {
    uint32_t lo_off, hi_off;   // byte offsets from the tile base
};

__host__ __device__ inline WordLoc word_loc(int nblk, int r, int b) {
    const int ng = nblk / kGroupCols;
    WordLoc w;
    if (b < ng * kGroupCols) {
        const int g = b / kGroupCols, k = b % kGroupCols;
        w.lo_off = static_cast<uint32_t>(g * kGroupBytes + 16 * r + 4 * k);
        w.hi_off = static_cast<uint32_t>(g * kGroupBytes + 1024 + 8 * r + 2 * k);
    } else {
        const int s = nblk - ng * kGroupCols, k = b - ng * kGroupCols;
        const int base = ng * kGroupBytes;
        w.lo_off = static_cast<uint32_t>(base + 4 * s * r + 4 * k);
        w.hi_off = static_cast<uint32_t>(k < 2 ? base + 256 * s + 2 * (s < 2 ? s : 2) * r + 2 * k
                                               : base + 1024 + 2 * r);
    }
    return w;
}

}  // namespace tetra
