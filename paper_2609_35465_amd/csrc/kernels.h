// HIP kernels for gfx950: bulk decode, dense reconstruction, fused GEMV.
// Included once, by tetra.hip.
#pragma once

#include <hip/hip_runtime.h>

#include "device_tables.h"
#include "word_format.h"

namespace tetra_dev {

constexpr int kTile = 64;                 // rows per code tile = lanes per wave
constexpr int kChunk = kTile * 6;         // bytes per (tile, block column) chunk
constexpr int kGemvWaves = 16;
constexpr int kGemvThreads = kGemvWaves * 64;
constexpr int kMaxGroup = 16;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(4))) const uint32_t const_u32;

__device__ __forceinline__ float f16(uint16_t v) {
    return static_cast<float>(__builtin_bit_cast(_Float16, v));
}

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b), c,
                                  false);
}

__device__ __forceinline__ uint32_t pk_add(uint32_t a, uint32_t b) {
    return __builtin_bit_cast(uint32_t, __builtin_bit_cast(half2_t, a) + __builtin_bit_cast(half2_t, b));
}

// ------------------------------------------------- canonical-word decode
//
// Fig. 4 on canonical words: path bytes from the flattened trellis table,
// three rank rows (the middle one through its own list), r3 = p ^ r ^ delta
// (Eq. 3).  Coordinate value of offset o = p + 2c and rank rho: the rho-th
// element of o + 4Z outward from zero, positive first, which equals
// (2p-1)(1-2c)(-1)^rho (2 rho + 1) + (1-p).

__device__ __forceinline__ int canonical_value(uint32_t pat, const uint32_t rho[3], uint32_t p,
                                               int j) {
    const uint32_t c = pat >> j & 1u;
    const uint32_t rk = rho[j >> 3] >> (4 * (j & 7)) & 15u;
    const int u = static_cast<int>(2 * rk + 1);
    const uint32_t neg = (rk ^ c ^ p ^ 1u) & 1u;
    return (neg ? -u : u) + static_cast<int>(1u - p);
}

__global__ __launch_bounds__(256) void decode_kernel(const uint16_t* __restrict__ words, size_t n,
                                                     int8_t* __restrict__ y_out,
                                                     float* __restrict__ scale_out) {
    __shared__ uint32_t s_path[4096], s_rows[4096];
    __shared__ float s_inv[32], s_gain[2];
    for (int i = threadIdx.x; i < 4096; i += blockDim.x) {
        s_path[i] = g_canonical.path_bytes[i];
        s_rows[i] = g_canonical.rows[i];
    }
    if (threadIdx.x < 32) s_inv[threadIdx.x] = g_canonical.invnorm[threadIdx.x];
    if (threadIdx.x < 2) s_gain[threadIdx.x] = g_canonical.gain[threadIdx.x];
    __syncthreads();
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x; i < n;
         i += static_cast<size_t>(gridDim.x) * blockDim.x) {
        const uint64_t w = words[3 * i] | static_cast<uint64_t>(words[3 * i + 1]) << 16 |
                           static_cast<uint64_t>(words[3 * i + 2]) << 32;
        const tetra::CanonicalFields f = tetra::canonical_fields(w);
        const uint32_t pat = s_path[f.s8 | f.b1 << 6 | f.b2 << 7 | f.b3 << 11];
        const uint32_t delta = f.i2 >= tetra::kMidClass0Rows ? 1u : 0u;
        const uint32_t mid = delta ? 2048u + (f.i2 - tetra::kMidClass0Rows) : f.i2;
        const uint32_t r3 = f.p ^ f.r ^ delta;
        const uint32_t rho[3] = {s_rows[f.r << 11 | f.i1], s_rows[mid], s_rows[r3 << 11 | f.i3]};
        int sq = 0;
        uint32_t* yo = reinterpret_cast<uint32_t*>(y_out + 24 * i);
        for (int q = 0; q < 6; ++q) {
            uint32_t v = 0;
            for (int e = 0; e < 4; ++e) {
                const int yv = canonical_value(pat, rho, f.p, 4 * q + e);
                sq += yv * yv;
                v |= (static_cast<uint32_t>(yv) & 0xFFu) << (8 * e);
            }
            yo[q] = v;
        }
        if (scale_out) scale_out[i] = s_gain[f.g] * s_inv[(sq >> 4) & 31];
    }
}

// ---------------------------------------------------- packed-word decode
//
// Device words (word_format.h) against the packed tables: the signed rank
// values of a section come from LDS as fp16 pairs, the path's codeword bits
// flip their signs (F = (1-2c) U), and H = F - (1-p) gives the lattice point
// as y = (2p-1) H, so that sum y^2 = sum H^2 and y.x = (2p-1) H.x.

struct PackedDecode {
    uint32_t h[12];     // fp16 pairs of H, coordinate pairs (2j, 2j+1)
    uint32_t p, g;
};

__device__ __forceinline__ void stage_packed_tables(uint8_t* lds) {
    const uint4* src = reinterpret_cast<const uint4*>(&g_packed);
    uint4* dst = reinterpret_cast<uint4*>(lds);
    for (int i = threadIdx.x; i < static_cast<int>(kPackedTableBytes / 16); i += blockDim.x)
        dst[i] = src[i];
}

__device__ __forceinline__ PackedDecode decode_packed(uint32_t lo, uint32_t hi,
                                                      const uint32_t* s_rows,
                                                      const uint32_t* s_path) {
    PackedDecode d;
    const uint32_t pa = lo & 0xFFFu;
    d.g = lo >> 12 & 1u;
    const uint32_t a1 = lo >> 13 & 0xFFFu;
    const uint32_t i2 = __builtin_amdgcn_alignbit(hi, lo, 25) & 0x7FFu;
    const uint32_t am = i2 + tetra::kMidOffset;            // bit 11 = delta
    const uint32_t u3 = hi >> 4 & 0xFFFu;
    const uint32_t a3 = u3 ^ (am & 0x800u);
    d.p = (a1 ^ u3) >> 11;
    const uint32_t e = s_path[pa];
    const uint4 r0 = *reinterpret_cast<const uint4*>(s_rows + 4 * a1);
    const uint4 r1 = *reinterpret_cast<const uint4*>(s_rows + 4 * am);
    const uint4 r2 = *reinterpret_cast<const uint4*>(s_rows + 4 * a3);
    const uint32_t rv[12] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w, r2.x, r2.y, r2.z, r2.w};
    const uint32_t negq = d.p ? 0u : 0xBC00BC00u;          // fp16 pair (-1, -1) when p = 0
#pragma unroll
    for (int j = 0; j < 12; ++j) d.h[j] = pk_add(rv[j] ^ ((e << j) & 0x80008000u), negq);
    return d;
}

__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* __restrict__ codes,
                                                      const uint16_t* __restrict__ sigma, int M,
                                                      int K, int nblk, int T, size_t tail_off,
                                                      float* __restrict__ w_out) {
    extern __shared__ __align__(16) uint8_t lds[];
    stage_packed_tables(lds);
    __syncthreads();
    const uint32_t* s_rows = reinterpret_cast<const uint32_t*>(lds);
    const uint32_t* s_path = s_rows + 4096 * 4;
    const float* s_scale = reinterpret_cast<const float*>(s_path + 4096);
    const int lane = threadIdx.x & 63;
    const int tiles = (M + kTile - 1) / kTile;
    const size_t units = static_cast<size_t>(tiles) * nblk;
    const size_t wave0 = (blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x) >> 6;
    const size_t nwaves = (gridDim.x * static_cast<size_t>(blockDim.x)) >> 6;
    for (size_t u = wave0; u < units; u += nwaves) {
        const int tile = static_cast<int>(u / nblk);
        const int b = static_cast<int>(u % nblk);
        const int row = tile * kTile + lane;
        const uint8_t* tb = codes + static_cast<size_t>(tile) * nblk * kChunk;
        const tetra::WordLoc at = tetra::word_loc(nblk, lane, b);
        const uint32_t lo = *reinterpret_cast<const uint32_t*>(tb + at.lo_off);
        const uint32_t hi = *reinterpret_cast<const uint16_t*>(tb + at.hi_off);
        if (row >= M) continue;
        const PackedDecode d = decode_packed(lo, hi, s_rows, s_path);
        float sq = 0.f;
#pragma unroll
        for (int j = 0; j < 12; ++j) sq = dot2(d.h[j], d.h[j], sq);
        const float sblk = s_scale[1 << 6 | d.g << 5 | ((static_cast<int>(sq) >> 4) & 31)];
        const float sg = f16(sigma[row]);
        float* wo = w_out + static_cast<size_t>(row) * K + 24 * b;
#pragma unroll
        for (int j = 0; j < 12; ++j) {
            const float h0 = f16(static_cast<uint16_t>(d.h[j]));
            const float h1 = f16(static_cast<uint16_t>(d.h[j] >> 16));
            // y = (2p-1) H; 0 - H keeps the origin's zeros positive
            const float y0 = d.p ? h0 : __fsub_rn(0.f, h0), y1 = d.p ? h1 : __fsub_rn(0.f, h1);
            wo[2 * j] = __fmul_rn(__fmul_rn(y0, sblk), sg);
            wo[2 * j + 1] = __fmul_rn(__fmul_rn(y1, sblk), sg);
        }
    }
    const uint16_t* tail = reinterpret_cast<const uint16_t*>(codes + tail_off);
    for (size_t i = blockIdx.x * static_cast<size_t>(blockDim.x) + threadIdx.x;
         i < static_cast<size_t>(M) * T; i += static_cast<size_t>(gridDim.x) * blockDim.x) {
        const size_t row = i / T, t = i % T;
        w_out[row * K + 24 * nblk + t] = f16(tail[i]);
    }
}

// ------------------------------------------------------------------ GEMV
//
// One lane per output row (64-row tiles).  A persistent workgroup of 16
// waves works in rounds; a round is 1-4 consecutive tiles of one matrix
// (more tiles for short rows, so that every wave gets about six items).
// The round's items -- groups of four block columns, then the nblk mod 4
// single columns, tile by tile -- are dealt round-robin (item i to wave
// i mod 16), each wave prefetching its next item while it decodes the
// current one.  Partial sums are combined in LDS in a fixed order, so the
// result does not depend on timing.  Rounds go to workgroups in serpentine
// order over matrices sorted by decreasing row length (done on the host).
// The activation pairs of a block column are identical for all lanes and
// come through the scalar unit as SGPR operands of v_dot2_f32_f16.

constexpr int kMaxRoundTiles = 4;

struct GemvProblem {
    const uint8_t* codes;
    const uint16_t* sigma;
    const uint16_t* x;
    float* y;
    int M, K, nblk, T;
    unsigned long long tail_off;
    int tiles, round_tiles, round_begin, pad;
};

struct GemvGroup {
    GemvProblem prob[kMaxGroup];
    int n, total_rounds, pad0, pad1;
};

// tiles per round for a matrix with `items` items per tile (B: batch)
inline int round_tiles_for(int items, int B) {
    int t = 1;
    while (t < kMaxRoundTiles && t * B * 2 <= 8 && t * items < 6 * kGemvWaves) t *= 2;
    return t;
}

inline size_t gemv_lds_bytes(int B) {
    return kPackedTableBytes + sizeof(float) * kGemvWaves * 8 * 64 + 0 * B;
}

template <int B>
__global__ __launch_bounds__(kGemvThreads) void gemv_kernel(const GemvGroup grp) {
    extern __shared__ __align__(16) uint8_t lds[];
    stage_packed_tables(lds);
    const uint32_t* s_rows = reinterpret_cast<const uint32_t*>(lds);
    const uint32_t* s_path = s_rows + 4096 * 4;
    const float* s_scale = reinterpret_cast<const float*>(s_path + 4096);
    float* s_red = reinterpret_cast<float*>(lds + kPackedTableBytes);   // [wave][slot][64]

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int G = gridDim.x;
    __syncthreads();

    for (int k = 0;; ++k) {
        const int r = k * G + ((k & 1) ? G - 1 - static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x));
        if (r >= grp.total_rounds) break;                  // uniform over the workgroup
        int pi = 0;
        while (pi + 1 < grp.n && r >= grp.prob[pi + 1].round_begin) ++pi;
        const GemvProblem& P = grp.prob[pi];
        const int tile0 = (r - P.round_begin) * P.round_tiles;
        const int ntr = min(P.round_tiles, P.tiles - tile0);
        const int nblk = P.nblk;
        const int ng = nblk / tetra::kGroupCols;
        const int per_tile = ng + (nblk - ng * tetra::kGroupCols);
        const int total = ntr * per_tile;
        const size_t tile_bytes = static_cast<size_t>(nblk) * kChunk;
        const uint8_t* tb0 = P.codes + static_cast<size_t>(tile0) * tile_bytes;
        const_u32* xc = (const_u32*)(P.x);
        const int kp = P.K >> 1;

        float acc[B];
#pragma unroll
        for (int bb = 0; bb < B; ++bb) acc[bb] = 0.f;
        auto block = [&](uint32_t lo, uint32_t hi, int b) {
            const PackedDecode d = decode_packed(lo, hi, s_rows, s_path);
            float sq = 0.f;
#pragma unroll
            for (int j = 0; j < 12; ++j) sq = dot2(d.h[j], d.h[j], sq);
            const float s = s_scale[d.p << 6 | d.g << 5 | ((static_cast<int>(sq) >> 4) & 31)];
#pragma unroll
            for (int bb = 0; bb < B; ++bb) {
                float dt = 0.f;
#pragma unroll
                for (int j = 0; j < 12; ++j) dt = dot2(d.h[j], xc[bb * kp + 12 * b + j], dt);
                acc[bb] = fmaf(s, dt, acc[bb]);
            }
        };
        // loads of item (t, j): a group j < ng, else the single column 4ng + j - ng
        auto fetch = [&](int t, int j, uint4& lo, uint2& hi) {
            const uint8_t* tb = tb0 + static_cast<size_t>(t) * tile_bytes;
            if (j < ng) {
                const uint8_t* gp = tb + static_cast<size_t>(j) * tetra::kGroupBytes;
                lo = *reinterpret_cast<const uint4*>(gp + 16 * lane);
                hi = *reinterpret_cast<const uint2*>(gp + 1024 + 8 * lane);
            } else {
                const tetra::WordLoc at = tetra::word_loc(nblk, lane, ng * tetra::kGroupCols + (j - ng));
                lo.x = *reinterpret_cast<const uint32_t*>(tb + at.lo_off);
                hi.x = *reinterpret_cast<const uint16_t*>(tb + at.hi_off);
            }
        };
        auto flush = [&](int t) {
#pragma unroll
            for (int bb = 0; bb < B; ++bb) {
                s_red[((wave * 8) + t * B + bb) * 64 + lane] = acc[bb];
                acc[bb] = 0.f;
            }
        };

        int t = 0, j = wave, done_t = 0;                   // item wave = (t, j)
        while (j >= per_tile && t < ntr) { j -= per_tile; ++t; }
        while (done_t < t && done_t < ntr) flush(done_t++);  // tiles before the first item
        uint4 lo = make_uint4(0, 0, 0, 0);
        uint2 hi = make_uint2(0, 0);
        if (t < ntr) fetch(t, j, lo, hi);
        while (t < ntr) {
            int nt = t, nj = j + kGemvWaves;
            while (nj >= per_tile && nt < ntr) { nj -= per_tile; ++nt; }
            uint4 nlo = lo;
            uint2 nhi = hi;
            if (nt < ntr) fetch(nt, nj, nlo, nhi);
            if (j < ng) {
                const int b = j * tetra::kGroupCols;
                block(lo.x, hi.x, b);
                block(lo.y, hi.x >> 16, b + 1);
                block(lo.z, hi.y, b + 2);
                block(lo.w, hi.y >> 16, b + 3);
            } else {
                block(lo.x, hi.x, ng * tetra::kGroupCols + (j - ng));
            }
            while (done_t < nt && done_t < ntr) flush(done_t++);   // leaving tile t
            t = nt;
            j = nj;
            lo = nlo;
            hi = nhi;
        }
        while (done_t < ntr) flush(done_t++);               // zeros for untouched tiles
        __syncthreads();
        if (wave < ntr * B) {
            const int tt = wave / B, bb = wave - tt * B;
            const int row = (tile0 + tt) * kTile + lane;
            if (row < P.M) {
                // sum in item-residue order: the wave holding items j = rho mod 16
                // of tile tt is (rho + tt * per_tile) mod 16, so the order of the
                // additions does not depend on how many tiles share the round
                float tot = 0.f;
                for (int rho = 0; rho < kGemvWaves; ++rho) {
                    const int w = (rho + tt * per_tile) & (kGemvWaves - 1);
                    tot += s_red[((w * 8) + tt * B + bb) * 64 + lane];
                }
                const uint16_t* tl =
                    reinterpret_cast<const uint16_t*>(P.codes + P.tail_off) + static_cast<size_t>(row) * P.T;
                const uint16_t* xt = P.x + static_cast<size_t>(bb) * P.K + 24 * nblk;
                float ts = 0.f;
                for (int q = 0; q < P.T; ++q) ts = fmaf(f16(tl[q]), f16(xt[q]), ts);
                P.y[static_cast<size_t>(bb) * P.M + row] = fmaf(f16(P.sigma[row]), tot, ts);
            }
        }
        __syncthreads();
    }
}

}  // namespace tetra_dev
