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
// Device words (word_format.h) against the packed tables.  With q = 1 - p,
// coordinate t of the block is y_t = (-1)^(c_t xor q) U(rho_t) + q: Eq. 1
// with the rank lists of Sec. 3.3 (o = 2 read as +2 first), since
// (2p - 1)(1 - 2c) = (-1)^(c xor q).  The codeword bits of the path,
// complemented when q = 1, set the sign bits of the fp8 row values; the
// values become fp16 pairs and q is added.  y is exact in fp16 (|y| <= 10).

typedef __attribute__((address_space(3))) const uint32_t lds_u32;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) const u32x2 lds_u2;
typedef __attribute__((address_space(3))) const float lds_f32;
typedef __attribute__((address_space(3))) const uint8_t lds_bytes;

// a block's table reads, issued ahead of the arithmetic that uses them
struct BlockFetch {
    uint32_t e;           // path_e of the path
    uint32_t r[6];        // fp8 rows of sections 1-3, two words each
    uint32_t pm;          // all ones when p = 1, zero when p = 0
    uint32_t bias;        // float bits of 2^23 + 4096 g
};

// lo: the 32-bit part of the word; hi: its 16-bit part in bits 0-15 (bits
// 16-31 are ignored)
__device__ __forceinline__ BlockFetch fetch_block(uint32_t lo, uint32_t hi, lds_bytes* L) {
    const uint32_t a_path = (lo << 2) & 0x3FFCu;                      // 4 * path
    const uint32_t a1 = (lo >> 10) & 0x7FF8u;                         // 8 * phys1
    const uint32_t i2 = __builtin_amdgcn_alignbit(hi, lo, 25) & 0x7FFu;
    const uint32_t am = i2 * 8u + 8u * tetra::kMidOffset;             // 8 * (808 + i2), bit 14 = delta
    const uint32_t u3 = (hi >> 1) & 0x7FF8u;                          // 8 * ((p ^ r) << 11 | i3')
    const uint32_t a3 = u3 ^ (am & 0x4000u);                          // 8 * phys3 (Eq. 3)
    BlockFetch f;
    f.pm = static_cast<uint32_t>(static_cast<int32_t>((a1 ^ u3) << 17) >> 31);   // p = r ^ (p ^ r)
    f.bias = (lo & 0x1000u) | 0x4B000000u;
    f.e = *(lds_u32*)(L + kPathOff + a_path);
    const u32x2 r0 = *(lds_u2*)(L + kRowsOff + a1);
    const u32x2 r1 = *(lds_u2*)(L + kRowsOff + am);
    const u32x2 r2 = *(lds_u2*)(L + kRowsOff + a3);
    f.r[0] = r0.x;
    f.r[1] = r0.y;
    f.r[2] = r1.x;
    f.r[3] = r1.y;
    f.r[4] = r2.x;
    f.r[5] = r2.y;
    return f;
}

template <bool High>
__device__ __forceinline__ uint32_t cvt_pair(uint32_t f8x4) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(f8x4, 1.0f, High));
}

// The 24 values of a block as fp16 pairs (coordinates 2j, 2j+1 in y[j]) and
// the byte offset of its scale in the table region: the norm 16 m is
// accumulated on top of 2^23 + 4096 g, whose float bits then read
// 0x4B000000 + 4096 g + 16 m, and bits 2-12 of that are 1024 g + 4 m.
__device__ __forceinline__ uint32_t block_values(const BlockFetch& f, uint32_t y[12]) {
    const uint32_t ep = f.e ^ (~f.pm & 0xFCFCFCFCu);
    const uint32_t qpair = ~f.pm & 0x3C003C00u;
#pragma unroll
    for (int k = 0; k < 6; ++k) {
        const uint32_t sg = f.r[k] ^ ((ep << k) & 0x80808080u);
        y[2 * k] = pk_add(cvt_pair<false>(sg), qpair);
        y[2 * k + 1] = pk_add(cvt_pair<true>(sg), qpair);
    }
    float sq = __builtin_bit_cast(float, f.bias);
#pragma unroll
    for (int j = 0; j < 12; ++j) sq = dot2(y[j], y[j], sq);
    return (__builtin_bit_cast(uint32_t, sq) >> 2) & 0x7FFu;
}

__device__ __forceinline__ void stage_packed_tables(uint4* dst) {
    const uint4* src = reinterpret_cast<const uint4*>(&g_packed);
    for (int i = threadIdx.x; i < static_cast<int>(kPackedTableBytes / 16); i += blockDim.x)
        dst[i] = src[i];
}

__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* __restrict__ codes,
                                                      const uint16_t* __restrict__ sigma, int M,
                                                      int K, int nblk, int T, size_t tail_off,
                                                      float* __restrict__ w_out) {
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    stage_packed_tables(s_tab);
    __syncthreads();
    lds_bytes* L = (lds_bytes*)(s_tab);
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
        const BlockFetch f = fetch_block(lo, hi, L);
        uint32_t y[12];
        const uint32_t sa = block_values(f, y);
        const float sblk = *(lds_f32*)(L + kScaleOff + sa);
        const float sg = f16(sigma[row]);
        float* wo = w_out + static_cast<size_t>(row) * K + 24 * b;
#pragma unroll
        for (int j = 0; j < 12; ++j) {
            wo[2 * j] = __fmul_rn(__fmul_rn(f16(static_cast<uint16_t>(y[j])), sblk), sg);
            wo[2 * j + 1] = __fmul_rn(__fmul_rn(f16(static_cast<uint16_t>(y[j] >> 16)), sblk), sg);
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
// The round's items -- groups of four block columns, then one item with
// the nblk mod 4 remaining columns, tile by tile -- are dealt round-robin
// (item i to wave i mod 16).  Each wave runs its blocks as a pipeline: the
// table reads and activation loads of the next block are issued before the
// current block's arithmetic, the current block's scale read is consumed
// one block later, and the code words of the next item are loaded one item
// ahead, so a wave waits at most once per block.  Partial sums are combined
// in LDS in a fixed order, so the result does not depend on timing or on
// the batch size.  Rounds go to workgroups in serpentine order over
// matrices sorted by decreasing row length (done on the host).  The
// activation pairs of a block column are identical for all lanes and come
// through the scalar unit as SGPR operands of v_dot2_f32_f16.

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

// reduction slots (tile x batch row) per wave
__host__ __device__ constexpr int red_slots(int B) { return B <= 4 ? 4 : 8; }

// workgroups that fit on one CU (LDS bound)
inline int gemv_wgs_per_cu(int B) { return B <= 2 ? 2 : 1; }

// tiles per round for a matrix with `items` items per tile (B: batch)
inline int round_tiles_for(int items, int B) {
    int t = 1;
    while (t < kMaxRoundTiles && 2 * t * B <= red_slots(B) && t * items < 6 * kGemvWaves) t *= 2;
    return t;
}


// code words of one item: up to four blocks; the 16-bit part of block k is
// in hi.x (k = 0, 1) or hi.y (k = 2, 3), low half for even k
struct ItemWords {
    uint4 lo;
    uint2 hi;
};

template <int K>
__device__ __forceinline__ void block_word(const ItemWords& w, uint32_t& lo, uint32_t& hi) {
    lo = K == 0 ? w.lo.x : K == 1 ? w.lo.y : K == 2 ? w.lo.z : w.lo.w;
    hi = K == 0 ? w.hi.x : K == 1 ? w.hi.x >> 16 : K == 2 ? w.hi.y : w.hi.y >> 16;
}

// per-wave pipeline state: the staged block, its activation pairs (B <= 2),
// and the previous block, whose scale read is still in flight
template <int B>
struct Pipe {
    static constexpr bool kStageX = B == 1;
    BlockFetch cur;
    uint32_t x[kStageX ? B : 1][12];
    float ps;              // scale of the previous block
    float pdt[B];          // its dot products
    int pend_t;            // its tile in the round (-1: none)
    int acc_t;             // tile of acc
    float acc[B];
};

template <int B>
__device__ __forceinline__ void load_x(uint32_t (&x)[Pipe<B>::kStageX ? B : 1][12], const_u32* xc, int kp,
                                       int col) {
    if constexpr (Pipe<B>::kStageX) {
#pragma unroll
        for (int bb = 0; bb < B; ++bb)
#pragma unroll
            for (int q = 0; q < 12; ++q) x[bb][q] = xc[bb * kp + 12 * col + q];
    }
}

// adds the previous block into acc, first storing acc when it ends a tile
template <int B>
__device__ __forceinline__ void finish_pending(Pipe<B>& st, float* red) {
    if (st.pend_t >= 0) {
        if (st.pend_t != st.acc_t) {
#pragma unroll
            for (int bb = 0; bb < B; ++bb) {
                red[(st.acc_t * B + bb) * 64] = st.acc[bb];
                st.acc[bb] = 0.f;
            }
            st.acc_t = st.pend_t;
        }
#pragma unroll
        for (int bb = 0; bb < B; ++bb) st.acc[bb] = fmaf(st.ps, st.pdt[bb], st.acc[bb]);
    }
}

// The NB blocks of one item (columns col0..col0+NB-1 of tile t), each one
// staging the next: block k+1 of this item, or block 0 of the next item
// (words nw, column ncol0; a repeat of this item when there is none).
template <int B, int NB>
__device__ __forceinline__ void run_item(Pipe<B>& st, const ItemWords& cw, const ItemWords& nw, int col0,
                                         int ncol0, int t, lds_bytes* L, const_u32* xc, int kp,
                                         float* red) {
#pragma unroll
    for (int k = 0; k < NB; ++k) {
        // issue the reads of the next block: block k+1 of this item or block 0 of the next
        uint32_t lo, hi;
        if (k + 1 < NB) {
            if (k == 0) block_word<1>(cw, lo, hi);
            else if (k == 1) block_word<2>(cw, lo, hi);
            else block_word<3>(cw, lo, hi);
        } else {
            block_word<0>(nw, lo, hi);
        }
        const int ncol = k + 1 < NB ? col0 + k + 1 : ncol0;
        const BlockFetch nxt = fetch_block(lo, hi, L);
        uint32_t xn[Pipe<B>::kStageX ? B : 1][12];
        load_x<B>(xn, xc, kp, ncol);
        __builtin_amdgcn_sched_barrier(0);
        // values and norm of the current block (its reads were waited for one block ago)
        uint32_t y[12];
        const uint32_t sa = block_values(st.cur, y);
        __builtin_amdgcn_sched_barrier(0);
        // one wait per block: the next block's reads and the previous block's scale
        __builtin_amdgcn_s_waitcnt(0xC07F);
        finish_pending<B>(st, red);
        st.ps = *(lds_f32*)(L + kScaleOff + sa);
#pragma unroll
        for (int bb = 0; bb < B; ++bb) {
            float dt = 0.f;
#pragma unroll
            for (int q = 0; q < 12; ++q) {
                uint32_t xv;
                if constexpr (Pipe<B>::kStageX) xv = st.x[bb][q];
                else xv = xc[bb * kp + 12 * (col0 + k) + q];
                dt = dot2(y[q], xv, dt);
            }
            asm volatile("" : : "v"(dt));      // computed here, not sunk into the next block
            st.pdt[bb] = dt;
        }
        st.pend_t = t;
        __builtin_amdgcn_sched_barrier(0);
        st.cur = nxt;
        if constexpr (Pipe<B>::kStageX) {
#pragma unroll
            for (int bb = 0; bb < B; ++bb)
#pragma unroll
                for (int q = 0; q < 12; ++q) st.x[bb][q] = xn[bb][q];
        }
    }
}

template <int B>
__global__ __launch_bounds__(kGemvThreads) __attribute__((amdgpu_waves_per_eu(B <= 2 ? 8 : 4)))
void gemv_kernel(const GemvGroup grp) {
    constexpr int S = red_slots(B);
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    __shared__ float s_red[kGemvWaves * S * 64];     // [wave][slot][64]
    stage_packed_tables(s_tab);
    lds_bytes* L = (lds_bytes*)(s_tab);

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int G = gridDim.x;
    __syncthreads();

    for (int kr = 0;; ++kr) {
        const int r = kr * G + ((kr & 1) ? G - 1 - static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x));
        if (r >= grp.total_rounds) break;                  // uniform over the workgroup
        int pi = 0;
        while (pi + 1 < grp.n && r >= grp.prob[pi + 1].round_begin) ++pi;
        const GemvProblem& P = grp.prob[pi];
        const int tile0 = (r - P.round_begin) * P.round_tiles;
        const int ntr = min(P.round_tiles, P.tiles - tile0);
        const int nblk = P.nblk;
        const int ng = nblk / tetra::kGroupCols;
        const int rem = nblk - ng * tetra::kGroupCols;
        const int per_tile = ng + (rem > 0 ? 1 : 0);
        const size_t tile_bytes = static_cast<size_t>(nblk) * kChunk;
        const uint8_t* tb0 = P.codes + static_cast<size_t>(tile0) * tile_bytes;
        const_u32* xc = (const_u32*)(P.x);
        const int kp = P.K >> 1;
        float* red = s_red + wave * S * 64 + lane;

        // this wave's slots start at zero: tiles it gets no item of stay zero
#pragma unroll
        for (int q = 0; q < S; ++q) red[q * 64] = 0.f;

        auto load_item = [&](int t, int j) {
            ItemWords w;
            const uint8_t* tb = tb0 + static_cast<size_t>(t) * tile_bytes;
            if (j < ng) {
                const uint8_t* gp = tb + static_cast<size_t>(j) * tetra::kGroupBytes;
                w.lo = *reinterpret_cast<const uint4*>(gp + 16 * lane);
                w.hi = *reinterpret_cast<const uint2*>(gp + 1024 + 8 * lane);
            } else {
                // the nblk mod 4 single columns, 384-byte runs
                const uint8_t* sp = tb + static_cast<size_t>(ng) * tetra::kGroupBytes;
                w.lo = make_uint4(0, 0, 0, 0);
                w.lo.x = *reinterpret_cast<const uint32_t*>(sp + 4 * lane);
                uint32_t h0 = *reinterpret_cast<const uint16_t*>(sp + 256 + 2 * lane), h1 = 0, h2 = 0;
                if (rem > 1) {
                    w.lo.y = *reinterpret_cast<const uint32_t*>(sp + kChunk + 4 * lane);
                    h1 = *reinterpret_cast<const uint16_t*>(sp + kChunk + 256 + 2 * lane);
                }
                if (rem > 2) {
                    w.lo.z = *reinterpret_cast<const uint32_t*>(sp + 2 * kChunk + 4 * lane);
                    h2 = *reinterpret_cast<const uint16_t*>(sp + 2 * kChunk + 256 + 2 * lane);
                }
                w.hi = make_uint2(h0 | h1 << 16, h2);
            }
            return w;
        };
        auto advance = [&](int& t, int& j) {
            while (j >= per_tile && t < ntr) { j -= per_tile; ++t; }
        };
        auto first_col = [&](int j) { return j < ng ? 4 * j : 4 * ng; };

        int t = 0, j = wave;
        advance(t, j);
        if (t < ntr) {
            Pipe<B> st;
            ItemWords cw = load_item(t, j);
            int nt = t, nj = j + kGemvWaves;
            advance(nt, nj);
            bool more = nt < ntr;
            ItemWords nw = load_item(more ? nt : t, more ? nj : j);
            {
                uint32_t lo, hi;
                block_word<0>(cw, lo, hi);
                st.cur = fetch_block(lo, hi, L);
                load_x<B>(st.x, xc, kp, first_col(j));
                __builtin_amdgcn_s_waitcnt(0xC07F);
            }
#pragma unroll
            for (int bb = 0; bb < B; ++bb) st.acc[bb] = st.pdt[bb] = 0.f;
            st.ps = 0.f;
            st.pend_t = -1;
            st.acc_t = t;
            for (;;) {
                const int ncol0 = first_col(more ? nj : j);
                if (j < ng) {
                    run_item<B, 4>(st, cw, nw, 4 * j, ncol0, t, L, xc, kp, red);
                } else if (rem == 1) {
                    run_item<B, 1>(st, cw, nw, 4 * ng, ncol0, t, L, xc, kp, red);
                } else if (rem == 2) {
                    run_item<B, 2>(st, cw, nw, 4 * ng, ncol0, t, L, xc, kp, red);
                } else {
                    run_item<B, 3>(st, cw, nw, 4 * ng, ncol0, t, L, xc, kp, red);
                }
                if (!more) break;
                t = nt;
                j = nj;
                cw = nw;
                nt = t;
                nj = j + kGemvWaves;
                advance(nt, nj);
                more = nt < ntr;
                nw = load_item(more ? nt : t, more ? nj : j);
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            finish_pending<B>(st, red);
#pragma unroll
            for (int bb = 0; bb < B; ++bb) red[(st.acc_t * B + bb) * 64] = st.acc[bb];
        }
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
                    tot += s_red[((w * S) + tt * B + bb) * 64 + lane];
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
