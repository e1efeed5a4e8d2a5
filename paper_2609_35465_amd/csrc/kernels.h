// HIP kernels for gfx950: bulk decode, dense reconstruction, fused GEMV.
// Included once, by tetra.hip.
#pragma once

#include <hip/hip_runtime.h>

#include "device_tables.h"
#include "word_format.h"

namespace tetra_dev {

constexpr int kTile = 64;                 // rows per code tile = lanes per wave
constexpr int kChunk = kTile * 6;         // bytes per (tile, block column) chunk
constexpr int kGemvWaves = 12;                 // waves per GEMV workgroup
constexpr int kGemvThreads = kGemvWaves * 64;
constexpr int kGemvGroupsPerCU = 2;            // at most (batch 1: 2 x 56.5 KB of LDS, 6 waves per SIMD)
constexpr int kMaxGroup = 32;

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(4))) const uint32_t const_u32;

__device__ __forceinline__ float f16(uint16_t v) {
    return static_cast<float>(__builtin_bit_cast(_Float16, v));
}

// fp16 bits of a float, round to nearest even
__device__ __forceinline__ uint16_t f16_bits(float v) {
    return __builtin_bit_cast(uint16_t, static_cast<_Float16>(v));
}

// the lane index, computed afresh at each use: the cold paths of the GEMV
// (tile tails, single columns, piece reduction) take their lane addresses
// from it, so that none of them is hoisted and kept live across the hot loop
__device__ __forceinline__ int lane_now() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
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
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
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
// 16-31 are ignored).  Cost: also the three rows' costs (cost, their sum of
// U^2), one byte each.
template <bool Cost = false>
__device__ __forceinline__ BlockFetch fetch_block(uint32_t lo, uint32_t hi, lds_bytes* L, uint32_t* cost = nullptr) {
    const uint32_t a_path = (lo << 2) & 0x3FFCu;                      // 4 * path
    // i2, am and phys1 are kept opaque, so that each address is one shift
    // (and add) of the field the cost read uses too, rather than a shift and
    // a mask of the word of its own
    uint32_t i2 = __builtin_amdgcn_alignbit(hi, lo, 25) & 0x7FFu;
    asm("" : "+v"(i2));
    uint32_t am = i2 * 8u + 8u * tetra::kMidOffset;                   // 8 * (808 + i2), bit 14 = delta
    asm("" : "+v"(am));
    uint32_t a1;                                                      // 8 * phys1
    uint32_t phys1 = 0;
    if constexpr (Cost) {
        phys1 = (lo >> 13) & 0xFFFu;
        asm("" : "+v"(phys1));
        a1 = phys1 << 3;
    } else {
        a1 = (lo >> 10) & 0x7FF8u;
    }
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
    if constexpr (Cost) {
        cost[0] = L[kCostOff + phys1];
        cost[1] = L[kCostOff + tetra::kMidOffset + i2];
        cost[2] = L[kCostOff + (a3 >> 3)];
    }
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

// Decoder tables into LDS: all loads first, then all stores, so that a
// workgroup pays one memory round trip (NT: threads of the workgroup).  The
// loads and stores are unconditional, so that none is sunk into a branch: a
// thread past the end loads and stores the last word again.  The staged
// words are one vector rather than an array of uint4, which the compiler
// may place in scratch memory when other loads are in flight beside it.
template <int NT>
struct TableStage {
    static constexpr int kN = static_cast<int>(kPackedTableBytes / 16);
    static constexpr int kPer = (kN + NT - 1) / NT;
    typedef uint32_t vec_t __attribute__((ext_vector_type(4 * kPer)));
    vec_t v;
    __device__ __forceinline__ void load() {
        const uint4* src = reinterpret_cast<const uint4*>(&g_packed);
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const uint4 t = src[min(static_cast<int>(threadIdx.x) + k * NT, kN - 1)];
            v[4 * k] = t.x;
            v[4 * k + 1] = t.y;
            v[4 * k + 2] = t.z;
            v[4 * k + 3] = t.w;
        }
    }
    __device__ __forceinline__ void store(uint4* dst) const {
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            dst[min(static_cast<int>(threadIdx.x) + k * NT, kN - 1)] = make_uint4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3]);
    }
};

template <int NT>
__device__ __forceinline__ void stage_packed_tables(uint4* dst) {
    TableStage<NT> ts;
    ts.load();
    ts.store(dst);
}

__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* __restrict__ codes,
                                                      const uint16_t* __restrict__ sigma, int M,
                                                      int K, int nblk, int T, size_t tail_off,
                                                      float* __restrict__ w_out) {
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    stage_packed_tables<256>(s_tab);
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
// One lane per output row (64-row tiles).  The blocks of all matrices of a
// launch form one sequence (matrix by matrix, tile by tile, block column by
// block column), and wave w of the W waves of the launch takes the
// contiguous range [floor(w Tot / W), floor((w+1) Tot / W)): every wave gets
// the same number of blocks to within one, whatever the shapes.  A range
// covers whole tiles and at most two pieces of tiles.  A whole tile is
// finished by its wave (row scale, unquantised tail, store of y).  The
// pieces of a tile are combined in two levels (gemv_kernel): in LDS among
// the waves of a workgroup, then through the per-device workspace among
// workgroups, each time by the last to count in, in a fixed order.  The
// ranges depend only on the shapes and W, never on timing, so the result is
// deterministic.  W depends on the batch only through the kernel's
// residency (gemv_waves): row b of a batch-B product is bit for bit the row
// of x_b at any batch size with the same residency.
//
// Inside its range a wave runs the blocks as a pipeline: the table reads and
// activation loads of the next block are issued before the current block's
// arithmetic, the current block's scale read is consumed one block later,
// and the code words of whole groups of four columns are loaded one group
// ahead, so a wave waits at most once per block; a tile's trailing columns
// run after the groups (run_piece).  The activation pairs of a block column
// are the same for all lanes and come through the scalar unit as SGPR
// operands of v_dot2_f32_f16.

struct GemvProblem {
    const uint8_t* codes;
    const uint16_t* sigma;
    const uint16_t* x;
    float* y;
    unsigned long long tail_off;
    uint32_t blk_base;             // index of the matrix's first block in the launch sequence
    int M, K, nblk, T;
    int tiles, ng, rem;
};

// The even split of one phase's block sequence (its problems, matrix by
// matrix, tile by tile, block column by block column) over its waves.
struct GemvSplit {
    double inv_total, inv_waves;   // 1 / total, 1 / waves
    uint32_t total;                // blocks in the phase (< 2^31)
    int waves;                     // waves that take a range
    int wpg;                       // of them per workgroup: wave v is wave v mod wpg of workgroup v / wpg
    int p0, n;                     // its problems: prob[p0 .. p0 + n - 1]
    int aligned;                   // 1: tile-aligned split (below), 0: even split of the block sequence
    int defer;                     // tiles that span workgroups are added up after the next barrier:
                                   // 1, their sums complete before it; 2, before the one after
                                   // (below); 0: not deferred
};

constexpr int kMaxPhases = 16;
constexpr int kChainTimeout = -6;   // TETRA_ETIMEOUT

// One launch: phases run in order, each split over the launch's waves; a
// wave starts phase k + 1 only after every workgroup of the launch has
// finished phase k (the chain barrier below).  A single-phase launch is a
// plain (grouped) product.
struct GemvChain {
    GemvProblem prob[kMaxGroup];   // blk_base counts from the start of the problem's phase
    GemvSplit ph[kMaxPhases];
    int n_phases;
    int buffers;                   // partial-sum buffers the phases rotate over: 1, or kChainBuffers
    int slot;                      // workspace slot of the launch (g_gemv_slots, g_chain_sync)
    uint32_t wait_limit;           // polls before a chain barrier wait gives up
    int* status;                   // device word for the launch's status, or null
};

// GEMV workspaces: a counter and two partial sums per workgroup.  One slot
// per stream that issues GEMV calls on a device, so that calls on different
// streams never share one; static device memory, zero when the code object
// loads, and every launch leaves its counters at zero again.  A slot covers
// kGemvMaxGroups workgroups, and its partial sums [groups][2][B][64] the
// largest batch at one workgroup per CU or batch 2 at two; for a chain, three
// such buffers (below) up to batch 5 at one workgroup per CU and batch 2 at
// two (1.9 MB per slot).
constexpr int kGemvSlots = 16;
constexpr int kGemvMaxCUs = 320;
constexpr int kGemvMaxGroups = kGemvMaxCUs * kGemvGroupsPerCU;
constexpr int kGemvSlotPartials = 3 * kGemvMaxCUs * 2 * 4 * 64 > kGemvMaxCUs * 2 * 8 * 64
                                      ? 3 * kGemvMaxCUs * 2 * 4 * 64
                                      : kGemvMaxCUs * 2 * 8 * 64;

struct GemvSlot {
    uint32_t counters[kGemvMaxGroups];
    float partials[kGemvSlotPartials];
};

__device__ GemvSlot g_gemv_slots[kGemvSlots];

// Words of the chain barrier of a slot.  The workgroups of a launch form
// kBarrierGroups groups (blockIdx mod 8); a workgroup done with phase k
// counts itself into its group's counter (a 128-byte line of its own), and
// the last of a group writes k + 1 into word q of every group's arrival
// line, where q is its group.  A group's workgroups poll their own arrival
// line with one vector load (a lane per word) until every group's word
// reads k + 1: the barrier's critical path is one atomic round trip, the
// stores and one poll, with no second-level counter between them.
// Spreading the arrivals over several counters keeps them from queueing on
// one address (with 512 workgroups, one counter for all made the decode
// step 15-18 % slower; 4, 8, 16 and 32 groups: 1.949-1.960, 1.950-1.969,
// 1.970-1.974 and 2.12 ms, the last with a whole line per poll).  All
// words are touched only with device-scope atomics.  Counts and arrival
// words grow within a launch; the last workgroup to finish the launch puts
// them back to zero.
constexpr int kBarrierGroups = 8;
static_assert((kBarrierGroups & (kBarrierGroups - 1)) == 0, "a power of two");
struct ChainSync {
    uint32_t grp[kBarrierGroups][32];
    uint32_t arrived[kBarrierGroups][32];   // line h: word q = phases group q has finished
    uint32_t exit[32];             // workgroups finished
    uint32_t expired[32];          // waits that gave up
};

__device__ ChainSync g_chain_sync[kGemvSlots];

__device__ __forceinline__ uint32_t dev_load(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t dev_add(uint32_t* p, uint32_t v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void dev_store(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// workgroup `wg` of `nwg` is done with phase k (one thread per workgroup)
__device__ __forceinline__ void chain_arrive(ChainSync& cs, int k, int wg, int nwg) {
    constexpr uint32_t G = kBarrierGroups;
    const uint32_t q = static_cast<uint32_t>(wg) % G;
    const uint32_t groups = static_cast<uint32_t>(nwg) < G ? static_cast<uint32_t>(nwg) : G;
    const uint32_t per = static_cast<uint32_t>(nwg) / G + (static_cast<uint32_t>(nwg) % G > q ? 1u : 0u);
    const uint32_t target = static_cast<uint32_t>(k) + 1u;
    if (dev_add(&cs.grp[q][0], 1u) + 1u == target * per)
        for (uint32_t h = 0; h < groups; ++h) dev_store(&cs.arrived[h][q], target);
}

// waits until every workgroup is done with phase k; false when it gave up
// after `limit` polls.  Run by all 64 lanes of one wave: lane l reads word
// l mod kBarrierGroups of the workgroup's arrival line (word 0 past the
// launch's groups).
__device__ __forceinline__ bool chain_wait(const ChainSync& cs, int k, int wg, int nwg, uint32_t limit) {
    const uint32_t q = static_cast<uint32_t>(wg) % kBarrierGroups;
    const uint32_t l = static_cast<uint32_t>(lane_now()) & (kBarrierGroups - 1);
    const uint32_t h = l < static_cast<uint32_t>(nwg) ? l : 0u;
    const uint32_t target = static_cast<uint32_t>(k) + 1u;
    for (uint32_t n = 0;;) {
        const bool behind = dev_load(&cs.arrived[q][h]) < target;
        if (__builtin_amdgcn_ballot_w64(behind) == 0) return true;
        __builtin_amdgcn_s_sleep(1);
        if (++n > limit) return false;
    }
}

// wave count of a single-phase launch: one round of the 768-thread
// workgroups a CU holds at once (`groups`: two at batch 1 and 2; one from
// batch 3 on, whose registers allow 12 waves per CU), fewer when the launch
// is small, so that each wave takes at least kGemvMinBlocks blocks (a wave's
// fixed cost, table staging and its share of the piece reduction, is worth
// several blocks of streaming; every range is non-empty).  A second round of
// workgroups would pay the launch start and the piece reduction twice.
constexpr uint32_t kGemvMinBlocks = 8;
inline int gemv_waves(uint32_t total, int cus, int groups) {
    const uint32_t cap = static_cast<uint32_t>(cus) * static_cast<uint32_t>(groups) * kGemvWaves;
    const uint32_t want = total / kGemvMinBlocks > 0 ? total / kGemvMinBlocks : 1u;
    return static_cast<int>(want < cap ? want : cap);
}

// Waves per workgroup in one phase of a chain: its launch holds a whole
// round of workgroups anyway, and the tables are staged once for all phases,
// so a wave is worth fewer blocks than in a single launch (at least
// kChainMinBlocks each, up to all kGemvWaves).  A multiple of the CU's four
// SIMDs, which take a workgroup's waves in turn: five waves would put two on
// one SIMD and one on each of the others, and that SIMD would take twice as
// long (measured on the 14B step: 2.44 -> 2.39 ms).
constexpr uint32_t kChainMinBlocks = 8;
constexpr int kSimdsPerCU = 4;
static_assert(kGemvWaves % kSimdsPerCU == 0, "whole rounds of SIMDs");
inline int chain_phase_wpg(uint32_t total, int groups) {
    const unsigned long long per = static_cast<unsigned long long>(kChainMinBlocks) * static_cast<uint32_t>(groups);
    const unsigned long long w = (total + per - 1) / per;
    const unsigned long long w4 = (w + kSimdsPerCU - 1) / kSimdsPerCU * kSimdsPerCU;
    return static_cast<int>(w4 > static_cast<unsigned long long>(kGemvWaves) ? kGemvWaves : w4);
}

// Partial-sum buffers of a chain whose phases defer (when three fit in the
// slot; otherwise every phase uses the one buffer and none defers): phase k
// writes buffer k mod 3.  A deferred phase's sums are read while the phase
// after it runs, and buffer k mod 3 is written again only by phase k + 3,
// which starts after every workgroup has arrived at the barrier that follows
// phase k + 1, and so after every read of phase k's sums.
constexpr int kChainBuffers = 3;

// largest workgroup count of a launch at batch B that the slot's partial
// sums hold
constexpr int gemv_max_groups(int B) {
    return kGemvSlotPartials / (2 * B * 64) < kGemvMaxGroups ? kGemvSlotPartials / (2 * B * 64) : kGemvMaxGroups;
}

// floor(n / d) for n < 2^53, from a reciprocal of d computed on the host
// (exact: the estimate is corrected by one in either direction)
__device__ __forceinline__ uint32_t div_exact(unsigned long long n, uint32_t d, double inv_d) {
    uint32_t q = static_cast<uint32_t>(static_cast<double>(n) * inv_d);
    const unsigned long long qd = static_cast<unsigned long long>(q) * d;
    if (qd > n) --q;
    else if (qd + d <= n) ++q;
    return q;
}

__device__ __forceinline__ uint32_t range_begin(int w, const GemvSplit& sp) {
    return div_exact(static_cast<unsigned long long>(sp.total) * static_cast<uint32_t>(w),
                     static_cast<uint32_t>(sp.waves), sp.inv_waves);
}

// the wave whose range holds block i: floor(((i + 1) W - 1) / total)
__device__ __forceinline__ int wave_of(uint32_t i, const GemvSplit& sp) {
    return static_cast<int>(div_exact(static_cast<unsigned long long>(i + 1) * static_cast<uint32_t>(sp.waves) - 1,
                                      sp.total, sp.inv_total));
}

// Tile-aligned split (when every tile can have a wave of its own): the
// waves are shared out over the tiles in proportion to their blocks, tile u
// (first block B_u) taking waves floor(B_u W / total) .. floor((B_u + nblk) W
// / total) - 1, and each tile's columns are split evenly over its waves.
// Every wave then holds one piece of one tile, so no wave waits for the
// reduction of one tile before it starts the next.  The first wave of the
// tile that starts at block t0:
__device__ __forceinline__ int tile_first_wave(uint32_t t0, const GemvSplit& sp) {
    return static_cast<int>(div_exact(static_cast<unsigned long long>(t0) * static_cast<uint32_t>(sp.waves),
                                      sp.total, sp.inv_total));
}


// code words of one item (a group of four block columns, or the nblk mod 4
// single columns of a tile): the 16-bit part of block k is in hi.x (k = 0,
// 1) or hi.y (k = 2, 3), low half for even k
struct ItemWords {
    uint4 lo;
    uint2 hi;
};

template <int K>
__device__ __forceinline__ void block_word(const ItemWords& w, uint32_t& lo, uint32_t& hi) {
    lo = K == 0 ? w.lo.x : K == 1 ? w.lo.y : K == 2 ? w.lo.z : w.lo.w;
    hi = K == 0 ? w.hi.x : K == 1 ? w.hi.x >> 16 : K == 2 ? w.hi.y : w.hi.y >> 16;
}

// per-wave pipeline state: the staged block and its activation pairs (batch
// 1), the previous block (scale read in flight, dot products), and the
// running sums of the current piece of a tile
template <int B>
struct Pipe {
    static constexpr bool kStageX = B == 1;
    BlockFetch cur;
    uint32_t x[kStageX ? B : 1][12];
    float ps;              // zero before the first block, so that adding the
    float pdt[B];          // "previous block" is a no-op there
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

template <int B>
__device__ __forceinline__ void finish_pending(Pipe<B>& st) {
#pragma unroll
    for (int bb = 0; bb < B; ++bb) st.acc[bb] = fmaf(st.ps, st.pdt[bb], st.acc[bb]);
}

// Blocks kb..ke-1 of one item (block k is column col0 + k), each one staging
// the next: block k+1 of this item, or block 0 of the next item (words nw,
// column ncol0; a repeat of this item at the end of a piece).  Full: the
// whole group of four.
template <int B, bool Full>
__device__ __forceinline__ void run_item(Pipe<B>& st, const ItemWords& cw, const ItemWords& nw, int col0,
                                         int ncol0, int kb, int ke, lds_bytes* L, const_u32* xc, int kp) {
    // batch > 1: one activation pointer per row for the item, so that the
    // block and word offsets go into the loads' immediate offsets instead of
    // one 64-bit address per block and row (which spilled into lanes of VGPRs)
    const_u32* xb[Pipe<B>::kStageX ? 1 : B];
    if constexpr (!Pipe<B>::kStageX) {
#pragma unroll
        for (int bb = 0; bb < B; ++bb) xb[bb] = xc + (bb * kp + 12 * col0);
    }
#pragma unroll
    for (int k = 0; k < tetra::kGroupCols; ++k) {
        if (Full || (k >= kb && k < ke)) {
            uint32_t lo, hi;
            int ncol;
            BlockFetch nxt;
            if (k + 1 < tetra::kGroupCols && (Full || k + 1 < ke)) {
                if (k == 0) block_word<1>(cw, lo, hi);
                else if (k == 1) block_word<2>(cw, lo, hi);
                else block_word<3>(cw, lo, hi);
                ncol = col0 + k + 1;
            } else {
                block_word<0>(nw, lo, hi);
                ncol = ncol0;
            }
            nxt = fetch_block(lo, hi, L);
            uint32_t xn[Pipe<B>::kStageX ? B : 1][12];
            load_x<B>(xn, xc, kp, ncol);
            // batch > 1: this block's activations, requested here so that the
            // scalar loads (often scalar-cache misses: B rows of x pass
            // through the cache) are in flight during the decode below; a
            // second set, one block ahead as at batch 1, would not fit in the
            // scalar registers
            uint32_t xk[Pipe<B>::kStageX ? 1 : B][12];
            if constexpr (!Pipe<B>::kStageX) {
#pragma unroll
                for (int bb = 0; bb < B; ++bb)
#pragma unroll
                    for (int q = 0; q < 12; ++q) xk[bb][q] = xb[bb][12 * k + q];
            }
            __builtin_amdgcn_sched_barrier(0);
            // values and norm of the current block (its reads were waited for one block ago)
            uint32_t y[12];
            const uint32_t sa = block_values(st.cur, y);
            __builtin_amdgcn_sched_barrier(0);
            // one wait per block: the next block's reads and the previous block's scale
            __builtin_amdgcn_s_waitcnt(0xC07F);
            finish_pending<B>(st);
            st.ps = *(lds_f32*)(L + kScaleOff + sa);
#pragma unroll
            for (int bb = 0; bb < B; ++bb) {
                float dt = 0.f;
#pragma unroll
                for (int q = 0; q < 12; ++q) {
                    uint32_t xv;
                    if constexpr (Pipe<B>::kStageX) xv = st.x[bb][q];
                    else xv = xk[bb][q];
                    dt = dot2(y[q], xv, dt);
                }
                asm volatile("" : : "v"(dt));      // computed here, not sunk into the next block
                st.pdt[bb] = dt;
            }
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
}

// code words of group j of a tile (four columns)
__device__ __forceinline__ ItemWords load_group(const uint8_t* tb, int j, int lane) {
    ItemWords w;
    const uint8_t* gp = tb + static_cast<size_t>(j) * tetra::kGroupBytes;
    w.lo = *reinterpret_cast<const uint4*>(gp + 16u * static_cast<uint32_t>(lane));
    w.hi = *reinterpret_cast<const uint2*>(gp + 1024u + 8u * static_cast<uint32_t>(lane));
    return w;
}

// code words of the rem = nblk mod 4 trailing columns of a tile (rem > 0),
// with the same five 4-byte loads whatever rem is (no branch, so that the
// loads never wait for one another): the 32-bit parts of columns
// min(k, rem - 1), and the 4-byte words that hold the 16-bit parts.  Where a
// 16-bit part shares its word with the neighbouring row's (rem = 1, and the
// third column of rem = 3), hi_shift tells how far to shift it down; the
// shift is applied when the words are used (trailing_fixup).
__device__ __forceinline__ ItemWords load_trailing(const uint8_t* tb, int ng, int rem) {
    const uint8_t* sp = tb + static_cast<size_t>(ng) * tetra::kGroupBytes;
    const int lane = lane_now();
    const uint32_t* lo = reinterpret_cast<const uint32_t*>(sp + 4 * rem * lane);
    const int h01 = rem == 1 ? 256 + 4 * (lane >> 1) : 256 * rem + 4 * lane;
    const int h2 = rem == 3 ? 1024 + 4 * (lane >> 1) : h01;
    ItemWords w;
    w.lo.x = lo[0];
    w.lo.y = lo[min(1, rem - 1)];
    w.lo.z = lo[min(2, rem - 1)];
    w.hi.x = *reinterpret_cast<const uint32_t*>(sp + h01);
    w.hi.y = *reinterpret_cast<const uint32_t*>(sp + h2);
    return w;
}

// the 16-bit parts of the trailing columns in place (see load_trailing)
__device__ __forceinline__ void trailing_fixup(ItemWords& w, int rem) {
    const uint32_t odd = (lane_now() & 1) ? 16u : 0u;
    if (rem == 1) w.hi.x >>= odd;
    w.hi.y >>= odd;            // only used when rem = 3
}

// A piece of a tile: block columns c0..c1-1 of tile t, in groups j..jg and,
// when the piece reaches them (tr), the trailing columns.  begin_piece issues
// the loads of its first two groups and of its trailing columns, so that all
// of them are in flight together; run_piece sums the piece for the wave's 64
// rows, the trailing columns after the groups, from their own registers (in
// the group pipeline, their loads would make it wait).
struct Piece {
    ItemWords cw, nw, tw;
    int t, c0, c1, j, jg;
    bool tr;
};

__device__ __forceinline__ Piece begin_piece(const GemvProblem& P, int t, int c0, int c1, int lane) {
    Piece pc;
    pc.t = t;
    pc.c0 = c0;
    pc.c1 = c1;
    pc.j = c0 >> 2;                                  // ng when the piece starts in the trailing columns
    pc.jg = min((c1 - 1) >> 2, P.ng - 1);            // last group of the piece (< j: none)
    pc.tr = c1 > 4 * P.ng;
    const uint8_t* tb = P.codes + static_cast<size_t>(t) * P.nblk * kChunk;
    if (pc.j <= pc.jg) {
        pc.cw = load_group(tb, pc.j, lane);
        pc.nw = load_group(tb, min(pc.j + 1, pc.jg), lane);
    }
    if (pc.tr) pc.tw = load_trailing(tb, P.ng, P.rem);
    return pc;
}

// 2 KB of zeros: the loads of a wave with no piece, or of a piece with no
// group (or no trailing columns), read here, so that they need no branch.
// Every offset load_group and load_trailing use is below 1536.
__device__ __align__(16) uint8_t g_zero_codes[2048];

// begin_piece for the first piece of a wave, with every load unconditional:
// the loads are issued between the table loads and the table stores, and a
// branch around them would make the stores wait for them too (the wait
// counter is not tracked across a join).  `live` is false for a wave past
// the last; its words are then never used.
__device__ __forceinline__ Piece begin_piece_live(const GemvProblem& P, int t, int c0, int c1, int lane, bool live) {
    Piece pc;
    pc.t = t;
    pc.c0 = c0;
    pc.c1 = c1;
    pc.j = c0 >> 2;
    pc.jg = min((c1 - 1) >> 2, P.ng - 1);
    pc.tr = c1 > 4 * P.ng;
    const uint8_t* tb = P.codes + static_cast<size_t>(t) * P.nblk * kChunk;
    const bool gok = live && pc.j <= pc.jg;
    const uint8_t* gb = gok ? tb : g_zero_codes;
    pc.cw = load_group(gb, gok ? pc.j : 0, lane);
    pc.nw = load_group(gb, gok ? min(pc.j + 1, pc.jg) : 0, lane);
    const bool tok = live && pc.tr;
    pc.tw = load_trailing(tok ? tb : g_zero_codes, tok ? P.ng : 0, tok ? P.rem : 1);
    return pc;
}

// blocks kb..ke-1 of item j (words cw; the next item's words nw, column
// ncol0), whole group or not
template <int B>
__device__ __forceinline__ void run_one_item(Pipe<B>& st, int kb, int ke, int col0, int ncol0,
                                             const ItemWords& cw, const ItemWords& nw, lds_bytes* L,
                                             const_u32* xc, int kp) {
    if (kb == 0 && ke == tetra::kGroupCols)
        run_item<B, true>(st, cw, nw, col0, ncol0, 0, tetra::kGroupCols, L, xc, kp);
    else
        run_item<B, false>(st, cw, nw, col0, ncol0, kb, ke, L, xc, kp);
}

// first block of a run of items: its table reads and activations, and an
// empty "previous block"
template <int B>
__device__ __forceinline__ void start_pipe(Pipe<B>& st, const ItemWords& w, int kb, int col, lds_bytes* L,
                                           const_u32* xc, int kp) {
    uint32_t lo, hi;
    if (kb == 0) block_word<0>(w, lo, hi);
    else if (kb == 1) block_word<1>(w, lo, hi);
    else if (kb == 2) block_word<2>(w, lo, hi);
    else block_word<3>(w, lo, hi);
    st.cur = fetch_block(lo, hi, L);
    load_x<B>(st.x, xc, kp, col);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    st.ps = 0.f;
#pragma unroll
    for (int bb = 0; bb < B; ++bb) st.pdt[bb] = 0.f;
}

// Issue priority from the share of a piece still to do (left of total
// groups): 3 above three quarters, down to 0 below one quarter.  A SIMD
// issues for the oldest of its ready waves first, so with equal pieces the
// first waves of a CU would finish long before the last ones, and the last
// ones would then run with too few waves beside them to hide their waits;
// a wave that has fallen behind now goes first.
__device__ __forceinline__ void progress_prio(int left, int total) {
    if (4 * left >= 3 * total) __builtin_amdgcn_s_setprio(3);
    else if (2 * left >= total) __builtin_amdgcn_s_setprio(2);
    else if (4 * left >= total) __builtin_amdgcn_s_setprio(1);
    else __builtin_amdgcn_s_setprio(0);
}

// The groups alternate between two sets of word registers, so that the
// loads of the group after next go straight into the registers just freed;
// the trailing columns follow from their own registers.
template <int B>
__device__ __forceinline__ void run_piece(const GemvProblem& P, Piece& pc, lds_bytes* L, float (&out)[B]) {
    const int lane = threadIdx.x & 63;
    const uint8_t* tb = P.codes + static_cast<size_t>(pc.t) * P.nblk * kChunk;
    const_u32* xc = (const_u32*)(P.x);
    const int kp = P.K >> 1;
    const int jg = pc.jg;
    int j = pc.j;
    int kb = pc.c0 - 4 * j;
    Pipe<B> st;
#pragma unroll
    for (int bb = 0; bb < B; ++bb) st.acc[bb] = 0.f;
    if (j <= jg) {
        // the last group ends the piece unless the trailing columns follow
        const int kl = __builtin_amdgcn_readfirstlane(pc.tr ? tetra::kGroupCols : pc.c1 - 4 * jg);
        start_pipe<B>(st, pc.cw, kb, pc.c0, L, xc, kp);
        ItemWords wa = pc.cw, wb = pc.nw;
        const int j0 = j, ngr = jg - j + 1;
        __builtin_amdgcn_s_setprio(3);
        for (;;) {
            run_one_item<B>(st, kb, j == jg ? kl : tetra::kGroupCols, 4 * j, 4 * min(j + 1, jg), wa, wb, L, xc, kp);
            if (j == jg) break;
            ++j;
            progress_prio(jg - j + 1, ngr);
            kb = 0;
            wa = load_group(tb, min(j + 1, jg), lane);
            run_one_item<B>(st, 0, j == jg ? kl : tetra::kGroupCols, 4 * j, 4 * min(j + 1, jg), wb, wa, L, xc, kp);
            if (j == jg) break;
            ++j;
            progress_prio(jg - j + 1, ngr);
            wb = load_group(tb, min(j + 1, jg), lane);
        }
        (void)j0;
        __builtin_amdgcn_s_waitcnt(0xC07F);
        finish_pending<B>(st);
        kb = 0;
    }
    if (pc.tr) {
        const int c = 4 * P.ng;
        ItemWords tw = pc.tw;
        trailing_fixup(tw, P.rem);
        start_pipe<B>(st, tw, kb, c + kb, L, xc, kp);
        run_item<B, false>(st, tw, tw, c, c, kb, pc.c1 - c, L, xc, kp);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        finish_pending<B>(st);
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int bb = 0; bb < B; ++bb) out[bb] = st.acc[bb];
}

// ------------------------------------------------ batch 3..8: matrix cores
//
// At batch B >= 3 the product of a block column is a small dense contraction
// (64 rows x 24 weights by 24 x B activations), and it goes to the matrix
// cores: v_mfma_f32_4x4x4f16 multiplies, in 16 blocks of four lanes, a 4 x 4
// fp16 operand held one row per lane by a 4 x 4 operand held one column per
// lane.  The A operand is the block's decoded values as the lane already
// holds them (lane = row, coordinates 4c..4c+3 in y[2c], y[2c+1]), the B
// operand four rows of x (lane 4i + j holds x_j), so six instructions give
// the block's dot products for four batch rows; a second set of six covers
// rows 4..7.  The result sits in lane 4i + j, register r: row 4i + r, batch
// row j.  Each row's block scale comes to the four lanes of its quad by a
// DPP quad broadcast, so the sums take four fused multiply-adds per block
// and set, where the VALU dot product took 12 per batch row.  Batches 1 and
// 2 keep the VALU dot product of run_item: at batch 2 its registers leave
// room for two workgroups per CU, which this path's do not (measured on a
// 14B decode step: the VALU path is 3 % faster at batch 2, this one 9 % at
// batch 3, 16 % at 4 and 48 % at 8).
//
// The activations of a group of four block columns pass through a 1 KB LDS
// slot per wave and set (MxSets::kRow bytes per block column and batch row,
// 48 of them used): one 16-byte load per lane, requested a group ahead
// together with the group's code words (so that waiting for it never waits
// for later code words), written at the group's start, and read back per
// block as three broadcast ds_read_b128 per lane (four distinct addresses
// per wave, 48 or 64 bytes apart: no bank conflict).  Every output column is
// computed by the same instructions whatever the other columns hold, so row
// b of a batch-B product (3 <= B <= 8) is the same bit for bit at every such
// B.

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_a4 __attribute__((ext_vector_type(4), aligned(4)));

constexpr int kXSlotBytes = 1024;      // per wave and set of four batch rows: x of four block columns, or the 4 x 64 sums

// kRow: bytes per block column and batch row in a slot.  With one set (batch
// 3-4) a row takes 64 bytes, so that a lane's segment follows from its index
// by shifts; with two sets (batch 5-8) rows are packed at 48 bytes (measured
// 6 % faster at batch 8, where the registers are at their limit).
template <int B>
struct MxSets {
    static constexpr int kN = (B + 3) / 4;
    static constexpr int kRow = kN == 1 ? 64 : 48;
    static constexpr int kBlock = 4 * kRow;
};

// one group's activations for every set of four batch rows, one 16-byte
// segment per lane (x_segment)
template <int B>
struct XGroup {
    u32x4 v[MxSets<B>::kN];
};

struct XSeg {
    int r, k, part;
};

// 64-byte rows: lane l holds part l & 3 of block column (l >> 2) & 3 of
// row l >> 4 (part 3 repeats part 2: a block row is 48 bytes).  48-byte rows:
// segment m = l mod 48 is part m mod 3 of block column (m mod 12) / 3 of row
// m / 12 (lanes 48-63 repeat lanes 0-15).
template <int B>
__device__ __forceinline__ XSeg x_segment() {
    const int l = lane_now();
    XSeg s;
    if constexpr (MxSets<B>::kRow == 64) {
        s.r = l >> 4;
        s.k = (l >> 2) & 3;
        s.part = l & 3;
    } else {
        const int m = l >= 48 ? l - 48 : l;
        s.r = m / 12;
        s.k = (m - 12 * s.r) / 3;
        s.part = m - 12 * s.r - 3 * s.k;
    }
    return s;
}

// activations of block columns 4j..4j+3 (clamped to the last block column;
// rows past the batch read the last row: their products are never used)
template <int B>
__device__ __forceinline__ XGroup<B> load_xgroup(const GemvProblem& P, int j) {
    const XSeg sg = x_segment<B>();
    const int col = min(4 * j + sg.k, P.nblk - 1);
    const uint8_t* xb = reinterpret_cast<const uint8_t*>(P.x) + 48 * col + 16 * min(sg.part, 2);
    XGroup<B> g;
#pragma unroll
    for (int s = 0; s < MxSets<B>::kN; ++s) {
        const int row = min(4 * s + sg.r, B - 1);
        g.v[s] = *reinterpret_cast<const u32x4_a4*>(xb + static_cast<size_t>(row) * P.K * 2);
    }
    return g;
}

// the activation load of a piece's first group (its trailing columns when
// it starts there), unconditional: a wave with no piece (live false) reads
// group 0
template <int B>
__device__ __forceinline__ XGroup<B> begin_xpiece(const GemvProblem& P, const Piece& pc, bool live) {
    return load_xgroup<B>(P, live ? pc.j : 0);
}

// xs: the wave's slots
template <int B>
__device__ __forceinline__ void write_xgroup(uint8_t* xs, const XGroup<B>& g) {
    const XSeg sg = x_segment<B>();
    const int off = sg.k * MxSets<B>::kBlock + sg.r * MxSets<B>::kRow + sg.part * 16;
#pragma unroll
    for (int s = 0; s < MxSets<B>::kN; ++s) *reinterpret_cast<u32x4*>(xs + s * kXSlotBytes + off) = g.v[s];
}

__device__ __forceinline__ half4_t as_half4(uint32_t a, uint32_t b) {
    const u32x2 v = {a, b};
    return __builtin_bit_cast(half4_t, v);
}

template <int I>
__device__ __forceinline__ float quad_bcast(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x55 * I, 0xF, 0xF, false));
}

template <int B>
struct MxPipe {
    BlockFetch cur;
    float ps;                          // scale of the previous block (zero before the first)
    f32x4 d[MxSets<B>::kN];            // products of the previous block
    f32x4 acc[MxSets<B>::kN];
};

template <int B>
__device__ __forceinline__ void mx_finish(MxPipe<B>& st) {
    const float p0 = quad_bcast<0>(st.ps), p1 = quad_bcast<1>(st.ps);
    const float p2 = quad_bcast<2>(st.ps), p3 = quad_bcast<3>(st.ps);
#pragma unroll
    for (int s = 0; s < MxSets<B>::kN; ++s) {
        st.acc[s].x = fmaf(p0, st.d[s].x, st.acc[s].x);
        st.acc[s].y = fmaf(p1, st.d[s].y, st.acc[s].y);
        st.acc[s].z = fmaf(p2, st.d[s].z, st.acc[s].z);
        st.acc[s].w = fmaf(p3, st.d[s].w, st.acc[s].w);
    }
}

// six products of a block for one set: y (A, this lane's row) by the three
// 16-byte reads of x (B)
__device__ __forceinline__ f32x4 mx_block(const uint32_t (&y)[12], u32x4 x0, u32x4 x1, u32x4 x2) {
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    f32x4 d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[0], y[1]), as_half4(x0.x, x0.y), z, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[2], y[3]), as_half4(x0.z, x0.w), d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[4], y[5]), as_half4(x1.x, x1.y), d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[6], y[7]), as_half4(x1.z, x1.w), d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[8], y[9]), as_half4(x2.x, x2.y), d, 0, 0, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(as_half4(y[10], y[11]), as_half4(x2.z, x2.w), d, 0, 0, 0);
    return d;
}

// Blocks kb..ke-1 of one item, as run_item; xr: the wave's slots plus kRow
// times the lane's batch row within a set (lane mod 4)
template <int B, bool Full>
__device__ __forceinline__ void run_item_mx(MxPipe<B>& st, const ItemWords& cw, const ItemWords& nw, int kb, int ke,
                                            lds_bytes* L, const uint8_t* xr) {
    constexpr int NS = MxSets<B>::kN;
#pragma unroll
    for (int k = 0; k < tetra::kGroupCols; ++k) {
        if (Full || (k >= kb && k < ke)) {
            uint32_t lo, hi;
            if (k + 1 < tetra::kGroupCols && (Full || k + 1 < ke)) {
                if (k == 0) block_word<1>(cw, lo, hi);
                else if (k == 1) block_word<2>(cw, lo, hi);
                else block_word<3>(cw, lo, hi);
            } else {
                block_word<0>(nw, lo, hi);
            }
            const BlockFetch nxt = fetch_block(lo, hi, L);
            u32x4 xv[NS][3];
#pragma unroll
            for (int s = 0; s < NS; ++s)
#pragma unroll
                for (int c = 0; c < 3; ++c)
                    xv[s][c] = *reinterpret_cast<const u32x4*>(xr + s * kXSlotBytes + k * MxSets<B>::kBlock + 16 * c);
            __builtin_amdgcn_sched_barrier(0);
            uint32_t y[12];
            const uint32_t sa = block_values(st.cur, y);
            __builtin_amdgcn_sched_barrier(0);
            // one wait per block: the next block's table reads, this block's
            // activations and the previous block's scale
            __builtin_amdgcn_s_waitcnt(0xC07F);
            mx_finish<B>(st);
            st.ps = *(lds_f32*)(L + kScaleOff + sa);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                st.d[s] = mx_block(y, xv[s][0], xv[s][1], xv[s][2]);
                asm volatile("" : : "v"(st.d[s]));     // computed here, not sunk into the next block
            }
            __builtin_amdgcn_sched_barrier(0);
            st.cur = nxt;
        }
    }
}

template <int B>
__device__ __forceinline__ void run_one_item_mx(MxPipe<B>& st, int kb, int ke, const ItemWords& cw,
                                                const ItemWords& nw, lds_bytes* L, const uint8_t* xr) {
    if (kb == 0 && ke == tetra::kGroupCols)
        run_item_mx<B, true>(st, cw, nw, 0, tetra::kGroupCols, L, xr);
    else
        run_item_mx<B, false>(st, cw, nw, kb, ke, L, xr);
}

template <int B>
__device__ __forceinline__ void start_pipe_mx(MxPipe<B>& st, const ItemWords& w, int kb, lds_bytes* L) {
    uint32_t lo, hi;
    if (kb == 0) block_word<0>(w, lo, hi);
    else if (kb == 1) block_word<1>(w, lo, hi);
    else if (kb == 2) block_word<2>(w, lo, hi);
    else block_word<3>(w, lo, hi);
    st.cur = fetch_block(lo, hi, L);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    st.ps = 0.f;
#pragma unroll
    for (int s = 0; s < MxSets<B>::kN; ++s) st.d[s] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// run_piece for 3 <= B <= 8.  xs: the wave's LDS slots (kXSlotBytes per
// set); the piece's sums come back one row per lane through the same slots.
template <int B>
__device__ __forceinline__ void run_piece_mx(const GemvProblem& P, Piece& pc, const XGroup<B>& xp, lds_bytes* L,
                                             uint8_t* xs, float (&out)[B]) {
    constexpr int NS = MxSets<B>::kN;
    const int lane = threadIdx.x & 63;
    const uint8_t* tb = P.codes + static_cast<size_t>(pc.t) * P.nblk * kChunk;
    const uint8_t* xr = xs + MxSets<B>::kRow * (threadIdx.x & 3);
    const int jg = pc.jg;
    int j = pc.j;
    int kb = pc.c0 - 4 * j;
    MxPipe<B> st;
#pragma unroll
    for (int s = 0; s < NS; ++s) st.acc[s] = f32x4{0.f, 0.f, 0.f, 0.f};
    // x of group j + 1 is requested at the start of group j; after the last
    // group that is the trailing columns' group (ng), when the piece has them
    const int jx = pc.tr ? P.ng : jg;
    XGroup<B> xn = xp;
    if (j <= jg) {
        const int kl = __builtin_amdgcn_readfirstlane(pc.tr ? tetra::kGroupCols : pc.c1 - 4 * jg);
        write_xgroup<B>(xs, xn);
        xn = load_xgroup<B>(P, min(j + 1, jx));
        start_pipe_mx<B>(st, pc.cw, kb, L);
        ItemWords wa = pc.cw, wb = pc.nw;
        for (;;) {
            run_one_item_mx<B>(st, kb, j == jg ? kl : tetra::kGroupCols, wa, wb, L, xr);
            if (j == jg) break;
            ++j;
            kb = 0;
            write_xgroup<B>(xs, xn);
            wa = load_group(tb, min(j + 1, jg), lane);
            xn = load_xgroup<B>(P, min(j + 1, jx));
            run_one_item_mx<B>(st, 0, j == jg ? kl : tetra::kGroupCols, wb, wa, L, xr);
            if (j == jg) break;
            ++j;
            write_xgroup<B>(xs, xn);
            wb = load_group(tb, min(j + 1, jg), lane);
            xn = load_xgroup<B>(P, min(j + 1, jx));
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);
        mx_finish<B>(st);
        kb = 0;
    }
    if (pc.tr) {
        const int c = 4 * P.ng;
        ItemWords tw = pc.tw;
        trailing_fixup(tw, P.rem);
        write_xgroup<B>(xs, xn);
        start_pipe_mx<B>(st, tw, kb, L);
        run_item_mx<B, false>(st, tw, tw, kb, pc.c1 - c, L, xr);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        mx_finish<B>(st);
    }
    // lane 4i + j holds rows 4i..4i+3 of batch row 4s + j: through the slots
    // (after the last reads of x, LDS operations of a wave being in order)
    // to one row per lane
#pragma unroll
    for (int s = 0; s < NS; ++s)
        *reinterpret_cast<f32x4*>(xs + s * kXSlotBytes + 256 * (threadIdx.x & 3) + 16 * ((threadIdx.x & 63) >> 2)) =
            st.acc[s];
#pragma unroll
    for (int bb = 0; bb < B; ++bb) out[bb] = *reinterpret_cast<const float*>(xs + 256 * bb + 4 * (threadIdx.x & 63));
}

// ------------------------------------------------ batch 1: matrix cores
//
// With q = 1 - p and s_t = (-1)^(c_t xor q) U(rho_t) (the signed row values,
// before q is added), a block's coordinates are y_t = s_t + q, so
//   dot(y, x) = sum s_t x_t + q sum x_t,
//   |y|^2 = 16 m = sum s_t^2 + q (2 sum s_t + 24).
// The products with x and the plain sums go to the matrix cores:
// v_mfma_f32_4x4x4f16 with its A operand broadcast from one block of four
// lanes (cbsz 4, abid b) computes, in every lane, D[r] += A_b[r] . B, where
// A_b[r] is lane 4b + r's four values and B the lane's own.  Lanes 4c
// (c < 6) hold chunk c of the block's activations (x_{4c..4c+3}) and lanes
// 4c + 1 four ones; lanes 32 + 4c hold the same chunk and lanes 33 + 4c four
// halves.  Six products with B = s (abid c) and six with B = (q, q, q, q)
// (abid 8 + c) leave D[0] = sum (s_t + q) x_t, the block's dot product, and
// D[1] = sum s_t + 12 q, so that 16 m = sum s_t^2 + 2 q D[1].  sum s_t^2
// does not depend on the signs: it is the three rows' stored costs (sum of
// U^2 over a row).  The vector unit keeps the conversions and the signs; the
// pk_adds of q, the dot products with x and the norm's squares leave it.
// All values on the norm's path are exact: sum s_t^2, D[1] and 2^23 + 4096 g
// + 16 m are integers below 2^24.
//
// The activations of an item pass through a per-wave LDS slot: lane l loads
// bytes 8 (l mod 24) .. +7 of the item's 192 (chunk (l mod 24) mod 6 of
// column (l mod 24) / 6; lanes past 24 repeat them) one item ahead, and the
// previous item's last block writes them to the slot; each block reads the
// next block's A operand with one ds_read_b64 per lane.  The constants sit
// after the four columns, repeated 48 bytes apart so that one immediate
// offset serves every lane.

constexpr int kX1Cols = 192;          // bytes of one item's activations in a slot
constexpr int kX1Slot = 352;          // + ones and halves at kX1Cols + 48 k (+ 8), k < 4
constexpr uint32_t kHalf2One = 0x3C003C00u, kHalf2Half = 0x38003800u;

// lane l's 8 bytes of the activations of the item whose first column is
// col0 (columns past the last one read the last column's last chunk)
__device__ __forceinline__ uint2 load_x1(const GemvProblem& P, int col0, int m8) {
    const uint32_t off = static_cast<uint32_t>(min(48 * col0 + m8, 48 * P.nblk - 8));
    return *reinterpret_cast<const uint2*>(reinterpret_cast<const uint8_t*>(P.x) + off);
}

// the lane's read offset in the slot for its A operand row
__device__ __forceinline__ int x1_read_off(int l) {
    const int b = l >> 2, r = l & 3;
    if (r == 0 && b < 6) return 8 * b;
    if (r == 0 && b >= 8 && b < 14) return 8 * (b - 8);
    return kX1Cols + (r == 1 && l >= 32 ? 8 : 0);
}

struct Pipe1 {
    BlockFetch cur;         // its bias holds 2^23 + 4096 g + the rows' costs
    u32x2 a;                // the current block's A operand
    float ps, pdt, acc;
};

// chunk C of a block (coordinates 4C..4C+3): its signed values into the
// product, and its four q's (abid 8 + C; independent of the values, so the
// two products need no wait between them beyond the conversions)
template <int C>
__device__ __forceinline__ void chunk_products(const BlockFetch& f, uint32_t ep, half4_t A, half4_t Q, f32x4& d) {
    const uint32_t sg = f.r[C] ^ ((ep << C) & 0x80808080u);
    const uint32_t s0 = cvt_pair<false>(sg), s1 = cvt_pair<true>(sg);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(A, Q, d, 4, 8 + C, 0);
    d = __builtin_amdgcn_mfma_f32_4x4x4f16(A, as_half4(s0, s1), d, 4, C, 0);
}

// D[0] = the block's dot product, D[1] = sum s_t + 12 q
__device__ __forceinline__ f32x4 block_products1(const BlockFetch& f, u32x2 a) {
    const uint32_t ep = f.e ^ (~f.pm & 0xFCFCFCFCu);
    const uint32_t qp = ~f.pm & kHalf2One;
    const half4_t A = as_half4(a.x, a.y), Q = as_half4(qp, qp);
    f32x4 d = {0.f, 0.f, 0.f, 0.f};
    chunk_products<0>(f, ep, A, Q, d);
    chunk_products<1>(f, ep, A, Q, d);
    chunk_products<2>(f, ep, A, Q, d);
    chunk_products<3>(f, ep, A, Q, d);
    chunk_products<4>(f, ep, A, Q, d);
    chunk_products<5>(f, ep, A, Q, d);
    return d;
}

// 2^23 + 4096 g + 16 m from the bias with the row costs (sum s_t^2) and
// D[1]: 16 m = sum s_t^2 + 2 q (sum s_t + 12)
__device__ __forceinline__ float block_norm1(const BlockFetch& f, float d1) {
    return fmaf(__builtin_bit_cast(float, ~f.pm & 0x40000000u), d1, __builtin_bit_cast(float, f.bias));
}

typedef __attribute__((address_space(3))) uint8_t lds_bytes_w;
typedef __attribute__((address_space(3))) u32x2 lds_u2_w;

__device__ __forceinline__ void put_x1(lds_bytes_w* xs, int m8, uint2 xw) {
    *(lds_u2_w*)(xs + m8) = u32x2{xw.x, xw.y};
}

// Blocks kb..ke-1 of one item (words cw; the next item's words nw and
// activations xn), as run_item.  Each block reads the next block's A operand
// with its table rows; the last one first writes the next item's
// activations to the slot (every read of this item's was issued before, and
// a wave's LDS operations complete in order).  xs: the wave's slot, m8 =
// 8 (lane mod 24), ro: x1_read_off.
template <bool Full>
__device__ __forceinline__ void run_item1(Pipe1& st, const ItemWords& cw, const ItemWords& nw, uint2 xn, int kb,
                                          int ke, lds_bytes* L, lds_bytes_w* xs, int m8, int ro) {
#pragma unroll
    for (int k = 0; k < tetra::kGroupCols; ++k) {
        if (Full || (k >= kb && k < ke)) {
            uint32_t lo, hi;
            int an;
            if (k + 1 < tetra::kGroupCols && (Full || k + 1 < ke)) {
                if (k == 0) block_word<1>(cw, lo, hi);
                else if (k == 1) block_word<2>(cw, lo, hi);
                else block_word<3>(cw, lo, hi);
                an = 48 * (k + 1);
            } else {
                block_word<0>(nw, lo, hi);
                put_x1(xs, m8, xn);
                an = 0;
            }
            const f32x4 d = block_products1(st.cur, st.a);
            __builtin_amdgcn_sched_barrier(0);
            uint32_t cn[3];
            BlockFetch nxt = fetch_block<true>(lo, hi, L, cn);
            const u32x2 a = *(lds_u2*)(xs + ro + an);
            const float sq = block_norm1(st.cur, d[1]);
            __builtin_amdgcn_sched_barrier(0);
            // one wait per block: the next block's reads and the previous
            // block's scale
            __builtin_amdgcn_s_waitcnt(0xC07F);
            st.acc = fmaf(st.ps, st.pdt, st.acc);
            const uint32_t sa = (__builtin_bit_cast(uint32_t, sq) >> 2) & 0x7FFu;
            st.ps = *(lds_f32*)(L + kScaleOff + sa);
            st.pdt = d[0];
            asm volatile("" : : "v"(st.pdt));
            __builtin_amdgcn_sched_barrier(0);
            nxt.bias += cn[0] + cn[1] + cn[2];
            st.cur = nxt;
            st.a = a;
        }
    }
}

__device__ __forceinline__ void run_one_item1(Pipe1& st, int kb, int ke, const ItemWords& cw, const ItemWords& nw,
                                              uint2 xn, lds_bytes* L, lds_bytes_w* xs, int m8, int ro) {
    if (kb == 0 && ke == tetra::kGroupCols)
        run_item1<true>(st, cw, nw, xn, 0, tetra::kGroupCols, L, xs, m8, ro);
    else
        run_item1<false>(st, cw, nw, xn, kb, ke, L, xs, m8, ro);
}

// first block of a run of items: the item's activations into the slot, the
// block's table reads and A operand, and an empty "previous block"
__device__ __forceinline__ void start_pipe1(Pipe1& st, const ItemWords& w, uint2 xw, int kb, lds_bytes* L,
                                            lds_bytes_w* xs, int m8, int ro) {
    uint32_t lo, hi;
    if (kb == 0) block_word<0>(w, lo, hi);
    else if (kb == 1) block_word<1>(w, lo, hi);
    else if (kb == 2) block_word<2>(w, lo, hi);
    else block_word<3>(w, lo, hi);
    put_x1(xs, m8, xw);
    uint32_t cn[3];
    st.cur = fetch_block<true>(lo, hi, L, cn);
    st.a = *(lds_u2*)(xs + ro + 48 * kb);
    __builtin_amdgcn_s_waitcnt(0xC07F);
    st.cur.bias += cn[0] + cn[1] + cn[2];
    st.ps = 0.f;
    st.pdt = 0.f;
}

// run_piece at batch 1.  The activations of an item are requested one item
// ahead, before the item's code words (so that waiting for them never waits
// for later words); after the last group they are those of the trailing
// columns, the item that follows it.  They are requested here, after the
// chain barrier: the piece's code words may have been requested before it.
__device__ __forceinline__ void run_piece1(const GemvProblem& P, Piece& pc, lds_bytes* L, lds_bytes_w* xs,
                                           float (&out)[1]) {
    const int lane = threadIdx.x & 63;
    const int m8 = 8 * (lane % 24);
    const int ro = x1_read_off(lane);
    const uint8_t* tb = P.codes + static_cast<size_t>(pc.t) * P.nblk * kChunk;
    const int jg = pc.jg;
    int j = pc.j;
    int kb = pc.c0 - 4 * j;
    Pipe1 st;
    st.acc = 0.f;
    uint2 xn = load_x1(P, 4 * j, m8);      // item j, or the trailing columns when j > jg
    if (j <= jg) {
        const int kl = __builtin_amdgcn_readfirstlane(pc.tr ? tetra::kGroupCols : pc.c1 - 4 * jg);
        ItemWords wa = pc.cw, wb = pc.nw;
        const uint2 xw = xn;
        xn = load_x1(P, 4 * (j + 1), m8);
        start_pipe1(st, wa, xw, kb, L, xs, m8, ro);
        const int ngr = jg - j + 1;
        __builtin_amdgcn_s_setprio(3);
        for (;;) {
            run_one_item1(st, kb, j == jg ? kl : tetra::kGroupCols, wa, wb, xn, L, xs, m8, ro);
            if (j == jg) break;
            ++j;
            progress_prio(jg - j + 1, ngr);
            kb = 0;
            xn = load_x1(P, 4 * (j + 1), m8);
            wa = load_group(tb, min(j + 1, jg), lane);
            run_one_item1(st, 0, j == jg ? kl : tetra::kGroupCols, wb, wa, xn, L, xs, m8, ro);
            if (j == jg) break;
            ++j;
            progress_prio(jg - j + 1, ngr);
            xn = load_x1(P, 4 * (j + 1), m8);
            wb = load_group(tb, min(j + 1, jg), lane);
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);
        st.acc = fmaf(st.ps, st.pdt, st.acc);
        kb = 0;
    }
    if (pc.tr) {
        ItemWords tw = pc.tw;
        trailing_fixup(tw, P.rem);
        start_pipe1(st, tw, xn, kb, L, xs, m8, ro);
        run_item1<false>(st, tw, tw, xn, kb, pc.c1 - 4 * P.ng, L, xs, m8, ro);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        st.acc = fmaf(st.ps, st.pdt, st.acc);
    }
    __builtin_amdgcn_s_setprio(1);
    out[0] = st.acc;
}

// the constants of a wave's slot (lanes 0-7: ones, halves of item column k)
__device__ __forceinline__ void x1_slot_init(lds_bytes_w* xs) {
    const int l = threadIdx.x & 63;
    const uint32_t v = (l & 1) ? kHalf2Half : kHalf2One;
    if (l < 8) *(lds_u2_w*)(xs + kX1Cols + 48 * (l >> 1) + 8 * (l & 1)) = u32x2{v, v};
}


// y of a tile's rows: sigma_row * sum + unquantised tail (T = K mod 24 is
// even, so the tail is at most 11 fp16 pairs).  load_rows issues the loads,
// store_rows does the arithmetic and the stores, so that the loads can be in
// flight while the sums are being combined.
struct RowTail {
    uint32_t tv[11];
    float sg;
};

__device__ __forceinline__ RowTail load_rows(const GemvProblem& P, int t) {
    RowTail r;
    const int row = min(t * kTile + lane_now(), P.M - 1);
    const uint32_t* tl =
        reinterpret_cast<const uint32_t*>(P.codes + P.tail_off) + static_cast<size_t>(row) * (P.T >> 1);
    r.sg = f16(P.sigma[row]);
#pragma unroll
    for (int q = 0; q < 11; ++q) r.tv[q] = 2 * q < P.T ? tl[q] : 0u;
    return r;
}

// The tail's activation pairs are loaded four at a time (pair q read from
// min(q, T/2 - 1), so every read is in bounds) and the pairs past the tail
// left out by a select: a load per pair behind its own branch would cost a
// round trip each.
template <int B>
__device__ __forceinline__ void store_rows(const GemvProblem& P, int t, const float (&tot)[B], const RowTail& r) {
    const int row = t * kTile + lane_now();
    if (row >= P.M) return;
    const_u32* xc = (const_u32*)(P.x);
    const int th = P.T >> 1;                                // tail pairs
#pragma unroll
    for (int bb = 0; bb < B; ++bb) {
        const int x0 = bb * (P.K >> 1) + 12 * P.nblk;     // first tail pair of x_b
        float ts = 0.f;
#pragma unroll
        for (int q0 = 0; q0 < 11; q0 += 4) {
            if (q0 < th) {
                uint32_t xv[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) xv[u] = xc[x0 + min(q0 + u, th - 1)];
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    if (q0 + u < 11) {
                        const float d = dot2(r.tv[q0 + u], xv[u], ts);
                        ts = q0 + u < th ? d : ts;
                    }
            }
        }
        P.y[static_cast<size_t>(bb) * P.M + row] = fmaf(r.sg, tot[bb], ts);
    }
}

// Where a wave's range of a phase starts: problem p (absolute index), tile
// t, columns c..c1-1 of its first piece, blocks i..end-1 of the phase's
// sequence; live is false for a wave past the phase's waves.
struct RangePos {
    int p, t, c, c1;
    uint32_t i, end;
    bool live;
};

// What a range position needs of the launch: the phase's split and the
// first block and block columns of its problems.  Read from the kernel
// arguments (phase 0, before anything is staged) or from the workgroup's
// copy in LDS (later phases: the arguments' lines have long left the scalar
// cache by then, and a chain of scalar misses would stall the wave for
// microseconds).
struct ArgSrc {
    const GemvChain& ch;
    __device__ __forceinline__ GemvSplit split(int k) const { return ch.ph[k]; }
    __device__ __forceinline__ uint32_t base(int q) const { return ch.prob[q].blk_base; }
    __device__ __forceinline__ int nblk(int q) const { return ch.prob[q].nblk; }
};

// the part of the kernel arguments that range positions read, staged in LDS
struct StagedChain {
    GemvSplit ph[kMaxPhases];
    uint32_t base[kMaxGroup];
    int nblk[kMaxGroup];
};
constexpr int kStagedWords = static_cast<int>(sizeof(StagedChain) / 4);
static_assert(sizeof(StagedChain) % 4 == 0 && sizeof(GemvSplit) % 4 == 0, "word copies");

constexpr int kSplitWords = static_cast<int>(sizeof(GemvSplit) / 4);

// word w of the staged copy, from the kernel arguments
__device__ __forceinline__ uint32_t staged_word(const GemvChain& ch, int w) {
    if (w < kSplitWords * kMaxPhases) return reinterpret_cast<const uint32_t*>(ch.ph)[w];
    if (w < kSplitWords * kMaxPhases + kMaxGroup) return ch.prob[w - kSplitWords * kMaxPhases].blk_base;
    return static_cast<uint32_t>(ch.prob[min(w - kSplitWords * kMaxPhases - kMaxGroup, kMaxGroup - 1)].nblk);
}

// the staged copy, read through an LDS pointer, one phase per lane (the
// ranges of all later phases are worked out at once, lane k for phase k)
struct LdsSrc {
    lds_u32* w;
    __device__ __forceinline__ uint32_t rd(int i) const { return w[i]; }
    __device__ __forceinline__ GemvSplit split(int k) const {
        uint32_t o[kSplitWords];
#pragma unroll
        for (int u = 0; u < kSplitWords; ++u) o[u] = rd(k * kSplitWords + u);
        return __builtin_bit_cast(GemvSplit, o);
    }
    __device__ __forceinline__ uint32_t base(int q) const { return rd(kSplitWords * kMaxPhases + q); }
    __device__ __forceinline__ int nblk(int q) const {
        return static_cast<int>(rd(kSplitWords * kMaxPhases + kMaxGroup + q));
    }
};

// Uniform: k is the same on every lane (the values go to scalar registers)
template <class Src, bool Uniform = true>
__device__ __forceinline__ RangePos range_pos(const Src& src, int k, int g, int wid) {
    auto rfl = [](uint32_t v) { return Uniform ? __builtin_amdgcn_readfirstlane(v) : v; };
    const GemvSplit sp = src.split(k);
    const int w = g * sp.wpg + wid;
    RangePos r;
    r.live = wid < sp.wpg && w < sp.waves;
    const int wr = r.live ? w : sp.waves - 1;
    if (sp.aligned) {
        // the tile of wave wr holds block floor(((wr + 1) total - 1) / W)
        const uint32_t bs = div_exact(static_cast<unsigned long long>(wr + 1) * sp.total - 1,
                                      static_cast<uint32_t>(sp.waves), sp.inv_waves);
        int q = sp.p0;
        while (q + 1 < sp.p0 + sp.n && bs >= src.base(q + 1)) ++q;
        const uint32_t nb = static_cast<uint32_t>(src.nblk(q));
        const uint32_t b0 = src.base(q);
        const uint32_t t0 = b0 + (bs - b0) / nb * nb;
        const int wa = tile_first_wave(t0, sp);
        const uint32_t n = static_cast<uint32_t>(tile_first_wave(t0 + nb, sp) - wa);
        const uint32_t j = static_cast<uint32_t>(wr - wa);
        r.i = rfl(t0 + j * nb / n);
        r.end = rfl(t0 + (j + 1) * nb / n);
        r.p = q;        // the tile's problem holds the whole range
    } else {
        r.i = rfl(range_begin(wr, sp));
        r.end = rfl(range_begin(wr + 1, sp));
        int q = sp.p0;
        while (q + 1 < sp.p0 + sp.n && r.i >= src.base(q + 1)) ++q;
        r.p = q;
    }
    const int nbp = src.nblk(r.p);
    const uint32_t rel = r.i - src.base(r.p);
    r.t = static_cast<int>(rfl(rel / static_cast<uint32_t>(nbp)));
    r.c = static_cast<int>(rfl(rel - static_cast<uint32_t>(r.t) * nbp));
    const uint32_t left = r.end - r.i;
    r.c1 = left < static_cast<uint32_t>(nbp - r.c) ? r.c + static_cast<int>(left) : nbp;
    return r;
}

// A wave's range of every later phase of a chain, worked out once (in the
// first barrier's window) and kept in LDS, 6 words per phase: each later
// transition reads it back instead of redoing the divisions.
constexpr int kRangeWords = 6;

__device__ __forceinline__ void put_range(uint32_t* slot, const RangePos& r) {
    slot[0] = r.i;
    slot[1] = r.end;
    slot[2] = static_cast<uint32_t>(r.t);
    slot[3] = static_cast<uint32_t>(r.c);
    slot[4] = static_cast<uint32_t>(r.c1);
    slot[5] = static_cast<uint32_t>(r.p) | (r.live ? 1u << 31 : 0u);
}

__device__ __forceinline__ RangePos get_range(lds_u32* slot) {
    RangePos r;
    r.i = __builtin_amdgcn_readfirstlane(slot[0]);
    r.end = __builtin_amdgcn_readfirstlane(slot[1]);
    r.t = static_cast<int>(__builtin_amdgcn_readfirstlane(slot[2]));
    r.c = static_cast<int>(__builtin_amdgcn_readfirstlane(slot[3]));
    r.c1 = static_cast<int>(__builtin_amdgcn_readfirstlane(slot[4]));
    const uint32_t w = __builtin_amdgcn_readfirstlane(slot[5]);
    r.p = static_cast<int>(w & 0x7FFFFFFFu);
    r.live = (w >> 31) != 0;
    return r;
}

// A tile of a deferred phase whose workgroup sums its first workgroup's last
// wave adds up later: problem p, tile t, workgroups ga..gb, the slot of ga's
// sum.  Packed into two wave-uniform words; p < 0: none.
struct Pending {
    int p, t, ga, gb, gs;
};

__device__ __forceinline__ Pending no_pending() { return Pending{-1, 0, 0, 0, 0}; }

// the workgroup sums ga..gb of tile t (slot gs for ga, 0 for the others),
// added in workgroup order, times sigma, plus the tail, into y
template <int B>
__device__ __forceinline__ void combine_groups(const GemvProblem& P, int t, int ga, int gb, int gs,
                                               const float* partials) {
    const int ln = lane_now();
    const RowTail rt = load_rows(P, t);   // in flight while the sums combine
    auto gslot_of = [&](int h) { return h > ga ? 0 : gs; };
    float out[B];
#pragma unroll
    for (int bb = 0; bb < B; ++bb) out[bb] = 0.f;
    // loads in batches of eight, added in workgroup order
    for (int h0 = ga; h0 <= gb; h0 += 8) {
        float pv[8][B];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int h = h0 + u;
            if (h <= gb) {
                const float* ph = partials + (static_cast<size_t>(h) * 2 + gslot_of(h)) * B * 64 + ln;
#pragma unroll
                for (int bb = 0; bb < B; ++bb)
                    pv[u][bb] = __hip_atomic_load(ph + bb * 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
            if (h0 + u <= gb) {
#pragma unroll
                for (int bb = 0; bb < B; ++bb) out[bb] += pv[u][bb];
            }
    }
    store_rows<B>(P, t, out, rt);
}

// Pieces of a tile are combined in two levels: the waves of one workgroup
// that hold pieces of the tile add them in LDS (the last of them to arrive,
// in wave order), and when the tile reaches into other workgroups each
// workgroup's sum goes to the workspace, where the last workgroup to arrive
// adds them in workgroup order.  In a deferred phase no workgroup waits
// for the others: the workgroup sums are complete at the next chain
// barrier, and the wave that wrote the first workgroup's sum adds them up
// while it waits at the barrier after that (or at the launch's end), which
// takes two device-wide round trips (a counter and the loads) off the
// phase's end.  Piece p (problem index) of a wave's range: its sum, then its
// share of the tile's reduction.  w0: the workgroup's first wave of the
// phase (g * wpg).
template <int B>
__device__ __forceinline__ void finish_piece(const GemvProblem& P, const GemvSplit& sp, int p, int t, int c,
                                             int c1, bool first, const float (&sum)[B], int w0, int g,
                                             float* s_piece, uint32_t* s_cnt, uint32_t* counters, float* partials,
                                             Pending& pend) {
    if (c == 0 && c1 == P.nblk) {
        const RowTail rt = load_rows(P, t);
        store_rows<B>(P, t, sum, rt);
        return;
    }
    const int wid = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int wlast = min(w0 + sp.wpg, sp.waves) - 1;
    const uint32_t t0 = P.blk_base + static_cast<uint32_t>(t) * P.nblk;
    // the tile's contributors wa..wb; slot of wave v's piece of this tile: 0
    // when the tile is where v's range starts, which holds for every
    // contributor but possibly the first (always, in a tile-aligned split)
    int wa, wb, slot_wa;
    if (sp.aligned) {
        wa = __builtin_amdgcn_readfirstlane(tile_first_wave(t0, sp));
        wb = __builtin_amdgcn_readfirstlane(tile_first_wave(t0 + P.nblk, sp)) - 1;
        slot_wa = 0;
    } else {
        wa = __builtin_amdgcn_readfirstlane(wave_of(t0, sp));
        wb = __builtin_amdgcn_readfirstlane(wave_of(t0 + P.nblk - 1, sp));
        slot_wa = __builtin_amdgcn_readfirstlane(range_begin(wa, sp) >= t0 ? 0 : 1);
    }
    auto slot_of = [&](int v) { return v > wa ? 0 : slot_wa; };
    const int a = max(wa, w0), b = min(wb, wlast);
    const int ln = lane_now();
    float* mine = s_piece + (wid * 2 + (first ? 0 : 1)) * B * 64 + ln;
#pragma unroll
    for (int bb = 0; bb < B; ++bb) mine[bb * 64] = sum[bb];
    // LDS operations of a wave complete in order, and the last wave reads the
    // pieces only after its own count: no fence is needed
    uint32_t arrived = 0;
    if (ln == 0)
        arrived = __hip_atomic_fetch_add(s_cnt + 2 * (b - w0) + slot_of(b), 1u, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_WORKGROUP);
    arrived = __builtin_amdgcn_readfirstlane(arrived);
    if (arrived != static_cast<uint32_t>(b - a)) return;
    // last of this workgroup's pieces of the tile: add them in wave order
    const bool inside = wa >= w0 && wb <= wlast;   // the tile lies in this workgroup
    RowTail rt;
    if (inside) rt = load_rows(P, t);   // in flight while the sums combine
    float tot[B];
#pragma unroll
    for (int bb = 0; bb < B; ++bb) tot[bb] = 0.f;
    for (int v = a; v <= b; ++v) {
        const float* pv = s_piece + ((v - w0) * 2 + slot_of(v)) * B * 64 + ln;
#pragma unroll
        for (int bb = 0; bb < B; ++bb) tot[bb] += pv[bb * 64];
    }
    if (inside) {
        store_rows<B>(P, t, tot, rt);
        return;
    }
    // the tile reaches into other workgroups: publish this workgroup's sum.
    // Workgroup sums and counters are accessed only with device-scope
    // atomics, which are coherent across the chip's L2 caches; the wait
    // orders the sum before the count.
    const int ga = wa / sp.wpg, gb = wb / sp.wpg;
    // slot 0 holds the tile reaching in from earlier workgroups, slot 1 one
    // that starts inside the workgroup and reaches past it
    const int gslot_ga = sp.aligned ? (ga * sp.wpg >= wa ? 0 : 1)
                                    : __builtin_amdgcn_readfirstlane(range_begin(ga * sp.wpg, sp) >= t0 ? 0 : 1);
    float* gp = partials + (static_cast<size_t>(g) * 2 + (g > ga ? 0 : gslot_ga)) * B * 64 + ln;
#pragma unroll
    for (int bb = 0; bb < B; ++bb)
        __hip_atomic_store(gp + bb * 64, tot[bb], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // The sum must be complete before the count, or before the barrier after
    // which it is read.  A wave's vector memory operations complete in the
    // order they were issued, so a sum that is read only after the barrier
    // that follows the next phase (defer 2) needs no wait here: the wave
    // waits for the code words of its next piece, requested after this
    // store, before it arrives there (a wave with no piece in that phase
    // waits for everything before it arrives).
    if (sp.defer != 2) __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
    if (sp.defer) {
        if (g == ga) pend = Pending{p, t, ga, gb, gslot_ga};
        return;
    }
    uint32_t garr = 0;
    if (ln == 0) garr = __hip_atomic_fetch_add(counters + gb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    garr = __builtin_amdgcn_readfirstlane(garr);
    if (garr != static_cast<uint32_t>(gb - ga)) return;
    if (ln == 0) __hip_atomic_store(counters + gb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    combine_groups<B>(P, t, ga, gb, gslot_ga, partials);
}

// The whole launch: decoder tables staged once, then the phases in order (one
// for a plain or grouped product, Chain false).  A wave walks the pieces of
// its range of a phase; at the range's end (Chain) it requests the code words
// of its first piece of the next phase, which no phase writes, and its
// workgroup waits at the chain barrier with those words in flight.  A wave
// with no range in a phase goes straight to the barrier.
template <int B, bool Chain>
__global__ __launch_bounds__(kGemvThreads) __attribute__((amdgpu_waves_per_eu(B <= 2 ? 6 : 3)))
void gemv_kernel(const GemvChain ch) {
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    __shared__ float s_piece[kGemvWaves * 2 * B * 64];   // [wave][first/last piece][B][64]
    __shared__ uint32_t s_cnt[2 * kGemvWaves + 1];       // piece counts; the last word: the launch is abandoned
    constexpr int kAbandoned = 2 * kGemvWaves;
    constexpr bool kMx = B >= 3;
    __shared__ uint4 s_xs[kMx ? kGemvWaves * MxSets<B>::kN * kXSlotBytes / 16 : 1];   // batch >= 3: x slots per wave
    constexpr bool kX1 = B == 1;
    __shared__ uint2 s_x1[kX1 ? kGemvWaves * kX1Slot / 8 : 1];                         // batch 1: x slots per wave
    __shared__ uint32_t s_ch[Chain ? kStagedWords : 1];   // StagedChain
    __shared__ uint32_t s_rng[Chain ? kGemvWaves * kMaxPhases * kRangeWords : 1];   // [wave][phase] ranges
    if (threadIdx.x < 2 * kGemvWaves) s_cnt[threadIdx.x] = 0;
    lds_bytes* L = (lds_bytes*)(s_tab);
    const int lane = threadIdx.x & 63;
    const int wid = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int g = static_cast<int>(blockIdx.x);
    TableStage<kGemvThreads> ts;
    ts.load();
    static_assert(kStagedWords <= kGemvThreads, "one word per thread");
    const uint32_t chw = Chain ? staged_word(ch, min(static_cast<int>(threadIdx.x), kStagedWords - 1)) : 0u;
    uint32_t* const counters = g_gemv_slots[ch.slot].counters;
    float* const partials = g_gemv_slots[ch.slot].partials;
    // the first piece's code words are requested while the tables arrive;
    // the barrier orders LDS only, so they stay in flight across it
    RangePos r = range_pos(ArgSrc{ch}, 0, g, wid);
    int p = r.p, t = r.t, c = r.c, c1 = r.c1;
    uint32_t i = r.i, end = r.end;
    Piece pc = begin_piece_live(ch.prob[p], t, c, c1, lane, r.live);
    lds_bytes_w* const x1s = (lds_bytes_w*)(s_x1) + (kX1 ? wid * kX1Slot : 0);
    if constexpr (kX1) x1_slot_init(x1s);
    XGroup<B> xp;
    if constexpr (kMx) xp = begin_xpiece<B>(ch.prob[p], pc, r.live);
    uint8_t* xs = reinterpret_cast<uint8_t*>(s_xs) + (kMx ? wid * MxSets<B>::kN * kXSlotBytes : 0);
    ts.store(s_tab);
    if (Chain && threadIdx.x < kStagedWords) s_ch[threadIdx.x] = chw;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    if constexpr (!Chain) {
        if (!r.live) return;
    }
    int k = 0;                    // the phase
    bool live = r.live;
    bool first = true;
    // tiles of deferred phases this wave adds up: from the phase before the
    // last barrier (old) and from the current phase (cur)
    Pending pend_old = no_pending(), pend_cur = no_pending();
    const size_t pstride = static_cast<size_t>(gridDim.x) * 2 * B * 64;
    bool abandoned = false;
    for (;;) {
        if (!Chain || live) {
            const GemvProblem& P = ch.prob[p];
            float sum[B];
            if constexpr (kMx) run_piece_mx<B>(P, pc, xp, L, xs, sum);
            else if constexpr (kX1) run_piece1(P, pc, L, x1s, sum);
            else run_piece<B>(P, pc, L, sum);
            finish_piece<B>(P, ch.ph[k], p, t, c, c1, first, sum, g * ch.ph[k].wpg, g, s_piece, s_cnt, counters,
                            partials + (Chain ? (k % ch.buffers) * pstride : 0), pend_cur);
            i += static_cast<uint32_t>(c1 - c);
            if (i < end) {
                first = false;
                c = 0;
                if (++t == ch.prob[p].tiles) {
                    t = 0;
                    ++p;
                }
                const uint32_t left = end - i;
                c1 = left < static_cast<uint32_t>(ch.prob[p].nblk) ? static_cast<int>(left) : ch.prob[p].nblk;
                pc = begin_piece(ch.prob[p], t, 0, c1, lane);
                if constexpr (kMx) xp = begin_xpiece<B>(ch.prob[p], pc, true);
                continue;
            }
        }
        if constexpr (!Chain) {
            break;
        } else {
            // the wave's range of phase k is done
            if (++k == ch.n_phases) break;
            // every wave of the workgroup is done with phase k - 1 (and with its
            // LDS pieces and counts); one lane counts the workgroup in and
            // waits.  Meanwhile every wave adds up the deferred tiles it holds,
            // finds its range of phase k and requests the code words of its
            // first piece, which no phase writes.  A wave that had no piece in
            // phase k - 1 may still have sums of phase k - 2 in flight.
            if (!live) __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
            {
                // the thread index from the lane at hand: an address kept
                // from the launch's start would hold a register throughout
                const int tx = wid * 64 + lane_now();
                if (tx < 2 * kGemvWaves) s_cnt[tx] = 0;
            }
            const bool polls = threadIdx.x == 0;    // the lane that counts the workgroup in and waits
            ChainSync& cs = g_chain_sync[ch.slot];
            if (polls) chain_arrive(cs, k - 1, g, static_cast<int>(gridDim.x));
            // at the first barrier, lane k works out the wave's range of phase
            // k for every later phase (only this wave reads them, and its LDS
            // operations complete in order)
            uint32_t* const rng = s_rng + wid * kMaxPhases * kRangeWords;
            if (k == 1) {
                // the lane index afresh: an address kept from the launch's
                // start would hold a register throughout
                const int ln = lane_now();
                if (ln >= 1 && ln < ch.n_phases)
                    put_range(rng + ln * kRangeWords, range_pos<LdsSrc, false>(LdsSrc{(lds_u32*)(s_ch)}, ln, g, wid));
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            r = get_range((lds_u32*)(rng + k * kRangeWords));
            p = r.p;
            t = r.t;
            c = r.c;
            c1 = r.c1;
            i = r.i;
            end = r.end;
            live = r.live;
            first = true;
            pc = begin_piece_live(ch.prob[p], t, c, c1, lane, live);
            if constexpr (kMx) xp = begin_xpiece<B>(ch.prob[p], pc, live);
            // the deferred tiles of phase k - 2, complete since the barrier
            // before phase k - 1 (after the code-word requests, so that the
            // waves waiting for those do not wait for this tile's y stores)
            if (pend_old.p >= 0)
                combine_groups<B>(ch.prob[pend_old.p], pend_old.t, pend_old.ga, pend_old.gb, pend_old.gs,
                                  partials + ((k - 2) % ch.buffers) * pstride);
            pend_old = pend_cur;
            pend_cur = no_pending();
            if (wid == 0) {
                const bool met = chain_wait(cs, k - 1, g, static_cast<int>(gridDim.x), ch.wait_limit);
                if (polls) {
                    if (!met) dev_add(&cs.expired[0], 1u);
                    s_cnt[kAbandoned] = met ? 0u : 1u;
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
            // a wait that gave up abandons the launch: running ahead could
            // overwrite piece sums that a slower workgroup has yet to read
            if (__builtin_amdgcn_readfirstlane(s_cnt[kAbandoned])) {
                abandoned = true;
                break;
            }
            // before the last phase: the deferred tiles of phase k - 1,
            // complete now, rather than at the launch's end, where they
            // would add to its tail
            if (k + 1 == ch.n_phases && pend_old.p >= 0) {
                combine_groups<B>(ch.prob[pend_old.p], pend_old.t, pend_old.ga, pend_old.gb, pend_old.gs,
                                  partials + ((k - 1) % ch.buffers) * pstride);
                pend_old = no_pending();
            }
        }
    }
    if constexpr (Chain) {
        // the deferred tiles of the next-to-last phase (the last phase is
        // never deferred)
        if (!abandoned && pend_old.p >= 0)
            combine_groups<B>(ch.prob[pend_old.p], pend_old.t, pend_old.ga, pend_old.gb, pend_old.gs,
                              partials + ((ch.n_phases - 2) % ch.buffers) * pstride);
        // the last workgroup to finish reports the status and clears the
        // barrier words for the next launch on the slot (every workgroup has
        // passed its last wait by then)
        ChainSync& cs = g_chain_sync[ch.slot];
        if (threadIdx.x == 0 && dev_add(&cs.exit[0], 1u) + 1u == gridDim.x) {
            const uint32_t gave_up = dev_load(&cs.expired[0]);
            if (ch.status)
                __hip_atomic_store(ch.status, gave_up ? kChainTimeout : 0, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            for (int h = 0; h < kBarrierGroups; ++h) {
                dev_store(&cs.grp[h][0], 0u);
                for (int q = 0; q < kBarrierGroups; ++q) dev_store(&cs.arrived[h][q], 0u);
            }
            // an abandoned launch may leave tiles half counted
            if (gave_up)
                for (uint32_t h = 0; h < gridDim.x; ++h) dev_store(counters + h, 0u);
            dev_store(&cs.expired[0], 0u);
            dev_store(&cs.exit[0], 0u);
        }
    }
}

// ----------------------------------------------------- int4 projections
//
// The int4 records of a served file (Sec. 4.1, Sec. 4.3): 4-bit weights in
// groups of G = 128 along K with an fp16 scale and offset per group,
// w = scale * q + offset, q the unsigned nibble (element 2i in the low
// nibble of byte i).  The 4-bit output head (Sec. 4.4) has the same form
// with G = 64.  Per group the product is
//   sum_k w_k x_k = scale * sum_k q_k x_k + offset * sum_k x_k,
// so the nibbles go to fp16 unscaled and the group's scale and offset are
// applied once per lane and group.
//
// Layout: q [M][K/2] bytes, scale/offset [M][K/G][2] fp16, both row-major.
// A wave takes 2 rows and walks K in steps of 1024 weights, 16 per lane (8
// bytes of q per row, coalesced into 512-byte runs); two steps are loaded
// before either is used, so that a wave keeps 2 KB of q in flight.  Few rows
// per wave give many waves, which is what hides the memory latency (4 rows
// per wave ran 1.4-2.5x slower).  Nibble k of a dword and nibble k+4 become
// one fp16 pair with a single and-or against the bits of 1024.0 (giving
// 1024 + q exactly); the activation pairs are permuted to match, and 1024
// times the lane's activation sum is taken back out.  Lanes are added with a
// fixed butterfly, so results are deterministic and batch-invariant.

constexpr int kInt4Group = 128;
constexpr int kHead4Group = 64;
constexpr int kInt4RowsPerWave = 2;
constexpr int kInt4Waves = 4;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// one lane's 16 activations of batch row b at k0, paired (k, k+4) within each
// 8 to match the nibble pairs, and their sum
template <int B>
struct Int4X {
    uint32_t xp[B][8];
    float sx[B];
};

template <int B>
__device__ __forceinline__ void int4_load_x(Int4X<B>& a, const uint16_t* __restrict__ x, int K, int k0) {
#pragma unroll
    for (int bb = 0; bb < B; ++bb) {
        const uint4* xs = reinterpret_cast<const uint4*>(x + static_cast<size_t>(bb) * K + k0);
        const uint4 u = xs[0], v = xs[1];
        const uint32_t n[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};   // pairs (2i, 2i+1)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            // elements 8h..8h+7: natural pairs n[4h..4h+3]; wanted (e, e+4) for e = 0..3
            a.xp[bb][4 * h + 0] = __builtin_amdgcn_perm(n[4 * h + 2], n[4 * h + 0], 0x05040100u);
            a.xp[bb][4 * h + 1] = __builtin_amdgcn_perm(n[4 * h + 2], n[4 * h + 0], 0x07060302u);
            a.xp[bb][4 * h + 2] = __builtin_amdgcn_perm(n[4 * h + 3], n[4 * h + 1], 0x05040100u);
            a.xp[bb][4 * h + 3] = __builtin_amdgcn_perm(n[4 * h + 3], n[4 * h + 1], 0x07060302u);
        }
        float sacc = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) sacc = dot2(n[i], 0x3C003C00u, sacc);
        a.sx[bb] = sacc;
    }
}

// the rows' q words and group scale/offset at k0
struct Int4W {
    uint2 w[kInt4RowsPerWave];
    uint32_t so[kInt4RowsPerWave];
};

template <int G>
__device__ __forceinline__ void int4_load_w(Int4W& a, const uint8_t* __restrict__ q, const uint16_t* __restrict__ so,
                                            int M, int K, int r0, int k0) {
    const int groups = K / G;
#pragma unroll
    for (int r = 0; r < kInt4RowsPerWave; ++r) {
        const int row = min(r0 + r, M - 1);
        a.w[r] = *reinterpret_cast<const uint2*>(q + static_cast<size_t>(row) * (K >> 1) + (k0 >> 1));
        a.so[r] = *reinterpret_cast<const uint32_t*>(so + (static_cast<size_t>(row) * groups + k0 / G) * 2);
    }
}

template <int B>
__device__ __forceinline__ void int4_step(float (&acc)[kInt4RowsPerWave][B], const Int4W& a, const Int4X<B>& xa) {
#pragma unroll
    for (int r = 0; r < kInt4RowsPerWave; ++r) {
        const float sc = f16(static_cast<uint16_t>(a.so[r])), of = f16(static_cast<uint16_t>(a.so[r] >> 16));
        uint32_t np[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t d = h ? a.w[r].y : a.w[r].x;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                np[4 * h + e] = ((d >> (4 * e)) & 0x000F000Fu) | 0x64006400u;   // (1024 + q_e, 1024 + q_{e+4})
        }
#pragma unroll
        for (int bb = 0; bb < B; ++bb) {
            float dt = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) dt = dot2(np[i], xa.xp[bb][i], dt);
            // sum q x = dt - 1024 sx; times scale, plus offset * sx
            acc[r][bb] = fmaf(sc, fmaf(-1024.f, xa.sx[bb], dt), fmaf(of, xa.sx[bb], acc[r][bb]));
        }
    }
}

template <int B, int G>
__global__ __launch_bounds__(kInt4Waves * 64) void int4_gemv_kernel(const uint8_t* __restrict__ q,
                                                                   const uint16_t* __restrict__ so,
                                                                   const uint16_t* __restrict__ x,
                                                                   float* __restrict__ y, int M, int K) {
    const int lane = threadIdx.x & 63;
    const int wave = blockIdx.x * kInt4Waves + (threadIdx.x >> 6);
    const int r0 = wave * kInt4RowsPerWave;
    if (r0 >= M) return;
    float acc[kInt4RowsPerWave][B];
#pragma unroll
    for (int r = 0; r < kInt4RowsPerWave; ++r)
#pragma unroll
        for (int bb = 0; bb < B; ++bb) acc[r][bb] = 0.f;
    for (int k0 = 16 * lane; k0 < K; k0 += 2048) {
        // two steps' loads before either step's arithmetic (the second step
        // exists for every lane or for none when K is a multiple of 1024)
        const int k1 = k0 + 1024;
        const bool two = k1 < K;
        Int4W wa, wb;
        Int4X<B> xa, xb;
        int4_load_w<G>(wa, q, so, M, K, r0, k0);
        if (two) int4_load_w<G>(wb, q, so, M, K, r0, k1);
        int4_load_x<B>(xa, x, K, k0);
        if (two) int4_load_x<B>(xb, x, K, k1);
        int4_step<B>(acc, wa, xa);
        if (two) int4_step<B>(acc, wb, xb);
    }
#pragma unroll
    for (int r = 0; r < kInt4RowsPerWave; ++r)
#pragma unroll
        for (int bb = 0; bb < B; ++bb) {
            const float v = wave_sum(acc[r][bb]);
            if (lane == 0 && r0 + r < M) y[static_cast<size_t>(bb) * M + r0 + r] = v;
        }
}

// Large int4 launches: persistent 16-wave workgroups that stage the
// activations once, already in the form every step uses (for each batch row
// and 16-weight chunk: the eight permuted fp16 pairs and the chunk's sum), so
// that the steps read them from LDS instead of fetching the vector from L2
// for every pair of rows (that traffic was twice the weight stream).  Each
// wave then takes row pairs rg, rg + waves, ... of the launch.

constexpr int kInt4LdsWaves = 16;
constexpr int kInt4LdsThreads = kInt4LdsWaves * 64;
constexpr int kInt4LdsMaxBatch = 5;    // larger batches would spill at four waves per SIMD

// workgroups per CU of the persistent kernel: two at batch 1 (64 VGPRs),
// one above
inline int int4_lds_groups_per_cu(int B) { return B == 1 ? 2 : 1; }

// LDS bytes of the staged activations for K and B: [B][K/16][8] pairs, then
// [B][K/16] sums
__host__ __device__ constexpr size_t int4_lds_bytes(int K, int B) {
    return static_cast<size_t>(B) * (K / 16) * (8 * 4 + 4);
}

template <int B, int G>
__global__ __launch_bounds__(kInt4LdsThreads) __attribute__((amdgpu_waves_per_eu(B == 1 ? 8 : 4)))
void int4_gemv_lds_kernel(const uint8_t* __restrict__ q,
                                                                       const uint16_t* __restrict__ so,
                                                                       const uint16_t* __restrict__ x,
                                                                       float* __restrict__ y, int M, int K) {
    extern __shared__ uint4 s_x4[];
    uint32_t* s_xp = reinterpret_cast<uint32_t*>(s_x4);                 // [B][K/16][8]
    const int chunks = K / 16;
    float* s_sx = reinterpret_cast<float*>(s_xp + static_cast<size_t>(B) * chunks * 8);   // [B][K/16]
    for (int c = threadIdx.x; c < chunks; c += kInt4LdsThreads) {
        Int4X<B> a;
        int4_load_x<B>(a, x, K, 16 * c);
#pragma unroll
        for (int bb = 0; bb < B; ++bb) {
            uint4* d = reinterpret_cast<uint4*>(s_xp + (static_cast<size_t>(bb) * chunks + c) * 8);
            d[0] = make_uint4(a.xp[bb][0], a.xp[bb][1], a.xp[bb][2], a.xp[bb][3]);
            d[1] = make_uint4(a.xp[bb][4], a.xp[bb][5], a.xp[bb][6], a.xp[bb][7]);
            s_sx[bb * chunks + c] = a.sx[bb];
        }
    }
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const int pairs = (M + kInt4RowsPerWave - 1) / kInt4RowsPerWave;
    const int waves = gridDim.x * kInt4LdsWaves;
    for (int rg = blockIdx.x * kInt4LdsWaves + (threadIdx.x >> 6); rg < pairs; rg += waves) {
        const int r0 = rg * kInt4RowsPerWave;
        float acc[kInt4RowsPerWave][B];
#pragma unroll
        for (int r = 0; r < kInt4RowsPerWave; ++r)
#pragma unroll
            for (int bb = 0; bb < B; ++bb) acc[r][bb] = 0.f;
        for (int k0 = 16 * lane; k0 < K; k0 += 2048) {
            const int k1 = k0 + 1024;
            const bool two = k1 < K;
            Int4W wa, wb;
            Int4X<B> xa;
            int4_load_w<G>(wa, q, so, M, K, r0, k0);
            if (two) int4_load_w<G>(wb, q, so, M, K, r0, k1);
            auto lds_x = [&](Int4X<B>& a, int k) {
#pragma unroll
                for (int bb = 0; bb < B; ++bb) {
                    const uint4* sp = reinterpret_cast<const uint4*>(s_xp + (static_cast<size_t>(bb) * chunks + k / 16) * 8);
                    const uint4 u = sp[0], v = sp[1];
                    a.xp[bb][0] = u.x; a.xp[bb][1] = u.y; a.xp[bb][2] = u.z; a.xp[bb][3] = u.w;
                    a.xp[bb][4] = v.x; a.xp[bb][5] = v.y; a.xp[bb][6] = v.z; a.xp[bb][7] = v.w;
                    a.sx[bb] = s_sx[bb * chunks + k / 16];
                }
            };
            // each step's activations just before the step (one register set)
            lds_x(xa, k0);
            int4_step<B>(acc, wa, xa);
            if (two) {
                lds_x(xa, k1);
                int4_step<B>(acc, wb, xa);
            }
        }
#pragma unroll
        for (int r = 0; r < kInt4RowsPerWave; ++r)
#pragma unroll
            for (int bb = 0; bb < B; ++bb) {
                const float v = wave_sum(acc[r][bb]);
                if (lane == 0 && r0 + r < M) y[static_cast<size_t>(bb) * M + r0 + r] = v;
            }
    }
}

// ------------------------------------------------- activation rotation
//
// The online rotation of the activations (Sec. 3.1, Sec. 5.1): a randomized
// Hadamard transform, block by block.  For each block of n = 2^k elements,
//   out[j0 + i] = (1/sqrt n) sum_m H_n[i][m] s[j0 + m] x[j0 + m],
// H_n the Sylvester Hadamard matrix, s = -1 where the caller's sign bit is
// set.  A workgroup of T threads takes a segment of 4T elements of one
// batch row (T = 256 for n <= 1024, so a segment holds whole blocks; T = n/4
// above), four consecutive elements per thread.  The butterflies of strides
// 1 and 2 stay in the thread, strides up to 128 go through lane shuffles,
// larger ones through LDS.  fp32 throughout, rounded to fp16 at the end.

template <int T>
__global__ __launch_bounds__(T) void rotate_kernel(const uint16_t* __restrict__ x, const uint8_t* __restrict__ bits,
                                                   uint16_t* out, int K, int n, float scale) {
    __shared__ float s_v[4 * T];
    const int t = threadIdx.x;
    const long long row = blockIdx.y;
    const int k = blockIdx.x * (4 * T) + 4 * t;     // first element of this thread
    const bool live = k < K;                        // K is a multiple of 4 and of n
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (live) {
        const uint2 u = *reinterpret_cast<const uint2*>(x + row * K + k);
        const uint32_t sb = bits[k >> 3] >> (k & 7);   // k is a multiple of 4: four bits in one byte
        v[0] = f16(static_cast<uint16_t>(u.x));
        v[1] = f16(static_cast<uint16_t>(u.x >> 16));
        v[2] = f16(static_cast<uint16_t>(u.y));
        v[3] = f16(static_cast<uint16_t>(u.y >> 16));
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (sb >> e & 1u) v[e] = -v[e];
    }
    // strides 1 and 2: inside the thread
    {
        const float a0 = v[0] + v[1], a1 = v[0] - v[1], a2 = v[2] + v[3], a3 = v[2] - v[3];
        v[0] = a0;
        v[1] = a1;
        v[2] = a2;
        v[3] = a3;
        if (n > 2) {
            const float b0 = v[0] + v[2], b1 = v[1] + v[3], b2 = v[0] - v[2], b3 = v[1] - v[3];
            v[0] = b0;
            v[1] = b1;
            v[2] = b2;
            v[3] = b3;
        }
    }
    // strides 4 .. n/2: partner thread t ^ (h / 4); the thread whose bit is
    // set keeps the difference partner - own, the other the sum
    for (int h = 4; h < n; h <<= 1) {
        const int d = h >> 2;
        const bool hi = (t & d) != 0;
        float p[4];
        if (d < 64) {
#pragma unroll
            for (int e = 0; e < 4; ++e) p[e] = __shfl_xor(v[e], d, 64);
        } else {
            __syncthreads();                         // the previous exchange has been read
#pragma unroll
            for (int e = 0; e < 4; ++e) s_v[4 * t + e] = v[e];
            __syncthreads();
#pragma unroll
            for (int e = 0; e < 4; ++e) p[e] = s_v[4 * (t ^ d) + e];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = hi ? p[e] - v[e] : v[e] + p[e];
    }
    if (live) {
        uint2 o;
        o.x = static_cast<uint32_t>(f16_bits(v[0] * scale)) | static_cast<uint32_t>(f16_bits(v[1] * scale)) << 16;
        o.y = static_cast<uint32_t>(f16_bits(v[2] * scale)) | static_cast<uint32_t>(f16_bits(v[3] * scale)) << 16;
        *reinterpret_cast<uint2*>(out + row * K + k) = o;
    }
}

// ------------------------------------------------ 4-bit embedding rows
//
// One row of a 4-bit embedding table (Sec. 4.4): groups of 64 along the
// embedding dimension, fp16 scale and offset per group, same nibble order;
// out[k] = fl32(fl32(scale * q_k) + offset).  One thread per byte.

constexpr int kEmbGroup = 64;

__global__ __launch_bounds__(256) void emb4_gather_kernel(const uint8_t* __restrict__ q,
                                                          const uint16_t* __restrict__ so, int rows, int dim,
                                                          const int* __restrict__ tokens, int n,
                                                          float* __restrict__ out) {
    const int half = dim >> 1;
    for (long long i = blockIdx.x * static_cast<long long>(blockDim.x) + threadIdx.x;
         i < static_cast<long long>(n) * half; i += static_cast<long long>(gridDim.x) * blockDim.x) {
        const int tok_i = static_cast<int>(i / half), b = static_cast<int>(i - static_cast<long long>(tok_i) * half);
        const long long row = tokens[tok_i];
        const int k = 2 * b;
        float* o = out + static_cast<long long>(tok_i) * dim + k;
        if (row < 0 || row >= rows) {     // a token outside the table gives zeros
            o[0] = 0.f;
            o[1] = 0.f;
            continue;
        }
        const uint32_t v = q[row * half + b];
        const uint32_t sov =
            *reinterpret_cast<const uint32_t*>(so + (row * (dim / kEmbGroup) + k / kEmbGroup) * 2);
        const float sc = f16(static_cast<uint16_t>(sov)), of = f16(static_cast<uint16_t>(sov >> 16));
        o[0] = __fadd_rn(__fmul_rn(sc, static_cast<float>(v & 15u)), of);
        o[1] = __fadd_rn(__fmul_rn(sc, static_cast<float>(v >> 4)), of);
    }
}

}  // namespace tetra_dev
