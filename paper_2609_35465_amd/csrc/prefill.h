// Tetra matrix times many activation rows (a prompt, Sec. 6: the served
// model runs a prompt in one call): decode on the vector unit, products on
// the matrix cores.  Included by tetra.hip after kernels.h.
//
// y[n][row] = sigma_row * sum_blk s_blk * sum_j y_j x[n][24 blk + j]
//             + sum_t tail_t x[n][24 nblk + t]
//
// is the same sum as the GEMV's.  The decoded
// y_j are exact integers in fp16; the block's scale is folded into them as
// fp16(s_blk y_j), rounded once from the fp32 product, so that three
// v_mfma_f32_32x32x8_f16 (8 k each) per block accumulate straight into the
// sums across blocks; sigma and the tail are applied at the end.  The fold
// costs one rounding of each weight to fp16: a relative error of at most
// 2^-11 per weight, so at most 2^-11 (4.9e-4) of sum |w x| per output, inside
// the 1e-3 bound of the products (the GEMV keeps the scale in fp32).  Folding
// replaced 16 fp32 multiply-adds per block and 32-token group (64 per block
// at four groups) by the fold's mixed-precision fmas (v_fma_mix: an fp16
// value times the fp32 scale, rounded once to fp16): 12 per block, against
// 30 for the conversions, multiplies and packs of a plain fp32 product.  The
// product is bound by latency, not issue: 82 -> 64 VALU instructions per
// block and wave left its time unchanged (250-253 TFLOP/s).
//
// MFMA roles: A = activations (32 tokens x 8 k), B = decoded weights (8 k x
// 32 rows), D = 32 tokens x 32 rows.  Lane l holds A[l % 32][4h..4h+3] and
// B[4h..4h+3][l % 32] with h = l / 32, and D[8g + 4h + r][l % 32] in
// register 4g + r.  So the lanes l and l + 32 of a wave both take row
// l % 32 of the wave's 32 rows: each decodes the 12 coordinates of a block
// that its half of the B operand needs (sections 0-2, coordinates 4h..4h+3),
// the two halves of the norm meet in one lane exchange, and both get the
// row's block scale, which then scales all 16 outputs of the lane (one row,
// 16 tokens).
//
// A workgroup of 4 waves takes 128 tokens and either two 64-row tiles (each
// wave 32 rows by all 128 tokens, four 32-token MFMA groups: every decoded
// block feeds twelve MFMAs) or one tile (each wave 32 rows by 64 tokens, two
// groups), chosen per launch (gemm_kernel<TG>).  The activations of the 128
// tokens go through LDS in chunks of 96 k (one group of four block columns),
// the decoder tables are staged as in the GEMV.
//
// Work split: an item is a (tile or tile pair, 128-token group) and a unit is
// one chunk of an item (the trailing block columns of a row make one more,
// shorter unit).  A fixed number of workgroups (two per CU, fewer for few
// items) take equal contiguous ranges of the items' units, so no launch
// leaves most of the chip idle in a last partial wave of workgroups, however
// many tiles and tokens there are.  An item whose units span several
// workgroups is combined as in the GEMV: each publishes its sums through the
// per-device workspace and the last to count in adds the pieces in workgroup
// order, which makes the result independent of timing.
#pragma once

namespace tetra_dev {

constexpr int kPfTokens = 128;             // tokens per workgroup
constexpr int kPfWaves = 4;
constexpr int kPfThreads = kPfWaves * 64;
constexpr int kPfChunk = 96;               // k per chunk: four blocks
constexpr int kPfXStride = 104;            // fp16 per token row of the LDS chunk (96 + 8)
constexpr int kPfGroupsPerCU = 2;          // 2 x 75 KB of LDS, 2 waves per SIMD

constexpr int kPfMaxTG = 4;                // 32-token MFMA groups per wave, at most
constexpr int kPfSlot = kPfThreads * 16 * kPfMaxTG;   // floats of one workgroup's piece of an item

struct GemmArgs {
    const uint8_t* codes;
    const uint16_t* sigma;
    const uint16_t* x;                     // [N][K] fp16
    float* y;                              // [N][M]
    unsigned long long tail_off;
    int M, K, N, nblk, T, ng, rem;
    int tgroups;                           // token groups of kPfTokens
    int tiles;                             // 64-row tiles
    int upi;                               // units per item: ng, plus one when rem > 0
    int workers;                           // workgroups of the launch
    unsigned long long units;              // items * upi
    uint32_t* counters;                    // [workers], zero between launches
    float* partials;                       // [workers][2][kPfSlot]
    int partial_bytes;                     // size of the partials array
};

// pieces go through the workspace in 16-byte buffer accesses with the cache
// policy of device-scope atomics (coherent across the chip's L2 caches):
// quad q of a thread's sums at byte 16 (256 q + thread) of its slot
typedef uint32_t pf_u32x4 __attribute__((ext_vector_type(4)));
constexpr int kPfCoherent = 16;            // sc1
constexpr int kPfRsrcWord3 = 0x00020000;   // raw 32-bit buffer, gfx9

__device__ __forceinline__ __amdgpu_buffer_rsrc_t pf_rsrc(const GemmArgs& a) {
    return __builtin_amdgcn_make_buffer_rsrc(a.partials, static_cast<short>(0), a.partial_bytes, kPfRsrcWord3);
}

// Values pass through these helpers by value: __builtin_bit_cast applied
// directly to a subscript of a vector (acc[tg][i], q[i]) was compiled as a
// cast of element 0 whatever i was.
__device__ __forceinline__ uint32_t pf_bits(float f) { return __builtin_bit_cast(uint32_t, f); }
__device__ __forceinline__ float pf_float(uint32_t u) { return __builtin_bit_cast(float, u); }

// component i (a constant) of a quad
__device__ __forceinline__ uint32_t pf_part(const pf_u32x4& v, int i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

__device__ __forceinline__ uint32_t pf_slot_bytes(int worker, int side) {
    return static_cast<uint32_t>((worker * 2 + side) * kPfSlot) * 4u;
}

// workspace of a launch with at most `workers` workgroups: the counters
// (rounded up to 256 bytes), then two piece slots per workgroup
inline size_t gemm_counter_bytes(int workers) {
    return (sizeof(uint32_t) * static_cast<size_t>(workers) + 255) & ~static_cast<size_t>(255);
}
inline size_t gemm_workspace_bytes(int workers) {
    return gemm_counter_bytes(workers) + sizeof(float) * static_cast<size_t>(workers) * 2 * kPfSlot;
}

// a workgroup-uniform 64-bit value in scalar registers (the 64-bit divisions
// below run on the vector unit, which would leave every index derived from
// them, and the loops they bound, in vector registers)
__device__ __forceinline__ unsigned long long pf_uniform(unsigned long long v) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(v >> 32));
    return (static_cast<unsigned long long>(hi) << 32) | lo;
}

// first unit of workgroup w's range (w = workers gives the end)
__device__ __forceinline__ unsigned long long pf_range_begin(int w, const GemmArgs& a) {
    return pf_uniform(a.units * static_cast<unsigned long long>(w) / static_cast<unsigned long long>(a.workers));
}

// the workgroup whose range holds unit u
__device__ __forceinline__ int pf_worker_of(unsigned long long u, const GemmArgs& a) {
    return __builtin_amdgcn_readfirstlane(
        static_cast<int>(((u + 1) * static_cast<unsigned long long>(a.workers) - 1) / a.units));
}

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float16_t __attribute__((ext_vector_type(16)));

// the B operand of a block (three 8-k steps, this lane's 4 coordinates of
// each) and the block's scale
struct PfBlock {
    half4_t b[3];
    float s;
};

// a block's LDS reads in flight: its table entries and this lane's A
// operands (two 32-token groups, three 8-k steps)
struct PfFetch {
    BlockFetch f;
    half4_t a[2][3];
};

// finish a block from its table entries: this lane's half of the values
// times the block scale (the B operand)
__device__ __forceinline__ PfBlock pf_decode(const BlockFetch& f, int h, lds_bytes* L) {
    const uint32_t ep = f.e ^ (~f.pm & 0xFCFCFCFCu);
    const uint32_t qpair = ~f.pm & 0x3C003C00u;
    PfBlock o;
    float sq = 0.f;
#pragma unroll
    for (int kk = 0; kk < 3; ++kk) {
        // coordinates 8 kk + 4h .. 8 kk + 4h + 3: sign group 2 kk + h, row word 2 kk + h
        const int w = 2 * kk + h;
        const uint32_t rw = h ? f.r[2 * kk + 1] : f.r[2 * kk];
        const uint32_t sg = rw ^ ((ep << w) & 0x80808080u);
        const uint32_t p0 = pk_add(cvt_pair<false>(sg), qpair);
        const uint32_t p1 = pk_add(cvt_pair<true>(sg), qpair);
        sq = dot2(p0, p0, sq);
        sq = dot2(p1, p1, sq);
        const uint2 u = make_uint2(p0, p1);
        o.b[kk] = __builtin_bit_cast(half4_t, u);
    }
    // the other half's squares (exact integers), then the scale as in the GEMV
    sq += __shfl_xor(sq, 32, 64);
    const float sqb = __builtin_bit_cast(float, f.bias) + sq;
    o.s = *(lds_f32*)(L + kScaleOff + ((__builtin_bit_cast(uint32_t, sqb) >> 2) & 0x7FFu));
#pragma unroll
    for (int kk = 0; kk < 3; ++kk)
#pragma unroll
        for (int i = 0; i < 4; ++i) o.b[kk][i] = static_cast<_Float16>(__builtin_fmaf(static_cast<float>(o.b[kk][i]), o.s, 0.0f));
    return o;
}

// this lane's A operand for a block and 8-k step: token row tok of the LDS
// chunk, k = 24 blk + 8 kk + 4h
__device__ __forceinline__ half4_t pf_a(const _Float16* s_x, int tok, int blk, int kk, int h) {
    return *reinterpret_cast<const half4_t*>(s_x + tok * kPfXStride + 24 * blk + 8 * kk + 4 * h);
}

// this thread's index in the workgroup, read afresh at each use: an index
// derived from threadIdx once would stay in a register across the whole
// item loop
__device__ __forceinline__ int pf_tid() {
    return (__builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x)) & ~63) | lane_now();
}

// a full chunk of the workgroup's activations (128 tokens x 96 k) in
// registers: six 16-byte pieces per thread, loaded while the previous chunk
// is being used and written to LDS after it
constexpr int kPfPieces = kPfTokens * (kPfChunk / 8) / kPfThreads;
static_assert(kPfPieces * kPfThreads == kPfTokens * (kPfChunk / 8), "whole pieces per thread");

// one 24-dword vector rather than an array of six uint4: the array form was
// placed in scratch memory across the item loop
typedef uint32_t pf_u24 __attribute__((ext_vector_type(4 * kPfPieces)));
struct PfXRegs {
    pf_u24 v;
};

// where this thread's pieces of every chunk of an item come from and go to:
// piece i is 16 bytes of token tok_i at k offset 8 q_i of the chunk.  Byte
// offsets from x for chunk 0 (32-bit: the entry point keeps N K 2 below
// 2^31) and into the LDS chunk.  Tokens past N read row N-1: their products
// only reach outputs that are never stored.
struct PfXMap {
    uint32_t g[kPfPieces];
    uint32_t l[kPfPieces];
};

__device__ __forceinline__ PfXMap pf_map(const GemmArgs& a, int n0) {
    PfXMap m;
    const int t = pf_tid();
#pragma unroll
    for (int i = 0; i < kPfPieces; ++i) {
        const int idx = t + i * kPfThreads;
        const int tok = idx / (kPfChunk / 8), q = idx - tok * (kPfChunk / 8);
        m.g[i] = static_cast<uint32_t>(min(n0 + tok, a.N - 1)) * static_cast<uint32_t>(2 * a.K) + 16u * q;
        m.l[i] = static_cast<uint32_t>(tok * (2 * kPfXStride) + 16 * q);
    }
    return m;
}

__device__ __forceinline__ void pf_load_x(PfXRegs& r, const GemmArgs& a, const PfXMap& m, int k0) {
    const uint8_t* base = reinterpret_cast<const uint8_t*>(a.x + k0);
#pragma unroll
    for (int i = 0; i < kPfPieces; ++i) {
        const uint4 t = *reinterpret_cast<const uint4*>(base + m.g[i]);
        r.v[4 * i] = t.x;
        r.v[4 * i + 1] = t.y;
        r.v[4 * i + 2] = t.z;
        r.v[4 * i + 3] = t.w;
    }
}

__device__ __forceinline__ void pf_store_x(_Float16* s_x, const PfXRegs& r, const PfXMap& m) {
#pragma unroll
    for (int i = 0; i < kPfPieces; ++i)
        *reinterpret_cast<uint4*>(reinterpret_cast<uint8_t*>(s_x) + m.l[i]) =
            make_uint4(r.v[4 * i], r.v[4 * i + 1], r.v[4 * i + 2], r.v[4 * i + 3]);
}

// activations of the workgroup's tokens for k0 .. k0 + cols - 1 into LDS
// (zero for tokens past N); cols is a multiple of 8 and at most 96
__device__ __forceinline__ void pf_stage_x(_Float16* s_x, const GemmArgs& a, int n0, int k0, int cols) {
    const int per_tok = cols / 8;                        // 16-byte pieces per token
    for (int i = pf_tid(); i < kPfTokens * per_tok; i += kPfThreads) {
        const int tok = i / per_tok, q = i - tok * per_tok;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (n0 + tok < a.N)
            v = *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(n0 + tok) * a.K + k0 + 8 * q);
        *reinterpret_cast<uint4*>(s_x + tok * kPfXStride + 8 * q) = v;
    }
}

// TG = 4: an item is two tiles (128 rows) by 128 tokens and each wave takes
// 32 rows by all 128 tokens, so that every decoded block feeds four token
// groups.  TG = 2: an item is one tile by 128 tokens, each wave 32 rows by
// 64 tokens; items are then half the size, for shapes with few rows, whose
// items would otherwise be cut into many pieces.
template <int TG>
__global__ __launch_bounds__(kPfThreads) __attribute__((amdgpu_waves_per_eu(2))) void gemm_kernel(const GemmArgs a) {
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    __shared__ __attribute__((aligned(16))) _Float16 s_x[kPfTokens * kPfXStride];
    __shared__ uint32_t s_arrived;
    stage_packed_tables<kPfThreads>(s_tab);
    lds_bytes* L = (lds_bytes*)(s_tab);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5, jr = lane & 31;
    const int rin = (wave & 1) * 32 + jr;                 // row in the wave's 64-row tile
    const int tok0 = TG == 4 ? 0 : (wave >> 1) * 64;      // first of the wave's tokens in the chunk
    const int w = blockIdx.x;
    float16_t acc[TG];

    // the A operands of 32-token groups tg0, tg0 + 1 for a block
    auto load_a = [&](int blk, int tg0, half4_t (&av)[2][3]) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) av[q][kk] = pf_a(s_x, tok0 + 32 * (tg0 + q) + jr, blk, kk, h);
    };
    auto issue = [&](uint32_t lo, uint32_t hi, int blk, PfFetch& pf) {
        pf.f = fetch_block(lo, hi, L);
        load_a(blk, 0, pf.a);
    };
    // blocks 0 .. nb-1 of the staged chunk (words lo[k], hi[k]) as a pipeline:
    // while a block's products run on the matrix cores, the next block's LDS
    // reads are in flight and its values are formed on the vector unit.  The
    // four token groups go in two pairs; the second pair's activations are
    // read while the first pair's products run.
    auto run_chunk = [&](const uint32_t (&lo)[4], const uint32_t (&hi)[4], int nb) {
        PfFetch nx;
        issue(lo[0], hi[0], 0, nx);
        PfBlock cur = pf_decode(nx.f, h, L);
        half4_t a01[2][3];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) a01[q][kk] = nx.a[q][kk];
        for (int blk = 0; blk < nb; ++blk) {
            const bool more = blk + 1 < nb;
            if (more) issue(lo[min(blk + 1, 3)], hi[min(blk + 1, 3)], blk + 1, nx);
#pragma unroll
            for (int kk = 0; kk < 3; ++kk)
#pragma unroll
                for (int q = 0; q < 2; ++q)
                    acc[q] = __builtin_amdgcn_mfma_f32_32x32x8f16(a01[q][kk], cur.b[kk], acc[q], 0, 0, 0);
            half4_t a23[2][3];
            if constexpr (TG == 4) load_a(blk, 2, a23);
            PfBlock nxt;
            if (more) nxt = pf_decode(nx.f, h, L);
            if constexpr (TG == 4) {
#pragma unroll
                for (int kk = 0; kk < 3; ++kk)
#pragma unroll
                    for (int q = 0; q < 2; ++q)
                        acc[2 + q] = __builtin_amdgcn_mfma_f32_32x32x8f16(a23[q][kk], cur.b[kk], acc[2 + q], 0, 0, 0);
            }
            if (more) {
                cur = nxt;
#pragma unroll
                for (int q = 0; q < 2; ++q)
#pragma unroll
                    for (int kk = 0; kk < 3; ++kk) a01[q][kk] = nx.a[q][kk];
            }
        }
    };
    // sigma and the unquantised tail applied to an item's sums v for the
    // wave's tile wt (only when it holds rows); this lane's row, 16 tokens per
    // group
    auto finish = [&](const float16_t (&v)[TG], int wt, bool live, int n0) {
        // lane indices read afresh: derived from threadIdx they would be
        // computed once for all items and held in registers throughout
        const int ln = lane_now();
        const int fh = ln >> 5;
        const int frin = (__builtin_amdgcn_readfirstlane(threadIdx.x) & 64) / 2 + (ln & 31);
        const int ftok0 = TG == 4 ? 0 : (__builtin_amdgcn_readfirstlane(threadIdx.x) & 128) / 2;
        __syncthreads();
        // the tail columns of the tokens' activations, 4 bytes at a time (T is even)
        for (int i = pf_tid(); i < kPfTokens * (a.T >> 1); i += kPfThreads) {
            const int tok = i / (a.T >> 1), q = i - tok * (a.T >> 1);
            uint32_t xv = 0;
            if (n0 + tok < a.N)
                xv = *reinterpret_cast<const uint32_t*>(a.x + static_cast<size_t>(n0 + tok) * a.K + 24 * a.nblk +
                                                        2 * q);
            *reinterpret_cast<uint32_t*>(s_x + tok * kPfXStride + 2 * q) = xv;
        }
        __syncthreads();
        const int row = wt * kTile + frin;
        if (live && row < a.M) {
            const float sg = f16(a.sigma[row]);
            const uint32_t* tl =
                reinterpret_cast<const uint32_t*>(a.codes + a.tail_off) + static_cast<size_t>(row) * (a.T >> 1);
            uint32_t tv[11];
#pragma unroll
            for (int q = 0; q < 11; ++q) tv[q] = 2 * q < a.T ? tl[q] : 0u;
#pragma unroll
            for (int tg = 0; tg < TG; ++tg)
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int tok = ftok0 + 32 * tg + 8 * (e >> 2) + 4 * fh + (e & 3);
                    if (n0 + tok >= a.N) continue;
                    const uint32_t* xt = reinterpret_cast<const uint32_t*>(s_x + tok * kPfXStride);
                    float ts = 0.f;
#pragma unroll
                    for (int q = 0; q < 11; ++q)
                        if (2 * q < a.T) ts = dot2(tv[q], xt[q], ts);
                    a.y[static_cast<size_t>(n0 + tok) * a.M + row] = fmaf(sg, v[tg][e], ts);
                }
        }
    };

    const unsigned long long u0 = pf_range_begin(w, a), u1 = pf_range_begin(w + 1, a);
    for (unsigned long long base = pf_uniform(u0 - u0 % a.upi); base < u1; base += a.upi) {
        // this workgroup's units c0 .. c1-1 of the item starting at unit base
        const int item = __builtin_amdgcn_readfirstlane(static_cast<int>(base / a.upi));
        const int c0 = __builtin_amdgcn_readfirstlane(static_cast<int>((u0 > base ? u0 : base) - base));
        const int c1 = __builtin_amdgcn_readfirstlane(static_cast<int>((u1 < base + a.upi ? u1 : base + a.upi) - base));
        const int irow = item / a.tgroups;
        const int n0 = (item - irow * a.tgroups) * kPfTokens;
        // the wave's tile: with TG = 4 waves 0-1 take the item's first tile and
        // waves 2-3 the second (past the last tile they repeat it and store
        // nothing); with TG = 2 all four take the item's tile
        const int wt_raw =
            TG == 4 ? 2 * irow + (__builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x)) >> 7) : irow;
        const bool live = wt_raw < a.tiles;
        const int wt = min(wt_raw, a.tiles - 1);
        const uint8_t* tb = a.codes + static_cast<size_t>(wt) * a.nblk * kChunk;
#pragma unroll
        for (int tg = 0; tg < TG; ++tg)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[tg][e] = 0.f;

        // whole chunks: the next chunk's activations and code words are loaded
        // into registers while the current one runs
        const int g1 = min(c1, a.ng);
        if (c0 < g1) {
            const PfXMap xm = pf_map(a, n0);
            PfXRegs xr;
            pf_load_x(xr, a, xm, kPfChunk * c0);
            const uint8_t* gp0 = tb + static_cast<size_t>(c0) * tetra::kGroupBytes;
            uint4 l4 = *reinterpret_cast<const uint4*>(gp0 + 16 * rin);
            uint2 h2 = *reinterpret_cast<const uint2*>(gp0 + 1024 + 8 * rin);
            for (int g = c0; g < g1; ++g) {
                __syncthreads();                          // the previous chunk has been read
                pf_store_x(s_x, xr, xm);
                __syncthreads();
                const uint32_t lo[4] = {l4.x, l4.y, l4.z, l4.w};
                const uint32_t hi[4] = {h2.x, h2.x >> 16, h2.y, h2.y >> 16};
                if (g + 1 < g1) {
                    const uint8_t* gp = tb + static_cast<size_t>(g + 1) * tetra::kGroupBytes;
                    pf_load_x(xr, a, xm, kPfChunk * (g + 1));
                    l4 = *reinterpret_cast<const uint4*>(gp + 16 * rin);
                    h2 = *reinterpret_cast<const uint2*>(gp + 1024 + 8 * rin);
                }
                run_chunk(lo, hi, 4);
            }
        }
        if (a.rem > 0 && c1 == a.upi) {
            // the trailing columns: the words of row rin (word_loc gives them for
            // any lane's row)
            uint32_t lo[4], hi[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const tetra::WordLoc at = tetra::word_loc(a.nblk, rin, 4 * a.ng + min(k, a.rem - 1));
                lo[k] = *reinterpret_cast<const uint32_t*>(tb + at.lo_off);
                hi[k] = *reinterpret_cast<const uint16_t*>(tb + at.hi_off);
            }
            __syncthreads();
            pf_stage_x(s_x, a, n0, kPfChunk * a.ng, 24 * a.rem);
            __syncthreads();
            run_chunk(lo, hi, a.rem);
        }
        if (c0 == 0 && c1 == a.upi) {
            finish(acc, wt, live, n0);
            continue;
        }

        // a piece of an item that other workgroups share.  Slot 0 of a workgroup
        // holds the piece of the item where its range starts, slot 1 that of
        // the item where it ends.  The sums and the counters are accessed only
        // with device-scope atomics, coherent across the chip's L2 caches; the
        // wait orders each thread's sums before the barrier and the count.
        const __amdgpu_buffer_rsrc_t rs = pf_rsrc(a);
        {
            const uint32_t mine = pf_slot_bytes(w, u0 >= base ? 0 : 1) + 16u * static_cast<uint32_t>(pf_tid());
#pragma unroll
            for (int tg = 0; tg < TG; ++tg)
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const pf_u32x4 q = {pf_bits(acc[tg][4 * k]), pf_bits(acc[tg][4 * k + 1]),
                                        pf_bits(acc[tg][4 * k + 2]), pf_bits(acc[tg][4 * k + 3])};
                    __builtin_amdgcn_raw_buffer_store_b128(q, rs, mine + 16u * kPfThreads * (4 * tg + k), 0,
                                                           kPfCoherent);
                }
        }
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0)
        const int wf = pf_worker_of(base, a), wl = pf_worker_of(base + a.upi - 1, a);
        __syncthreads();
        if (threadIdx.x == 0)
            s_arrived = __hip_atomic_fetch_add(a.counters + wf, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __syncthreads();
        if (s_arrived != static_cast<uint32_t>(wl - wf)) continue;
        // the last piece in: add all of them in workgroup order (its own piece
        // too, read back like the others), PB pieces per round trip
        constexpr int PB = TG == 4 ? 2 : 4;
        const int side_wf = pf_range_begin(wf, a) >= base ? 0 : 1;
#pragma unroll
        for (int tg = 0; tg < TG; ++tg)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[tg][e] = 0.f;
        for (int v0 = wf; v0 <= wl; v0 += PB) {
            pf_u32x4 pv[PB][4 * TG];
#pragma unroll
            for (int u = 0; u < PB; ++u) {
                const int v = min(v0 + u, wl);          // past the last: the last again, not added
                const uint32_t src = pf_slot_bytes(v, v > wf ? 0 : side_wf) + 16u * static_cast<uint32_t>(pf_tid());
#pragma unroll
                for (int q = 0; q < 4 * TG; ++q)
                    pv[u][q] = __builtin_amdgcn_raw_buffer_load_b128(rs, src + 16u * kPfThreads * q, 0, kPfCoherent);
            }
#pragma unroll
            for (int u = 0; u < PB; ++u)
                if (v0 + u <= wl) {
#pragma unroll
                    for (int tg = 0; tg < TG; ++tg)
#pragma unroll
                        for (int e = 0; e < 16; ++e)
                            acc[tg][e] += pf_float(pf_part(pv[u][4 * tg + (e >> 2)], e & 3));
                }
        }
        if (threadIdx.x == 0) __hip_atomic_store(a.counters + wf, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        finish(acc, wt, live, n0);
    }
}

}  // namespace tetra_dev
