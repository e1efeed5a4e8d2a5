// Tetra matrix times many activation rows (a prompt, Sec. 6: the served
// model runs a prompt in one call): decode on the vector unit, products on
// the matrix cores.  Included by tetra.hip after kernels.h.
//
// y[n][row] = sigma_row * sum_blk s_blk * sum_j y_j x[n][24 blk + j]
//             + sum_t tail_t x[n][24 nblk + t]
//
// is the same sum as the GEMV's, and it is formed the same way: the decoded
// y_j stay exact integers in fp16, each block's 24-term products come from
// three v_mfma_f32_32x32x8_f16 (8 k each) and are scaled by that block's
// s_blk in fp32, sigma and the tail are applied at the end.
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
// A workgroup of 4 waves covers one 64-row tile (two 32-row halves) and 128
// tokens (two 64-token halves, two 32-token MFMA groups per wave).  The
// activations of the 128 tokens go through LDS in chunks of 96 k (one group
// of four block columns), the decoder tables are staged as in the GEMV.
#pragma once

namespace tetra_dev {

constexpr int kPfTokens = 128;             // tokens per workgroup
constexpr int kPfWaves = 4;
constexpr int kPfThreads = kPfWaves * 64;
constexpr int kPfChunk = 96;               // k per chunk: four blocks
constexpr int kPfXStride = 104;            // fp16 per token row of the LDS chunk (96 + 8)

struct GemmArgs {
    const uint8_t* codes;
    const uint16_t* sigma;
    const uint16_t* x;                     // [N][K] fp16
    float* y;                              // [N][M]
    unsigned long long tail_off;
    int M, K, N, nblk, T, ng, rem;
};

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

// finish a block from its table entries: this lane's half of the values (the
// B operand) and the block scale
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
    return o;
}

// this lane's A operand for a block and 8-k step: token row tok of the LDS
// chunk, k = 24 blk + 8 kk + 4h
__device__ __forceinline__ half4_t pf_a(const _Float16* s_x, int tok, int blk, int kk, int h) {
    return *reinterpret_cast<const half4_t*>(s_x + tok * kPfXStride + 24 * blk + 8 * kk + 4 * h);
}

// a full chunk of the workgroup's activations (128 tokens x 96 k) in
// registers: six 16-byte pieces per thread, loaded while the previous chunk
// is being used and written to LDS after it
constexpr int kPfPieces = kPfTokens * (kPfChunk / 8) / kPfThreads;
static_assert(kPfPieces * kPfThreads == kPfTokens * (kPfChunk / 8), "whole pieces per thread");

struct PfXRegs {
    uint4 v[kPfPieces];
};

__device__ __forceinline__ void pf_load_x(PfXRegs& r, const GemmArgs& a, int n0, int k0) {
#pragma unroll
    for (int i = 0; i < kPfPieces; ++i) {
        const int idx = static_cast<int>(threadIdx.x) + i * kPfThreads;
        const int tok = idx / (kPfChunk / 8), q = idx - tok * (kPfChunk / 8);
        const int n = min(n0 + tok, a.N - 1);                 // rows past N are loaded from row N-1, then zeroed
        r.v[i] = *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(n) * a.K + k0 + 8 * q);
        if (n0 + tok >= a.N) r.v[i] = make_uint4(0, 0, 0, 0);
    }
}

__device__ __forceinline__ void pf_store_x(_Float16* s_x, const PfXRegs& r) {
#pragma unroll
    for (int i = 0; i < kPfPieces; ++i) {
        const int idx = static_cast<int>(threadIdx.x) + i * kPfThreads;
        const int tok = idx / (kPfChunk / 8), q = idx - tok * (kPfChunk / 8);
        *reinterpret_cast<uint4*>(s_x + tok * kPfXStride + 8 * q) = r.v[i];
    }
}

// activations of the workgroup's tokens for k0 .. k0 + cols - 1 into LDS
// (zero for tokens past N); cols is a multiple of 8 and at most 96
__device__ __forceinline__ void pf_stage_x(_Float16* s_x, const GemmArgs& a, int n0, int k0, int cols) {
    const int per_tok = cols / 8;                        // 16-byte pieces per token
    for (int i = threadIdx.x; i < kPfTokens * per_tok; i += kPfThreads) {
        const int tok = i / per_tok, q = i - tok * per_tok;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (n0 + tok < a.N)
            v = *reinterpret_cast<const uint4*>(a.x + static_cast<size_t>(n0 + tok) * a.K + k0 + 8 * q);
        *reinterpret_cast<uint4*>(s_x + tok * kPfXStride + 8 * q) = v;
    }
}

__global__ __launch_bounds__(kPfThreads) void gemm_kernel(const GemmArgs a) {
    __shared__ uint4 s_tab[kPackedTableBytes / 16];
    __shared__ __attribute__((aligned(16))) _Float16 s_x[kPfTokens * kPfXStride];
    stage_packed_tables<kPfThreads>(s_tab);
    lds_bytes* L = (lds_bytes*)(s_tab);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int h = lane >> 5, jr = lane & 31;
    const int tile = blockIdx.x;
    const int n0 = blockIdx.y * kPfTokens;
    const int rin = (wave & 1) * 32 + jr;                 // row in the 64-row tile
    const int tok0 = (wave >> 1) * 64;                    // first of the wave's 64 tokens in the chunk
    const uint8_t* tb = a.codes + static_cast<size_t>(tile) * a.nblk * kChunk;
    float16_t acc[2];
#pragma unroll
    for (int tg = 0; tg < 2; ++tg)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[tg][e] = 0.f;

    auto issue = [&](uint32_t lo, uint32_t hi, int blk, PfFetch& pf) {
        pf.f = fetch_block(lo, hi, L);
#pragma unroll
        for (int tg = 0; tg < 2; ++tg)
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) pf.a[tg][kk] = pf_a(s_x, tok0 + 32 * tg + jr, blk, kk, h);
    };
    // blocks 0 .. nb-1 of the staged chunk (words lo[k], hi[k]) as a pipeline:
    // while a block's products run on the matrix cores, the next block's LDS
    // reads are in flight and its values are formed on the vector unit
    auto run_chunk = [&](const uint32_t (&lo)[4], const uint32_t (&hi)[4], int nb) {
        PfFetch nx;
        issue(lo[0], hi[0], 0, nx);
        PfBlock cur = pf_decode(nx.f, h, L);
        half4_t a[2][3];
#pragma unroll
        for (int tg = 0; tg < 2; ++tg)
#pragma unroll
            for (int kk = 0; kk < 3; ++kk) a[tg][kk] = nx.a[tg][kk];
        for (int blk = 0; blk < nb; ++blk) {
            const bool more = blk + 1 < nb;
            if (more) issue(lo[min(blk + 1, 3)], hi[min(blk + 1, 3)], blk + 1, nx);
            float16_t p[2];
#pragma unroll
            for (int tg = 0; tg < 2; ++tg) {
#pragma unroll
                for (int e = 0; e < 16; ++e) p[tg][e] = 0.f;
            }
#pragma unroll
            for (int kk = 0; kk < 3; ++kk)
#pragma unroll
                for (int tg = 0; tg < 2; ++tg)
                    p[tg] = __builtin_amdgcn_mfma_f32_32x32x8f16(a[tg][kk], cur.b[kk], p[tg], 0, 0, 0);
            PfBlock nxt;
            if (more) nxt = pf_decode(nx.f, h, L);
#pragma unroll
            for (int tg = 0; tg < 2; ++tg)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[tg][e] = fmaf(cur.s, p[tg][e], acc[tg][e]);
            if (more) {
                cur = nxt;
#pragma unroll
                for (int tg = 0; tg < 2; ++tg)
#pragma unroll
                    for (int kk = 0; kk < 3; ++kk) a[tg][kk] = nx.a[tg][kk];
            }
        }
    };

    // whole chunks: the next chunk's activations and code words are loaded
    // into registers while the current one runs
    if (a.ng > 0) {
        PfXRegs xr;
        pf_load_x(xr, a, n0, 0);
        uint4 l4 = *reinterpret_cast<const uint4*>(tb + 16 * rin);
        uint2 h2 = *reinterpret_cast<const uint2*>(tb + 1024 + 8 * rin);
        for (int g = 0; g < a.ng; ++g) {
            __syncthreads();                              // the previous chunk has been read
            pf_store_x(s_x, xr);
            __syncthreads();
            const uint32_t lo[4] = {l4.x, l4.y, l4.z, l4.w};
            const uint32_t hi[4] = {h2.x, h2.x >> 16, h2.y, h2.y >> 16};
            if (g + 1 < a.ng) {
                const uint8_t* gp = tb + static_cast<size_t>(g + 1) * tetra::kGroupBytes;
                pf_load_x(xr, a, n0, kPfChunk * (g + 1));
                l4 = *reinterpret_cast<const uint4*>(gp + 16 * rin);
                h2 = *reinterpret_cast<const uint2*>(gp + 1024 + 8 * rin);
            }
            run_chunk(lo, hi, 4);
        }
    }
    if (a.rem > 0) {
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
    // epilogue: sigma and the unquantised tail; this lane's row and 16 tokens
    // per group
    __syncthreads();
    // the tail columns of the tokens' activations, 4 bytes at a time (T is even)
    for (int i = threadIdx.x; i < kPfTokens * (a.T >> 1); i += kPfThreads) {
        const int tok = i / (a.T >> 1), q = i - tok * (a.T >> 1);
        uint32_t v = 0;
        if (n0 + tok < a.N)
            v = *reinterpret_cast<const uint32_t*>(a.x + static_cast<size_t>(n0 + tok) * a.K + 24 * a.nblk + 2 * q);
        *reinterpret_cast<uint32_t*>(s_x + tok * kPfXStride + 2 * q) = v;
    }
    __syncthreads();
    const int row = tile * kTile + rin;
    if (row >= a.M) return;
    const float sg = f16(a.sigma[row]);
    const uint32_t* tl = reinterpret_cast<const uint32_t*>(a.codes + a.tail_off) + static_cast<size_t>(row) * (a.T >> 1);
    uint32_t tv[11];
#pragma unroll
    for (int q = 0; q < 11; ++q) tv[q] = 2 * q < a.T ? tl[q] : 0u;
#pragma unroll
    for (int tg = 0; tg < 2; ++tg)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int tok = tok0 + 32 * tg + 8 * (e >> 2) + 4 * h + (e & 3);
            if (n0 + tok >= a.N) continue;
            const uint32_t* xt = reinterpret_cast<const uint32_t*>(s_x + tok * kPfXStride);
            float ts = 0.f;
#pragma unroll
            for (int q = 0; q < 11; ++q)
                if (2 * q < a.T) ts = dot2(tv[q], xt[q], ts);
            a.y[static_cast<size_t>(n0 + tok) * a.M + row] = fmaf(sg, acc[tg][e], ts);
        }
}

}  // namespace tetra_dev
