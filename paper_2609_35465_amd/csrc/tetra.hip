// Tetra decode and fused decode-GEMV for MI355X (gfx950), C ABI in
// include/tetra.h.
//
// Decode of one 48-bit word (Sec. 3.3-3.4, Fig. 4 of the paper):
//   * the 12 path bits (s8, b1, b2, b3) select one of the 4,096 paths of
//     the octad-order Golay trellis (Sec. 3.2); the three trellis reads of
//     Fig. 4 are flattened into one read of a 4,096-entry path table that
//     holds the three pattern bytes of each path (16 KiB in LDS; LDS on
//     gfx950 is 160 KiB, so the extra 14 KiB buys away the dependent read);
//   * three reads of the shared rank table give the rank vectors of the
//     sections: rows[2048 r + i1], the middle row through its own list
//     (first 1240 class-0 rows, then class-1 rows), and rows[2048 r3 + i3]
//     with r3 = p ^ r ^ delta (Eq. 3), delta = [i2 >= 1240];
//   * coordinate j of section s has offset o = p + 2 c_j and rank rho; its
//     value is the rho-th element of o + 4Z counted outward from zero with
//     the positive one first at equal magnitude, which equals
//         (2p-1)(1-2c_j)(-1)^rho (2 rho + 1) + (1-p)
//     (checked for every o in {0..3} and rho in {0..7});
//   * m = sum_j y_j^2 / 16 and s_blk = fl32(gain[g] * invnorm[m]) (Eq. 2).
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/tetra.h"
#include "tables.h"

namespace {

constexpr int kTile = TETRA_ROW_TILE;        // rows per code tile (= wave size)
constexpr int kChunk = kTile * 6;            // bytes per (tile, block column) chunk
constexpr int kWaves = 4;                    // waves per workgroup
constexpr int kThreads = kWaves * 64;

// ---------------------------------------------------------------- tables

struct DeviceTables {
    uint32_t path_bytes[4096];
    uint32_t rows[4096];
    float invnorm[32];
    float gain[2];
    uint32_t pad[2];
};

__device__ DeviceTables g_tables;

constexpr int kMaxDevices = 64;
std::mutex g_init_mu;
bool g_init_done[kMaxDevices];

int ensure_tables(int* dev_out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TETRA_EDEVICE;
    *dev_out = dev;
    std::lock_guard<std::mutex> lk(g_init_mu);
    if (g_init_done[dev]) return TETRA_OK;
    const tetra::HostTables* T = nullptr;
    try {
        T = &tetra::host_tables();
    } catch (...) {
        return TETRA_EDEVICE;
    }
    DeviceTables h;
    std::memset(&h, 0, sizeof(h));
    std::memcpy(h.path_bytes, T->path_bytes, sizeof(h.path_bytes));
    std::memcpy(h.rows, T->rows, sizeof(h.rows));
    std::memcpy(h.invnorm, T->invnorm, sizeof(h.invnorm));
    std::memcpy(h.gain, T->gain, sizeof(h.gain));
    if (hipMemcpyToSymbol(HIP_SYMBOL(g_tables), &h, sizeof(h), 0, hipMemcpyHostToDevice) != hipSuccess)
        return TETRA_EDEVICE;
    g_init_done[dev] = true;
    return TETRA_OK;
}

// ------------------------------------------------------------ block decode

struct BlockCode {
    uint32_t pat;        // P1 | P2 << 8 | P3 << 16
    uint32_t rho[3];     // rank rows of the three sections
    uint32_t p, g;
};

__device__ __forceinline__ BlockCode read_code(uint32_t lo, uint32_t hi, const uint32_t* path_bytes,
                                               const uint32_t* rows) {
    BlockCode bc;
    const uint32_t s8 = lo & 63u;
    const uint32_t p = lo >> 6 & 1u;
    const uint32_t r = lo >> 7 & 1u;
    const uint32_t edges = lo >> 8 & 63u;          // b1 | b2 << 1 | b3 << 5
    bc.g = lo >> 14 & 1u;
    const uint32_t i1 = lo >> 15 & 2047u;
    const uint32_t i2 = (lo >> 26 | hi << 6) & 2047u;
    const uint32_t i3 = hi >> 5 & 2047u;
    bc.pat = path_bytes[s8 | edges << 6];
    const uint32_t delta = i2 >= 1240u ? 1u : 0u;
    const uint32_t mid = i2 + (delta ? 2048u - 1240u : 0u);
    const uint32_t r3 = p ^ r ^ delta;
    bc.rho[0] = rows[r << 11 | i1];
    bc.rho[1] = rows[mid];
    bc.rho[2] = rows[r3 << 11 | i3];
    bc.p = p;
    return bc;
}

// value of coordinate t of section s
__device__ __forceinline__ int coord_value(const BlockCode& bc, int s, int t) {
    const uint32_t c = bc.pat >> (8 * s + t) & 1u;
    const uint32_t rho = bc.rho[s] >> (4 * t) & 15u;
    const int u = static_cast<int>(2 * rho + 1);
    const uint32_t neg = (rho ^ c ^ bc.p ^ 1u) & 1u;
    return (neg ? -u : u) + static_cast<int>(1u - bc.p);
}

__device__ __forceinline__ void load_tables_to_lds(uint32_t* s_path, uint32_t* s_rows, float* s_inv,
                                                   float* s_gain) {
    for (int i = threadIdx.x; i < 4096; i += blockDim.x) {
        s_path[i] = g_tables.path_bytes[i];
        s_rows[i] = g_tables.rows[i];
    }
    if (threadIdx.x < 32) s_inv[threadIdx.x] = g_tables.invnorm[threadIdx.x];
    if (threadIdx.x < 2) s_gain[threadIdx.x] = g_tables.gain[threadIdx.x];
    __syncthreads();
}

// ------------------------------------------------------------ decode kernel

__global__ __launch_bounds__(256) void decode_kernel(const uint16_t* __restrict__ words, size_t n,
                                                     int8_t* __restrict__ y_out,
                                                     float* __restrict__ scale_out) {
    __shared__ uint32_t s_path[4096], s_rows[4096];
    __shared__ float s_inv[32], s_gain[2];
    load_tables_to_lds(s_path, s_rows, s_inv, s_gain);
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
         i += (size_t)gridDim.x * blockDim.x) {
        const uint32_t lo = words[3 * i] | static_cast<uint32_t>(words[3 * i + 1]) << 16;
        const uint32_t hi = words[3 * i + 2];
        const BlockCode bc = read_code(lo, hi, s_path, s_rows);
        int sq = 0;
        uint32_t packed[6];
        for (int q = 0; q < 6; ++q) {
            uint32_t v = 0;
            for (int e = 0; e < 4; ++e) {
                const int j = 4 * q + e;
                const int yv = coord_value(bc, j >> 3, j & 7);
                sq += yv * yv;
                v |= (static_cast<uint32_t>(yv) & 0xFFu) << (8 * e);
            }
            packed[q] = v;
        }
        uint32_t* yo = reinterpret_cast<uint32_t*>(y_out + 24 * i);
        for (int q = 0; q < 6; ++q) yo[q] = packed[q];
        if (scale_out) scale_out[i] = s_gain[bc.g] * s_inv[(sq >> 4) & 31];
    }
}

// ----------------------------------------------------------- dequant kernel

__global__ __launch_bounds__(256) void dequant_kernel(const uint8_t* __restrict__ codes,
                                                      const uint16_t* __restrict__ sigma, int M,
                                                      int K, int nblk, int T, size_t tail_off,
                                                      float* __restrict__ w_out) {
    __shared__ uint32_t s_path[4096], s_rows[4096];
    __shared__ float s_inv[32], s_gain[2];
    load_tables_to_lds(s_path, s_rows, s_inv, s_gain);
    const int lane = threadIdx.x & 63;
    const int tiles = (M + kTile - 1) / kTile;
    const size_t units = static_cast<size_t>(tiles) * nblk;       // (tile, column) chunks
    const size_t wave0 = (blockIdx.x * (size_t)blockDim.x + threadIdx.x) >> 6;
    const size_t nwaves = (gridDim.x * (size_t)blockDim.x) >> 6;
    for (size_t u = wave0; u < units; u += nwaves) {
        const int tile = static_cast<int>(u / nblk);
        const int b = static_cast<int>(u % nblk);
        const int row = tile * kTile + lane;
        const uint8_t* chunk = codes + u * kChunk;
        const uint32_t lo = reinterpret_cast<const uint32_t*>(chunk)[lane];
        const uint32_t hi = reinterpret_cast<const uint16_t*>(chunk + 4 * kTile)[lane];
        if (row >= M) continue;
        const BlockCode bc = read_code(lo, hi, s_path, s_rows);
        int yv[24];
        int sq = 0;
        for (int j = 0; j < 24; ++j) {
            yv[j] = coord_value(bc, j >> 3, j & 7);
            sq += yv[j] * yv[j];
        }
        const float sblk = s_gain[bc.g] * s_inv[(sq >> 4) & 31];
        const float sg = static_cast<float>(__builtin_bit_cast(_Float16, sigma[row]));
        float* wo = w_out + static_cast<size_t>(row) * K + 24 * b;
        for (int j = 0; j < 24; ++j) {
            const float a = __fmul_rn(static_cast<float>(yv[j]), sblk);
            wo[j] = __fmul_rn(a, sg);
        }
    }
    // tail weights
    const uint16_t* tail = reinterpret_cast<const uint16_t*>(codes + tail_off);
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < static_cast<size_t>(M) * T;
         i += (size_t)gridDim.x * blockDim.x) {
        const size_t row = i / T, t = i % T;
        w_out[row * K + 24 * nblk + t] = static_cast<float>(__builtin_bit_cast(_Float16, tail[i]));
    }
}

// -------------------------------------------------------------- GEMV kernel
//
// One lane per output row, 64 rows per tile; the four waves of a workgroup
// split the block columns of a tile and combine their partial sums in LDS.
// The activation slice of a block column is the same for every lane of a
// wave, so it is read through the scalar path.  Workgroups are persistent
// over tiles so the decoder tables are staged into LDS once.

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

template <int B>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const uint8_t* __restrict__ codes,
                                                        const uint16_t* __restrict__ sigma,
                                                        const uint16_t* __restrict__ x,
                                                        float* __restrict__ y, int M, int K,
                                                        int nblk, int T, size_t tail_off) {
    __shared__ uint32_t s_path[4096], s_rows[4096];
    __shared__ float s_inv[32], s_gain[2];
    __shared__ float s_red[kWaves][B][64];
    load_tables_to_lds(s_path, s_rows, s_inv, s_gain);

    const int wave = threadIdx.x >> 6;
    const int lane = threadIdx.x & 63;
    const int c0 = wave * nblk / kWaves, c1 = (wave + 1) * nblk / kWaves;
    const int tiles = (M + kTile - 1) / kTile;
    const uint32_t* x32 = reinterpret_cast<const uint32_t*>(x);   // fp16 pairs
    const int kpairs = K >> 1;

    for (int tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
        float acc[B];
        for (int bb = 0; bb < B; ++bb) acc[bb] = 0.f;
        for (int b = c0; b < c1; ++b) {
            const uint8_t* chunk = codes + (static_cast<size_t>(tile) * nblk + b) * kChunk;
            const uint32_t lo = reinterpret_cast<const uint32_t*>(chunk)[lane];
            const uint32_t hi = reinterpret_cast<const uint16_t*>(chunk + 4 * kTile)[lane];
            const BlockCode bc = read_code(lo, hi, s_path, s_rows);
            float dot[B];
            for (int bb = 0; bb < B; ++bb) dot[bb] = 0.f;
            int sq = 0;
#pragma unroll
            for (int k = 0; k < 12; ++k) {
                const int j0 = 2 * k;
                const int v0 = coord_value(bc, j0 >> 3, j0 & 7);
                const int v1 = coord_value(bc, (j0 + 1) >> 3, (j0 + 1) & 7);
                sq += v0 * v0 + v1 * v1;
                half2_t yv;
                yv.x = static_cast<_Float16>(v0);
                yv.y = static_cast<_Float16>(v1);
#pragma unroll
                for (int bb = 0; bb < B; ++bb) {
                    const uint32_t xp = x32[bb * kpairs + 12 * b + k];
                    dot[bb] = __builtin_amdgcn_fdot2(yv, __builtin_bit_cast(half2_t, xp), dot[bb], false);
                }
            }
            const float sblk = s_gain[bc.g] * s_inv[(sq >> 4) & 31];
#pragma unroll
            for (int bb = 0; bb < B; ++bb) acc[bb] = fmaf(sblk, dot[bb], acc[bb]);
        }
#pragma unroll
        for (int bb = 0; bb < B; ++bb) s_red[wave][bb][lane] = acc[bb];
        __syncthreads();
        if (wave == 0) {
            const int row = tile * kTile + lane;
            if (row < M) {
                const float sg = static_cast<float>(__builtin_bit_cast(_Float16, sigma[row]));
                const uint16_t* tail = reinterpret_cast<const uint16_t*>(codes + tail_off) +
                                       static_cast<size_t>(row) * T;
#pragma unroll
                for (int bb = 0; bb < B; ++bb) {
                    float tot = 0.f;
                    for (int w = 0; w < kWaves; ++w) tot += s_red[w][bb][lane];
                    float tsum = 0.f;
                    for (int t = 0; t < T; ++t)
                        tsum = fmaf(static_cast<float>(__builtin_bit_cast(_Float16, tail[t])),
                                    static_cast<float>(__builtin_bit_cast(
                                        _Float16, x[bb * K + 24 * nblk + t])),
                                    tsum);
                    y[static_cast<size_t>(bb) * M + row] = fmaf(sg, tot, tsum);
                }
            }
        }
        __syncthreads();
    }
}

// ----------------------------------------------------------------- helpers

struct Shape {
    int nblk, T, tiles;
    size_t code_bytes, tail_off, total;
};

bool shape_of(int M, int K, Shape* s) {
    if (M < 1 || K < 24 || (K & 1)) return false;
    s->nblk = K / 24;
    s->T = K % 24;
    s->tiles = (M + kTile - 1) / kTile;
    s->code_bytes = static_cast<size_t>(s->tiles) * s->nblk * kChunk;
    s->tail_off = (s->code_bytes + 15) & ~static_cast<size_t>(15);
    s->total = s->tail_off + static_cast<size_t>(M) * s->T * 2;
    return true;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

int num_cus() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return 256;
    return n;
}

int launch_status() { return hipGetLastError() == hipSuccess ? TETRA_OK : TETRA_EDEVICE; }

}  // namespace

// ================================================================== C ABI

extern "C" {

const char* tetra_status_string(int status) {
    switch (status) {
        case TETRA_OK: return "ok";
        case TETRA_EINVAL: return "invalid argument";
        case TETRA_EALIGN: return "misaligned device pointer";
        case TETRA_EDEVICE: return "HIP runtime error";
        case TETRA_EUNSUPPORTED: return "unsupported request";
        default: return "unknown status";
    }
}

int tetra_get_tables(void* out, size_t bytes) {
    if (!out || bytes < TETRA_TABLE_BLOB_BYTES) return TETRA_EINVAL;
    try {
        const std::vector<uint8_t> blob = tetra::canonical_blob();
        if (blob.size() != TETRA_TABLE_BLOB_BYTES) return TETRA_EDEVICE;
        std::memcpy(out, blob.data(), blob.size());
    } catch (...) {
        return TETRA_EDEVICE;
    }
    return TETRA_OK;
}

size_t tetra_codes_bytes(int M, int K) {
    Shape s;
    return shape_of(M, K, &s) ? s.total : 0;
}

size_t tetra_tail_offset(int M, int K) {
    Shape s;
    return shape_of(M, K, &s) ? s.tail_off : 0;
}

int tetra_pack_rows(const uint64_t* words, const uint16_t* tail, int M, int K, void* out,
                    size_t out_bytes) {
    Shape s;
    if (!words || !out || !shape_of(M, K, &s)) return TETRA_EINVAL;
    if (s.T > 0 && !tail) return TETRA_EINVAL;
    if (out_bytes < s.total) return TETRA_EINVAL;
    const size_t nw = static_cast<size_t>(M) * s.nblk;
    for (size_t i = 0; i < nw; ++i)
        if (words[i] >> 48) return TETRA_EINVAL;
    uint8_t* o = static_cast<uint8_t*>(out);
    std::memset(o, 0, s.total);
    for (int row = 0; row < M; ++row) {
        const int tile = row / kTile, r = row % kTile;
        for (int b = 0; b < s.nblk; ++b) {
            const uint64_t w = words[static_cast<size_t>(row) * s.nblk + b];
            uint8_t* chunk = o + (static_cast<size_t>(tile) * s.nblk + b) * kChunk;
            const uint32_t lo = static_cast<uint32_t>(w);
            const uint16_t hi = static_cast<uint16_t>(w >> 32);
            std::memcpy(chunk + 4 * r, &lo, 4);
            std::memcpy(chunk + 4 * kTile + 2 * r, &hi, 2);
        }
    }
    if (s.T > 0) std::memcpy(o + s.tail_off, tail, static_cast<size_t>(M) * s.T * 2);
    return TETRA_OK;
}

int tetra_unpack_rows(const void* codes, size_t codes_bytes, int M, int K, uint64_t* words,
                      uint16_t* tail) {
    Shape s;
    if (!codes || !words || !shape_of(M, K, &s) || codes_bytes < s.total) return TETRA_EINVAL;
    if (s.T > 0 && !tail) return TETRA_EINVAL;
    const uint8_t* c = static_cast<const uint8_t*>(codes);
    for (int row = 0; row < M; ++row) {
        const int tile = row / kTile, r = row % kTile;
        for (int b = 0; b < s.nblk; ++b) {
            const uint8_t* chunk = c + (static_cast<size_t>(tile) * s.nblk + b) * kChunk;
            uint32_t lo;
            uint16_t hi;
            std::memcpy(&lo, chunk + 4 * r, 4);
            std::memcpy(&hi, chunk + 4 * kTile + 2 * r, 2);
            words[static_cast<size_t>(row) * s.nblk + b] = lo | static_cast<uint64_t>(hi) << 32;
        }
    }
    if (s.T > 0) std::memcpy(tail, c + s.tail_off, static_cast<size_t>(M) * s.T * 2);
    return TETRA_OK;
}

int tetra_gemv(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M,
               int K, int batch, hipStream_t stream) {
    Shape s;
    if (!codes || !row_scales || !x || !y || !shape_of(M, K, &s)) return TETRA_EINVAL;
    if (batch < 1 || batch > TETRA_MAX_BATCH) return TETRA_EINVAL;
    if (!aligned(codes, 16) || !aligned(x, 4)) return TETRA_EALIGN;
    int dev;
    if (int st = ensure_tables(&dev)) return st;
    const int grid = std::min(s.tiles, num_cus() * 4);
    const uint8_t* c = static_cast<const uint8_t*>(codes);
#define TETRA_LAUNCH(B)                                                                          \
    case B:                                                                                      \
        hipLaunchKernelGGL(gemv_kernel<B>, dim3(grid), dim3(kThreads), 0, stream, c, row_scales, \
                           x, y, M, K, s.nblk, s.T, s.tail_off);                                 \
        break;
    switch (batch) {
        TETRA_LAUNCH(1) TETRA_LAUNCH(2) TETRA_LAUNCH(3) TETRA_LAUNCH(4)
        TETRA_LAUNCH(5) TETRA_LAUNCH(6) TETRA_LAUNCH(7) TETRA_LAUNCH(8)
        default: return TETRA_EINVAL;
    }
#undef TETRA_LAUNCH
    return launch_status();
}

int tetra_decode(const void* words, size_t n, int8_t* y_out, float* blk_scale_out,
                 hipStream_t stream) {
    if (!words || !y_out || n == 0) return TETRA_EINVAL;
    if (!aligned(words, 2) || !aligned(y_out, 4) || (blk_scale_out && !aligned(blk_scale_out, 4)))
        return TETRA_EALIGN;
    int dev;
    if (int st = ensure_tables(&dev)) return st;
    const size_t blocks = std::min<size_t>((n + 255) / 256, static_cast<size_t>(num_cus()) * 8);
    hipLaunchKernelGGL(decode_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(words), n, y_out, blk_scale_out);
    return launch_status();
}

int tetra_dequant(const void* codes, const uint16_t* row_scales, int M, int K, float* w_out,
                  hipStream_t stream) {
    Shape s;
    if (!codes || !row_scales || !w_out || !shape_of(M, K, &s)) return TETRA_EINVAL;
    if (!aligned(codes, 16) || !aligned(w_out, 4)) return TETRA_EALIGN;
    int dev;
    if (int st = ensure_tables(&dev)) return st;
    const size_t units = static_cast<size_t>(s.tiles) * s.nblk;
    const size_t blocks = std::min<size_t>((units + 3) / 4, static_cast<size_t>(num_cus()) * 8);
    hipLaunchKernelGGL(dequant_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       static_cast<const uint8_t*>(codes), row_scales, M, K, s.nblk, s.T,
                       s.tail_off, w_out);
    return launch_status();
}

}  // extern "C"
