// Nearest-point encoder of 24-weight blocks (the offline step of Sec. 3.1,
// run here on the GPU, one workgroup per block).  Included by tetra.hip
// after kernels.h.
//
// Shape-gain (Eq. 2): a block comes back as y / ||y|| * gain[g] * sigma, so
// the encoder wants the kept lattice point closest in direction to the
// block.  At each of two trial radii a it takes the kept point nearest to
// a w / ||w||, then keeps the trial point of better direction and the gain
// nearest to the block's projection on it.
//
// Nearest point at one radius.  With integer targets T_j = rint(w_j a 2^16 /
// ||w||) the point maximises S(y) = sum_j (2 T_j y_j - 2^16 y_j^2), an exact
// integer that splits over the three sections of Sec. 3.2:
//   * a section's score depends on the parity p, its pattern byte P (one of
//     the 128 even-weight bytes, named by its low seven bits) and its rank
//     row; for each (p, P, class) the best row of the section's list
//     (Sec. 3.3: the class halves of the table for sections 1 and 3, the
//     middle list for section 2) is kept, the first of equal scores.  A
//     thread scores one eighth of the rows for eight bytes that differ only
//     in bits 4-6 (bit 7 is their parity): the eight sums share the first
//     four coordinates and build on each other over the last four;
//   * the three are joined over the 4096 trellis paths and the parities r
//     and delta, with r3 = p xor r xor delta (Eq. 3); equal sums go to the
//     smallest key (s8 | p << 6 | r << 7 | b1 << 8 | b2 << 9 | b3 << 13) * 2
//     + delta, so the result does not depend on the order threads finish.
// The direction and gain choices are float64 sums in coordinate order on one
// thread: the same operations, in the same order, as any other
// implementation of this definition.
#pragma once

namespace tetra_dev {

constexpr int kEncThreads = 256;
constexpr int kEncScale = 1 << 16;
constexpr int kEncJoinKeys = 32768;                 // 4096 paths x p x r x delta
constexpr double kEncMaxRadius = 25.0;              // keeps every score inside int32

struct EncodeArgs {
    const float* w;                                 // [n][24], block order
    const float* sigma;                             // [n]
    uint16_t* words;                                // [n][3], canonical little-endian
    size_t n;
    double alpha[2];                                // trial radii
};

// value of rank rk in o + 4Z counted outward from zero, positive first at
// equal magnitude (o = p + 2c)
__device__ __forceinline__ int enc_value(int o, int rk) {
    const int p = o & 1, c = o >> 1;
    const int u = 2 * rk + 1;
    const int neg = (rk ^ c ^ p ^ 1) & 1;
    return (neg ? -u : u) + (1 - p);
}

// first (start, length) of the class-c list of section s, in table rows
__device__ __forceinline__ void enc_list(int s, int c, int* start, int* len) {
    if (s == 1) {
        *start = c ? 2048 : 0;
        *len = c ? 2048 - static_cast<int>(tetra::kMidClass0Rows) : static_cast<int>(tetra::kMidClass0Rows);
    } else {
        *start = c ? 2048 : 0;
        *len = 2048;
    }
}

__device__ __forceinline__ bool enc_better(int s, int k, int bs, int bk) { return s > bs || (s == bs && k < bk); }

__global__ __launch_bounds__(kEncThreads) void encode_kernel(const EncodeArgs a) {
    __shared__ uint32_t s_rows[4096];
    __shared__ uint32_t s_path[4096];
    __shared__ int s_E[24 * 4 * 8];                 // [j][o][rank]: 2 T_j v - 2^16 v^2
    __shared__ int s_best[3 * 2 * 128 * 2];         // [s][p][P & 127][c]
    __shared__ short s_arg[3 * 2 * 128 * 2];
    __shared__ int s_sl_s[8 * 32 * 8];              // [slice][p, low bits][high bits]: best score
    __shared__ short s_sl_i[8 * 32 * 8];            // and its row in the list
    __shared__ int s_red_s[kEncThreads / 64], s_red_k[kEncThreads / 64];
    __shared__ int s_T[24];
    __shared__ double s_f[2];
    __shared__ int s_zero;
    for (int i = threadIdx.x; i < 4096; i += kEncThreads) {
        s_rows[i] = g_canonical.rows[i];
        s_path[i] = g_canonical.path_bytes[i];
    }
    const int t = threadIdx.x;
    const int lane = t & 63, wave = t >> 6;
    // this thread's part of the section search: a slice of the rows, the
    // parity p and the low four bits of the pattern-byte index
    const int my_slice = t >> 5, my_combo = t & 31;
    const int my_p = my_combo >> 4, my_lo = my_combo & 15;
    const int my_par = __builtin_popcount(my_lo) & 1;
    for (size_t blk = blockIdx.x; blk < a.n; blk += gridDim.x) {
        const float* w = a.w + 24 * blk;
        __syncthreads();                            // tables staged; the previous block is done with LDS
        if (t == 0) {
            double n2 = 0.0;
            for (int j = 0; j < 24; ++j) n2 += static_cast<double>(w[j]) * static_cast<double>(w[j]);
            s_zero = !(n2 > 0.0) || !(n2 <= 1.0e300);
            const double rn = s_zero ? 1.0 : sqrt(n2);
            for (int q = 0; q < 2; ++q) s_f[q] = a.alpha[q] * static_cast<double>(kEncScale) / rn;
        }
        __syncthreads();
        if (s_zero) {
            if (t < 3) a.words[3 * blk + t] = 0;
            continue;
        }
        double best_c = 0.0;                        // thread 0's running choice over the trials
        uint32_t best_f[4] = {0, 0, 0, 0};          // key, i1, i2, i3
        for (int trial = 0; trial < 2; ++trial) {
            if (t < 24) s_T[t] = static_cast<int>(rint(static_cast<double>(w[t]) * s_f[trial]));
            __syncthreads();
            for (int i = t; i < 24 * 4 * 8; i += kEncThreads) {
                const int j = i >> 5, o = (i >> 3) & 3, rk = i & 7;
                const int v = enc_value(o, rk);
                s_E[i] = 2 * s_T[j] * v - kEncScale * v * v;
            }
            __syncthreads();
            // best row of each section's list per (p, P, class): thread t scans
            // slice t / 32 of the list for parity p and the eight pattern bytes
            // whose index has the low bits of t % 16; the slices then meet in
            // row order
            for (int sec = 0; sec < 3; ++sec) {
                const int* Ep = s_E + 256 * sec + 8 * my_p;      // E[j][p + 2x][r] at Ep[32 j + 16 x + r]
                for (int c = 0; c < 2; ++c) {
                    int start, len;
                    enc_list(sec, c, &start, &len);
                    const int i0 = (len * my_slice) >> 3, i1 = (len * (my_slice + 1)) >> 3;
                    int bs[8], bi[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        bs[k] = INT_MIN;
                        bi[k] = 0;
                    }
                    for (int i = i0; i < i1; ++i) {
                        const uint32_t row = s_rows[start + i];
                        int r[8];
#pragma unroll
                        for (int j = 0; j < 8; ++j) r[j] = static_cast<int>((row >> (4 * j)) & 15u);
                        int base = 0;
#pragma unroll
                        for (int j = 0; j < 4; ++j) base += Ep[32 * j + 16 * ((my_lo >> j) & 1) + r[j]];
                        int e[4][2];
#pragma unroll
                        for (int j = 0; j < 4; ++j) {
                            e[j][0] = Ep[32 * (4 + j) + r[4 + j]];
                            e[j][1] = Ep[32 * (4 + j) + 16 + r[4 + j]];
                        }
                        // coordinate 7 is the parity bit of the byte
                        const int f0 = my_par ? e[3][1] : e[3][0];
                        const int f1 = my_par ? e[3][0] : e[3][1];
                        int s4[2], s45[4];
#pragma unroll
                        for (int a4 = 0; a4 < 2; ++a4) s4[a4] = base + e[0][a4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) s45[q] = s4[q & 1] + e[1][q >> 1];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const int sc = s45[k & 3] + e[2][k >> 2] + ((__builtin_popcount(k) & 1) ? f1 : f0);
                            if (sc > bs[k]) {
                                bs[k] = sc;
                                bi[k] = i;
                            }
                        }
                    }
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        s_sl_s[(my_slice * 32 + my_combo) * 8 + k] = bs[k];
                        s_sl_i[(my_slice * 32 + my_combo) * 8 + k] = static_cast<short>(bi[k]);
                    }
                    __syncthreads();
                    {
                        // thread t: combination t / 8, byte k = t % 8, slices in row order
                        const int cb = t >> 3, k = t & 7;
                        int ws = INT_MIN, wi = 0;
                        for (int sl = 0; sl < 8; ++sl) {
                            const int v = s_sl_s[(sl * 32 + cb) * 8 + k];
                            if (v > ws) {
                                ws = v;
                                wi = s_sl_i[(sl * 32 + cb) * 8 + k];
                            }
                        }
                        const int pp = cb >> 4, i7 = (cb & 15) | (k << 4);
                        const int at = ((sec * 2 + pp) * 128 + i7) * 2 + c;
                        s_best[at] = ws;
                        s_arg[at] = static_cast<short>(wi);
                    }
                    __syncthreads();
                }
            }
            // join over the trellis: keys t, t + 256, ... in ascending order
            int js = INT_MIN, jk = 0;
            for (int k = t; k < kEncJoinKeys; k += kEncThreads) {
                const int d = k & 1, s8 = (k >> 1) & 63, p = (k >> 7) & 1, r = (k >> 8) & 1;
                const int b1 = (k >> 9) & 1, b2 = (k >> 10) & 15, b3 = (k >> 14) & 1;
                const uint32_t pb = s_path[s8 | b1 << 6 | b2 << 7 | b3 << 11];
                const int r3 = p ^ r ^ d;
                const int sc = s_best[((0 * 2 + p) * 128 + (pb & 127)) * 2 + r] +
                               s_best[((1 * 2 + p) * 128 + ((pb >> 8) & 127)) * 2 + d] +
                               s_best[((2 * 2 + p) * 128 + ((pb >> 16) & 127)) * 2 + r3];
                if (sc > js) {
                    js = sc;
                    jk = k;
                }
            }
            for (int off = 32; off > 0; off >>= 1) {
                const int os = __shfl_xor(js, off, 64), ok = __shfl_xor(jk, off, 64);
                if (enc_better(os, ok, js, jk)) {
                    js = os;
                    jk = ok;
                }
            }
            if (lane == 0) {
                s_red_s[wave] = js;
                s_red_k[wave] = jk;
            }
            __syncthreads();
            if (t == 0) {
                int ws = s_red_s[0], wk = s_red_k[0];
                for (int q = 1; q < kEncThreads / 64; ++q)
                    if (enc_better(s_red_s[q], s_red_k[q], ws, wk)) {
                        ws = s_red_s[q];
                        wk = s_red_k[q];
                    }
                // the trial's point, its row indices and its direction
                const int d = wk & 1, s8 = (wk >> 1) & 63, p = (wk >> 7) & 1, r = (wk >> 8) & 1;
                const int b1 = (wk >> 9) & 1, b2 = (wk >> 10) & 15, b3 = (wk >> 14) & 1;
                const uint32_t pb = s_path[s8 | b1 << 6 | b2 << 7 | b3 << 11];
                const int r3 = p ^ r ^ d;
                const uint32_t i1 = static_cast<uint16_t>(s_arg[((0 * 2 + p) * 128 + (pb & 127)) * 2 + r]);
                const uint32_t im = static_cast<uint16_t>(s_arg[((1 * 2 + p) * 128 + ((pb >> 8) & 127)) * 2 + d]);
                const uint32_t i3 = static_cast<uint16_t>(s_arg[((2 * 2 + p) * 128 + ((pb >> 16) & 127)) * 2 + r3]);
                const uint32_t rho[3] = {s_rows[r << 11 | i1], s_rows[d << 11 | im], s_rows[r3 << 11 | i3]};
                double dot = 0.0, yy = 0.0;
                for (int j = 0; j < 24; ++j) {
                    const int sec = j >> 3, q = j & 7;
                    const int o = p + 2 * static_cast<int>((pb >> (8 * sec + q)) & 1u);
                    const int v = enc_value(o, static_cast<int>((rho[sec] >> (4 * q)) & 15u));
                    dot += static_cast<double>(w[j]) * static_cast<double>(v);
                    yy += static_cast<double>(v) * static_cast<double>(v);
                }
                const double ny = sqrt(yy);
                const double cdir = ny > 0.0 ? dot / ny : -INFINITY;
                if (trial == 0 || cdir > best_c) {
                    best_c = cdir;
                    best_f[0] = static_cast<uint32_t>(wk);
                    best_f[1] = i1;
                    best_f[2] = d ? im + tetra::kMidClass0Rows : im;
                    best_f[3] = i3;
                }
            }
            __syncthreads();
        }
        if (t == 0) {
            // the gain nearest to the projection, then the canonical word
            const double gs = static_cast<double>(a.sigma[blk]);
            const double d0 = static_cast<double>(g_canonical.gain[0]) * gs - best_c;
            const double d1 = static_cast<double>(g_canonical.gain[1]) * gs - best_c;
            const uint64_t g = d1 * d1 < d0 * d0 ? 1u : 0u;
            const uint32_t k = best_f[0];
            const uint64_t s8 = (k >> 1) & 63, p = (k >> 7) & 1, r = (k >> 8) & 1;
            const uint64_t b1 = (k >> 9) & 1, b2 = (k >> 10) & 15, b3 = (k >> 14) & 1;
            const uint64_t word = s8 | p << 6 | r << 7 | b1 << 8 | b2 << 9 | b3 << 13 | g << 14 |
                                  static_cast<uint64_t>(best_f[1]) << 15 | static_cast<uint64_t>(best_f[2]) << 26 |
                                  static_cast<uint64_t>(best_f[3]) << 37;
            uint16_t* out = a.words + 3 * blk;
            out[0] = static_cast<uint16_t>(word);
            out[1] = static_cast<uint16_t>(word >> 16);
            out[2] = static_cast<uint16_t>(word >> 32);
        }
    }
}

}  // namespace tetra_dev
