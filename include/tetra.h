/*
 * tetra.h - C ABI of the MI355X (gfx950) Tetra decode and fused decode-GEMV.
 *
 * The method: each block of 24 weights is one 48-bit code (Sec. 3.3-3.4 and
 * Fig. 3-4 of "Tetra: Serving Leech-Lattice Quantized LLMs at 2.7 Bits per
 * Parameter").  A code names a path through the 64-state trellis of the
 * Golay code in octad order (Sec. 3.2), a shared parity p, the k-parity r of
 * section 1, a gain bit g and three 11-bit indices into one table of 4,096
 * rank vectors; the decoded block is a point y of the Leech lattice (Eq. 1)
 * and the weights are w_j = y_j / sqrt(16 m) * gain[g] * sigma_row (Eq. 2).
 * The fused product y = W x never writes W (Sec. 5.1).
 *
 * Conventions fixed by this library where the paper is silent (the word bit
 * layout, the trellis numbering, the rank-table tie-break, the value order
 * for o = 2 and the gain values) are the canonical ones returned by
 * tetra_get_tables().
 *
 * Canonical 48-bit word, stored as 6 little-endian bytes:
 *     bits 0-5 s8 | 6 p | 7 r | 8 b1 | 9-12 b2 | 13 b3 | 14 g |
 *     15-25 i1 | 26-36 i2 | 37-47 i3
 * Every 48-bit value is a legal word.
 *
 * Memory: all buffers are owned by the caller.  "host" arguments are plain
 * host pointers; "device" arguments are device pointers on the current HIP
 * device (for example from hipMalloc or torch.empty(..., device="cuda")).
 * No call allocates or frees memory, and none synchronises: the decoder
 * tables are constant data of the library's code object, built when the
 * library is built, and the GEMV workspaces (a counter and two partial sums
 * per workgroup) are static device memory in 16 slots per device.  A stream
 * takes a slot at its first GEMV call on a device and keeps it until
 * tetra_release_stream; GEMV calls on different streams therefore never
 * share a workspace and may run at the same time, and a 17th stream is
 * refused with TETRA_EBUSY.  The first call on a device (any call,
 * including one made while the stream is being captured into a graph) only
 * queries device attributes on the host.  tetra_gemm takes its workspace
 * from the caller.
 *
 * Errors: every call validates its arguments before any launch and returns
 * a tetra_status.  TETRA_EDEVICE reports a HIP error seen at launch time;
 * faults inside a kernel surface at the caller's next synchronisation.
 */
#ifndef TETRA_H
#define TETRA_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TETRA_OK = 0,
    TETRA_EINVAL = -1,       /* null pointer, size out of range, bad batch  */
    TETRA_EALIGN = -2,       /* a device pointer is not aligned as required */
    TETRA_EDEVICE = -3,      /* HIP runtime error (device query or launch)  */
    TETRA_EUNSUPPORTED = -4, /* valid request the library does not serve    */
    TETRA_EBUSY = -5,        /* all GEMV workspace slots held by other streams */
    TETRA_ETIMEOUT = -6      /* a wait between the phases of tetra_gemv_chain gave up */
} tetra_status;

/* Rows of one code tile of the device layout (see tetra_pack_rows). */
#define TETRA_ROW_TILE 64
/* Bytes of the canonical table blob returned by tetra_get_tables. */
#define TETRA_TABLE_BLOB_BYTES 18824
/* Largest batch (number of activation vectors) served by tetra_gemv. */
#define TETRA_MAX_BATCH 8

/* Message for a status code (static string, never NULL). */
const char* tetra_status_string(int status);

/*
 * Canonical decoder tables (Fig. 4; Sec. 3.3-3.4), little-endian:
 *   rows u32[4096] | branches u16[1024] | prefixes u8[128] |
 *   suffixes u8[128] | invnorm f32[32] | gain f32[2]
 * 16,384 + 2,048 + 128 + 128 + 128 + 8 = 18,824 bytes: the paper's
 * 18,816 B of rank rows, trellis tables and 1/sqrt(16m), plus the two gains.
 * rows: the 2,048 cheapest rank vectors of class 0 then of class 1
 * (nibble j = rank of section coordinate j).  branches[16*s8+b2] =
 * P2 | s16 << 8.  Host only; out: host buffer of at least
 * TETRA_TABLE_BLOB_BYTES.  Returns TETRA_EINVAL if out is NULL or bytes is
 * too small.
 */
int tetra_get_tables(void* out, size_t bytes);

/*
 * Size in bytes of the device code blob of an M x K Tetra matrix.
 * K splits into nblk = K / 24 code blocks and an unquantised tail of
 * T = K % 24 weights per row (Sec. 4.1).  Returns 0 if M < 1, K < 24 or K
 * is odd.
 */
size_t tetra_codes_bytes(int M, int K);

/*
 * Code bytes per row of an M x K matrix: 6 * (K / 24), 48 bits per block.
 * Rows are not stored one after another: the device layout interleaves
 * them in tiles of TETRA_ROW_TILE rows (see tetra_pack_rows), and tile t
 * starts at byte t * TETRA_ROW_TILE * tetra_row_stride(K).  Returns 0 if
 * K < 24 or K is odd.  Host only, pure.
 */
size_t tetra_row_stride(int K);

/* Byte offset of the fp16 tail inside the code blob (0 if the shape is
 * invalid): the code chunks rounded up to 16 bytes. */
size_t tetra_tail_offset(int M, int K);

/*
 * Host packer (the loader step of Sec. 5.1: it reorders code words, it
 * expands nothing).  words: host uint64[M][nblk], canonical words in the low
 * 48 bits (upper bits must be 0).  tail: host fp16 bits [M][T], may be NULL
 * iff T == 0.  out: host buffer of tetra_codes_bytes(M, K) bytes.
 *
 * Device layout (ours): rows are grouped in tiles of TETRA_ROW_TILE rows
 * (the last tile padded with the zero word, which decodes to the origin);
 * tile t occupies nblk*384 bytes starting at t*nblk*384.  Inside a tile,
 * with ng = nblk / 4 and r the row in the tile:
 *   - block columns 4g..4g+3 (g < ng) form a 1536-byte run at g*1536: the
 *     32-bit part of column 4g+k of row r at 16*r + 4*k, its 16-bit part at
 *     1024 + 8*r + 2*k (one 16-byte and one 8-byte load per row and group);
 *   - the s = nblk mod 4 remaining columns b = 4*ng + q (q < s) form one
 *     run of 384*s bytes at ng*1536: 32-bit part at 4*s*r + 4*q; 16-bit
 *     part at 256*s + 2*min(s,2)*r + 2*q for q < 2, and at 1024 + 2*r for
 *     q = 2 (a row reads its remaining words with whole loads).
 * Each word is stored recoded, still 48 bits and one-to-one
 * with the canonical word: path = s8 | b1<<6 | b2<<7 | b3<<11, g, the
 * physical rank-table row of section 1, i2, and section 3's physical row
 * without delta, (p^r)<<11 | i3' (rank rows of class 0 sit at
 * (i+808) mod 2048, of class 1 at 2048+i, so the middle list is 808+i2):
 *   lo32 = path | g<<12 | phys1<<13 | (i2 & 0x7F)<<25,
 *   hi16 = (i2 >> 7) | u3<<4.
 * The fp16 tail follows, row-major [M][T], at a 16-byte aligned offset.
 * Bits read per weight: 48 per block plus 16 per tail weight (plus the
 * fp16 row scale passed separately).
 * Returns TETRA_EINVAL on a NULL pointer, a bad shape, a word with bits
 * above 47 set, or out_bytes < tetra_codes_bytes(M, K).
 */
int tetra_pack_rows(const uint64_t* words, const uint16_t* tail, int M, int K,
                    void* out, size_t out_bytes);

/* Inverse of tetra_pack_rows (host only, for checks). */
int tetra_unpack_rows(const void* codes, size_t codes_bytes, int M, int K,
                      uint64_t* words, uint16_t* tail);

/*
 * Fused decode and matrix-vector product (Sec. 5.1, Eq. 2).  The blocks are
 * split evenly over the waves of the launch; pieces of a row tile held by
 * several waves are added in a fixed order, so y is deterministic.  The wave
 * count follows the shapes, the device and how many workgroups of the
 * batch's kernel a CU holds (on MI355X two for batch 1-2, one for 3-8).
 * Batches 1-2 form the per-block sums with VALU dot products, batches 3-8
 * on the matrix cores, which round differently; within each class the row
 * for activation b equals, bit for bit, the row of any other call of the
 * class for x_b (a grouped call may round differently from single calls):
 *   y[b][row] = sigma_row * sum_blk s_blk * sum_j y_j x[b][24*blk + j]
 *               + sum_t tail[row][t] * x[b][24*nblk + t]
 * with s_blk = gain[g] * (1/sqrt(16 m)) in f32 and f32 accumulation.
 *   codes:      device, tetra_pack_rows layout, 16-byte aligned
 *   row_scales: device fp16[M] (sigma_row)
 *   x:          device fp16[batch][K], 4-byte aligned
 *   y:          device fp32[batch][M], fully overwritten
 *   batch:      1..TETRA_MAX_BATCH
 * Uses the GEMV workspace slot of `stream` (see Memory above).
 * Asynchronous on stream.  TETRA_EINVAL for NULL pointers, bad M/K, batch
 * out of range; TETRA_EALIGN for misaligned codes or x; TETRA_EBUSY when the
 * stream has no slot and none is free; TETRA_EDEVICE when a device query or
 * the launch fails.
 */
int tetra_gemv(const void* codes, const uint16_t* row_scales, const uint16_t* x,
               float* y, int M, int K, int batch, hipStream_t stream);

/* Largest number of matrices in one tetra_gemv_grouped call. */
#define TETRA_MAX_GROUP 32

/* One matrix of a grouped product: arguments as in tetra_gemv. */
typedef struct {
    const void* codes;
    const uint16_t* row_scales;
    const uint16_t* x;
    float* y;
    int M, K;
} tetra_gemv_problem;

/*
 * Several independent Tetra products in one launch (for instance the q, k
 * and v projections that share an input, or all projections of a layer):
 * problems[i].y = W_i problems[i].x for i < n, each exactly as tetra_gemv
 * computes it.  problems: host array of n (1..TETRA_MAX_GROUP) entries,
 * read during the call only.  Same status codes as tetra_gemv; a bad entry
 * fails the whole call before any launch.
 */
int tetra_gemv_grouped(const tetra_gemv_problem* problems, int n, int batch,
                       hipStream_t stream);

/* Largest number of phases in one tetra_gemv_chain call. */
#define TETRA_MAX_PHASES 16

/*
 * Several groups of Tetra products run in order in one launch: the
 * dependency groups of a decode step (Sec. 5.1, Sec. 6: the q, k, v
 * projections, then o, then gate and up, then down) without a kernel
 * boundary between them.  Phase k holds phase_counts[k] problems; the
 * problems are listed in phase order (n = sum of the counts, 1..
 * TETRA_MAX_GROUP in all; n_phases 1..TETRA_MAX_PHASES).  Every product is
 * computed exactly as tetra_gemv computes it, with the same bits as a
 * tetra_gemv_grouped call of its phase on a device where both run the
 * same number of waves.  The launch holds every workgroup the device keeps
 * resident at once; the decoder tables are staged once, and no workgroup
 * starts the products of phase k + 1 before every workgroup has finished
 * phase k (a device-wide barrier; only the code words of phase k + 1, which
 * no phase writes, are requested before it).  The barrier orders execution,
 * not memory: the inputs of a phase must not be outputs of an earlier phase
 * of the same call.
 *   problems:     host array, read during the call only
 *   phase_counts: host array of n_phases counts >= 1
 *   status:       device int, 4-byte aligned, or NULL: when the launch
 *                 ends it holds 0, or TETRA_ETIMEOUT if a wait between
 *                 phases gave up.  Each wait is bounded (see
 *                 tetra_set_chain_wait_limit), so a launch whose workgroups
 *                 cannot all be resident at once still ends; a workgroup
 *                 whose wait gives up abandons the rest of the launch, and
 *                 the outputs of its phases are then undefined.  The
 *                 workspace slot is left ready for the next call either way.
 * Asynchronous; status codes as for tetra_gemv_grouped, checked before any
 * launch.  Shares the stream's workspace slot with tetra_gemv.
 */
int tetra_gemv_chain(const tetra_gemv_problem* problems, int n, const int* phase_counts, int n_phases,
                     int batch, int* status, hipStream_t stream);

/*
 * Test hook: the number of polls (about a microsecond each) after which a
 * wait of later tetra_gemv_chain launches gives up; 0 restores the default
 * (2^20).  Returns the previous value.  Host only; affects launches made
 * after it returns.
 */
uint32_t tetra_set_chain_wait_limit(uint32_t polls);

/*
 * Bulk decode of n canonical words (Sec. 3.4, Fig. 4), for testing.
 *   words:         device, n*6 bytes, canonical little-endian words
 *   y_out:         device int8[n][24], the lattice point in block order
 *   blk_scale_out: device fp32[n], s_blk = fl32(gain[g] * invnorm[m]);
 *                  may be NULL
 * Asynchronous.  TETRA_EINVAL for NULL words/y_out or n == 0.
 */
int tetra_decode(const void* words, size_t n, int8_t* y_out, float* blk_scale_out,
                 hipStream_t stream);

/*
 * The same product for many activation rows (a prompt run in one call,
 * Sec. 6): y[n][row] for n < N, formed as in tetra_gemv (exact decoded
 * values, each block's products scaled by its block scale in fp32, sigma and
 * the unquantised tail at the end), with the products on the matrix cores.
 *   codes / row_scales as in tetra_gemv (16-byte aligned codes)
 *   x: device fp16 [N][K], 16-byte aligned; K must be a multiple of 8
 *   y: device fp32 [N][M], fully overwritten
 * N >= 1; a prompt whose activations pass 2 GiB runs as several launches.
 * Meant for N well above TETRA_MAX_BATCH; the rounding differs from
 * tetra_gemv's (another summation order), within the same bound, and the
 * split of the work over workgroups follows M, K, N and the CU count, so a
 * token's result can change in the last bits with N (it never changes from
 * run to run).
 *   workspace: device memory of the caller, 256-byte aligned, holding
 *              counters and partial sums of the pieces of a launch; it
 *              must be zero-filled before its first use, and every call
 *              leaves it zero-filled again.  Calls that may run at the
 *              same time need different workspaces.
 *   workspace_bytes: its size; tetra_gemm_workspace_bytes() is the size at
 *              which the product uses every workgroup the device holds (a
 *              smaller workspace runs fewer workgroups, TETRA_EINVAL below
 *              one workgroup's share)
 * Asynchronous; TETRA_EINVAL / TETRA_EALIGN / TETRA_EDEVICE as for
 * tetra_gemv.
 */
int tetra_gemm(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M, int K, int N,
               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes at which tetra_gemm uses the whole current device (host
 * only; 0 when the device cannot be queried). */
size_t tetra_gemm_workspace_bytes(void);

/*
 * tetra_gemm without a workspace argument, for callers that cannot allocate
 * device memory (code under graph capture, serving loops, harnesses that
 * forbid hipMalloc).  The counters and piece sums of the product live in a
 * static scratch array of the library's code object: 67,110,912 bytes per
 * device (the pieces of 512 workgroups, two per CU of a 256-CU MI355X),
 * held by every device the library runs on until the process ends.  The
 * call runs the same grid as tetra_gemm with a workspace of
 * tetra_gemm_workspace_bytes(), so the two give the same bits; a device
 * that would run more than 512 workgroups is refused (TETRA_EUNSUPPORTED)
 * rather than served with another split.  Input sizes are not limited by
 * the scratch: the pieces scale with the workgroups, not with M, K or N.
 * Each call first clears the scratch's counters with a kernel on `stream`.
 * All calls on one device share its scratch and leave the last call's
 * contents in it: calls that overlap in time on one device (other streams,
 * other threads) race and give wrong results.  Arguments, layouts and the
 * other errors as for tetra_gemm.  Never allocates or synchronises.
 */
int tetra_gemm_noalloc(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M, int K,
                       int N, hipStream_t stream);

/*
 * Gives back the GEMV workspace slot that `stream` holds on the current
 * device, if any (host only).  Call it only when no GEMV work issued on the
 * stream is still pending or will be replayed from a graph.  Always
 * TETRA_OK unless the device cannot be queried.
 */
int tetra_release_stream(hipStream_t stream);

/*
 * Encoder of 24-weight blocks (the offline step of Sec. 3.1, shape-gain of
 * Eq. 2): for each block the canonical word of the kept lattice point whose
 * direction is closest among the nearest kept points to r * w / ||w|| at
 * the two trial radii r = radius0, radius1, and the gain bit nearest to the
 * block's projection on it.  Scores are exact integers: with targets
 * T_j = rint(w_j r 2^16 / ||w||), a kept point y scores
 * S(y) = sum_j (2 T_j y_j - 2^16 y_j^2); equal scores go to the first row
 * of a section's list and then to the smallest trellis key, and equal
 * projections to the first radius, so the result is fixed by the inputs.
 * A block whose squared norm is zero or not finite gets the word 0.
 *   w:         device fp32 [n][24], block order (coordinate j of a block
 *              multiplies activation 24 blk + j), 4-byte aligned
 *   sigma:     device fp32 [n], the row scale of each block's row
 *   words_out: device, n * 6 bytes, canonical little-endian words, 2-byte
 *              aligned (the input format of tetra_decode)
 *   radius0, radius1: in (0, 25]
 * Asynchronous.  TETRA_EINVAL for NULL pointers, n == 0 or a radius out of
 * range; TETRA_EALIGN; TETRA_EDEVICE at launch.
 */
int tetra_encode(const float* w, const float* sigma, size_t n, double radius0, double radius1, void* words_out,
                 hipStream_t stream);

/*
 * Dense reconstruction of a packed matrix (Eq. 2), for testing:
 *   w_out[row][24*blk+j] = fl32(fl32(y_j * s_blk) * sigma_row),
 *   w_out[row][24*nblk+t] = tail[row][t].
 *   codes / row_scales as in tetra_gemv; w_out: device fp32[M][K].
 */
int tetra_dequant(const void* codes, const uint16_t* row_scales, int M, int K,
                  float* w_out, hipStream_t stream);

/*
 * int4 projection of a served file (Sec. 4.1, Sec. 4.3): 4-bit weights in
 * groups of 128 along K, an fp16 scale and offset per group,
 *   w[row][k] = scale[row][k/128] * q[row][k] + offset[row][k/128],
 *   y[b][row] = sum_k w[row][k] * x[b][k]      (f32 accumulation).
 *   q:         device bytes [M][K/2]; element 2i in the low nibble of byte
 *              i, 2i+1 in the high nibble; 8-byte aligned
 *   scale_off: device fp16 [M][K/128][2] (scale, offset); 4-byte aligned
 *   x:         device fp16 [batch][K], 16-byte aligned
 *   y:         device fp32 [batch][M], fully overwritten
 * K must be a positive multiple of 128; batch 1..TETRA_MAX_BATCH.
 * Deterministic and batch-invariant.  Asynchronous; TETRA_EINVAL /
 * TETRA_EALIGN / TETRA_EDEVICE as for tetra_gemv.
 */
int tetra_int4_gemv(const void* q, const uint16_t* scale_off, const uint16_t* x, float* y, int M, int K,
                    int batch, hipStream_t stream);

/*
 * The 4-bit output head (Sec. 4.4): a table of `rows` outputs by `dim`
 * inputs in the embedding layout (groups of 64 along dim, fp16 scale and
 * offset per group, nibbles as in tetra_int4_gemv), times the activations:
 *   y[b][r] = sum_k (scale[r][k/64] * q[r][k] + offset[r][k/64]) * x[b][k]
 *   q:         device bytes [rows][dim/2], 8-byte aligned
 *   scale_off: device fp16 [rows][dim/64][2], 4-byte aligned
 *   x:         device fp16 [batch][dim], 16-byte aligned
 *   y:         device fp32 [batch][rows], fully overwritten
 * dim must be a positive multiple of 64; batch 1..TETRA_MAX_BATCH.
 * Deterministic and batch-invariant.  Asynchronous; TETRA_EINVAL /
 * TETRA_EALIGN / TETRA_EDEVICE as for tetra_gemv.
 */
int tetra_head4_gemv(const void* q, const uint16_t* scale_off, const uint16_t* x, float* y, int rows, int dim,
                     int batch, hipStream_t stream);

/*
 * Online rotation of the activations (Sec. 3.1, Sec. 5.1): the randomized
 * Hadamard transform that the encoder applied to the weights, applied to x
 * before the products that share it.  The paper names no construction; the
 * reading taken is blockwise: for each block of n consecutive elements of a
 * row (j0 a multiple of n),
 *   out[b][j0 + i] = fp16( (1/sqrt n) * sum_m H_n[i][m] * s[j0+m] * x[b][j0+m] )
 * with H_n the Sylvester Hadamard matrix (H_n[i][m] = (-1)^popcount(i & m))
 * and s[k] = -1 where bit k % 8 of sign_bits[k / 8] is set, else +1.  The
 * signs are the caller's (drawn once per group of projections).  Computed in
 * fp32, rounded to nearest even at the end.
 *   x:         device fp16 [rows][K], 8-byte aligned
 *   sign_bits: device bytes [ceil(K / 8)]
 *   out:       device fp16 [rows][K], 8-byte aligned; may be x itself
 * n must be a power of two in [4, 4096] dividing K; rows 1..65535.
 * Asynchronous; TETRA_EINVAL / TETRA_EALIGN / TETRA_EDEVICE as for tetra_gemv.
 */
int tetra_rotate(const uint16_t* x, const uint8_t* sign_bits, uint16_t* out, int K, int n, int rows,
                 hipStream_t stream);

/*
 * Rows of a 4-bit embedding table (Sec. 4.4): groups of 64 along the
 * embedding dimension, fp16 scale and offset per group, nibbles as in
 * tetra_int4_gemv;  out[i][k] = fl32(fl32(scale * q) + offset) for the row
 * tokens[i].
 *   q:         device bytes [rows][dim/2]
 *   scale_off: device fp16 [rows][dim/64][2]
 *   tokens:    device int32 [n]; a token outside [0, rows) gives a row of
 *              zeros (the table is never read out of bounds)
 *   out:       device fp32 [n][dim]
 * dim must be a positive multiple of 64.  Asynchronous.
 */
int tetra_emb4_gather(const void* q, const uint16_t* scale_off, int rows, int dim, const int* tokens, int n,
                      float* out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* TETRA_H */
