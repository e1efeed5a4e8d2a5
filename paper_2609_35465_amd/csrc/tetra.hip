// Tetra decode and fused decode-GEMV for MI355X (gfx950): the C ABI of
// include/tetra.h.  Host code here validates arguments, uploads the decoder
// tables once per device and launches the kernels of kernels.h, prefill.h
// and encoder.h.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>

#include <algorithm>
#include <atomic>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "../../include/tetra.h"
#include "device_tables.h"
#include "kernels.h"
#include "prefill.h"
#include "encoder.h"
#include "tables.h"
#include "word_format.h"

namespace {

using tetra_dev::kChunk;
using tetra_dev::kTile;

constexpr int kMaxDevices = 64;

// Scratch of tetra_gemm_noalloc: the counters and piece slots of up to
// kScratchWorkers workgroups of the many-token product, the whole chip's
// worth on a 256-CU part (two workgroups per CU).  Every device holds its own
// copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the device (DeviceState::scratch), never
// through the array's name.
constexpr int kScratchWorkers = 512;
constexpr size_t kScratchBytes = 67110912;   // gemm_workspace_bytes(kScratchWorkers)
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// What the host knows about a device, queried once and kept: no call makes
// the device do any work, allocate or wait to set it up.  Also the owners of
// the device's GEMV workspace slots (kernels.h, g_gemv_slots).
struct DeviceState {
    bool ready = false;
    int cus = 0;
    int gemv_groups[TETRA_MAX_BATCH + 1] = {};   // resident GEMV workgroups per CU, by batch
    int gemm_workers = 0;
    uint8_t* scratch = nullptr;                  // this device's copy of `scratch`
    bool slot_used[tetra_dev::kGemvSlots] = {};
    hipStream_t slot_stream[tetra_dev::kGemvSlots] = {};
    std::thread::id slot_thread[tetra_dev::kGemvSlots];
};

std::mutex g_mu;
DeviceState g_dev[kMaxDevices];

int num_cus(int dev) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return 256;
    return n;
}

// workgroups of gemv_kernel<B> one CU holds at once (registers and LDS of
// the compiled kernel), between 1 and kGemvGroupsPerCU; 0 on an error
template <int B>
int gemv_resident() {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(&tetra_dev::gemv_kernel<B, true>),
                                                     tetra_dev::kGemvThreads, 0) != hipSuccess)
        return 0;
    return std::max(1, std::min(n, tetra_dev::kGemvGroupsPerCU));
}

// the current device and its state (filled on first use); called with g_mu held
int device_state_locked(int* dev_out, DeviceState** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TETRA_EDEVICE;
    *dev_out = dev;
    DeviceState& d = g_dev[dev];
    if (!d.ready) {
        static_assert(TETRA_MAX_BATCH == 8, "one residency entry per batch size");
        const int resident[TETRA_MAX_BATCH + 1] = {0, gemv_resident<1>(), gemv_resident<2>(), gemv_resident<3>(),
                                                   gemv_resident<4>(), gemv_resident<5>(), gemv_resident<6>(),
                                                   gemv_resident<7>(), gemv_resident<8>()};
        for (int b = 1; b <= TETRA_MAX_BATCH; ++b)
            if (resident[b] == 0) return TETRA_EDEVICE;
        void* sp = nullptr;
        if (hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch)) != hipSuccess || !sp) return TETRA_EDEVICE;
        d.scratch = static_cast<uint8_t*>(sp);
        d.cus = num_cus(dev);
        for (int b = 0; b <= TETRA_MAX_BATCH; ++b) d.gemv_groups[b] = resident[b];
        d.gemm_workers = d.cus * tetra_dev::kPfGroupsPerCU;
        d.ready = true;
    }
    *out = &d;
    return TETRA_OK;
}

int device_state(int* dev_out, DeviceState* copy) {
    std::lock_guard<std::mutex> lk(g_mu);
    DeviceState* d = nullptr;
    if (int st = device_state_locked(dev_out, &d)) return st;
    if (copy) *copy = *d;
    return TETRA_OK;
}

// The per-thread default stream is a different stream in every thread.
bool same_stream(const DeviceState& d, int i, hipStream_t s) {
    return d.slot_stream[i] == s && (s != hipStreamPerThread || d.slot_thread[i] == std::this_thread::get_id());
}

// the GEMV workspace slot of `stream` on the current device, taking a free
// one on the stream's first call; TETRA_EBUSY when all are held by others
int gemv_slot(hipStream_t stream, DeviceState* copy, int* slot) {
    std::lock_guard<std::mutex> lk(g_mu);
    int dev;
    DeviceState* d = nullptr;
    if (int st = device_state_locked(&dev, &d)) return st;
    int free_slot = -1;
    for (int i = 0; i < tetra_dev::kGemvSlots; ++i) {
        if (d->slot_used[i] && same_stream(*d, i, stream)) {
            *slot = i;
            *copy = *d;
            return TETRA_OK;
        }
        if (!d->slot_used[i] && free_slot < 0) free_slot = i;
    }
    if (free_slot < 0) return TETRA_EBUSY;
    d->slot_used[free_slot] = true;
    d->slot_stream[free_slot] = stream;
    d->slot_thread[free_slot] = std::this_thread::get_id();
    *slot = free_slot;
    *copy = *d;
    return TETRA_OK;
}

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

int launch_status() { return hipGetLastError() == hipSuccess ? TETRA_OK : TETRA_EDEVICE; }

// polls before a chain barrier wait gives up (about one microsecond each)
std::atomic<uint32_t> g_chain_wait_limit{1u << 20};

// A plain or grouped product (one phase) or a chain of phases.  Problems are
// in phase order; phase k holds counts[k] of them.
int launch_gemv(const tetra_gemv_problem* probs, int n, const int* counts, int n_phases, int batch, int* status,
                hipStream_t stream) {
    if (!probs || n < 1 || n > TETRA_MAX_GROUP) return TETRA_EINVAL;
    if (n_phases < 1 || n_phases > TETRA_MAX_PHASES || (n_phases > 1 && !counts)) return TETRA_EINVAL;
    if (batch < 1 || batch > TETRA_MAX_BATCH) return TETRA_EINVAL;
    tetra_dev::GemvChain ch;
    std::memset(&ch, 0, sizeof(ch));
    int p = 0;
    for (int k = 0; k < n_phases; ++k) {
        const int cnt = counts ? counts[k] : n;
        if (cnt < 1 || cnt > n - p) return TETRA_EINVAL;
        unsigned long long total = 0;
        for (int i = p; i < p + cnt; ++i) {
            if (total >= (1ull << 31)) return TETRA_EINVAL;
            const tetra_gemv_problem& q = probs[i];
            Shape s;
            if (!q.codes || !q.row_scales || !q.x || !q.y || !shape_of(q.M, q.K, &s)) return TETRA_EINVAL;
            if (!aligned(q.codes, 16) || !aligned(q.x, 4)) return TETRA_EALIGN;
            tetra_dev::GemvProblem& P = ch.prob[i];
            P.codes = static_cast<const uint8_t*>(q.codes);
            P.sigma = q.row_scales;
            P.x = q.x;
            P.y = q.y;
            P.M = q.M;
            P.K = q.K;
            P.nblk = s.nblk;
            P.T = s.T;
            P.tail_off = s.tail_off;
            P.tiles = s.tiles;
            P.ng = s.nblk / tetra::kGroupCols;
            P.rem = s.nblk % tetra::kGroupCols;
            P.blk_base = static_cast<uint32_t>(total);
            total += static_cast<unsigned long long>(s.tiles) * s.nblk;
        }
        if (total >= (1ull << 31)) return TETRA_EINVAL;     // block indices are 32-bit
        ch.ph[k].p0 = p;
        ch.ph[k].n = cnt;
        ch.ph[k].total = static_cast<uint32_t>(total);
        p += cnt;
    }
    if (p != n) return TETRA_EINVAL;
    DeviceState ds;
    int slot = 0;
    if (int st = gemv_slot(stream, &ds, &slot)) return st;
    // the workspace slot holds kGemvMaxCUs CUs' worth of workgroups: a larger
    // part runs fewer waves
    const int cus = std::min(ds.cus, tetra_dev::kGemvMaxCUs);
    const int max_waves = std::min(cus * ds.gemv_groups[batch], tetra_dev::gemv_max_groups(batch)) *
                          tetra_dev::kGemvWaves;
    int grid;
    if (n_phases == 1) {
        ch.ph[0].waves = std::min(tetra_dev::gemv_waves(ch.ph[0].total, cus, ds.gemv_groups[batch]), max_waves);
        ch.ph[0].wpg = tetra_dev::kGemvWaves;
        grid = (ch.ph[0].waves + tetra_dev::kGemvWaves - 1) / tetra_dev::kGemvWaves;
    } else {
        // every workgroup the device holds at once, so that all of them are
        // resident together and the barriers between phases can be met; a
        // phase takes the same number of waves from every workgroup, so that
        // every CU gets the same share of it
        grid = max_waves / tetra_dev::kGemvWaves;
        for (int k = 0; k < n_phases; ++k) {
            ch.ph[k].wpg = tetra_dev::chain_phase_wpg(ch.ph[k].total, grid);
            ch.ph[k].waves = static_cast<int>(std::min<uint32_t>(ch.ph[k].total,
                                                                 static_cast<uint32_t>(grid * ch.ph[k].wpg)));
        }
    }
    // three partial-sum buffers for a chain when they fit in the slot (one
    // always does: gemv_max_groups)
    const bool rotate = n_phases > 1 && static_cast<size_t>(tetra_dev::kChainBuffers) * grid * 2 * batch * 64 <=
                                            static_cast<size_t>(tetra_dev::kGemvSlotPartials);
    ch.buffers = rotate ? tetra_dev::kChainBuffers : 1;
    for (int k = 0; k < n_phases; ++k) {
        tetra_dev::GemvSplit& sp = ch.ph[k];
        sp.inv_total = 1.0 / static_cast<double>(sp.total);
        sp.inv_waves = 1.0 / static_cast<double>(sp.waves);
        // tile-aligned when every tile gets a wave of its own (W nblk >= total
        // for the smallest nblk of the phase); waves <= total keeps every
        // tile's share at most its columns, so no range is empty
        int nblk_min = INT_MAX;
        for (int i = sp.p0; i < sp.p0 + sp.n; ++i) nblk_min = std::min(nblk_min, ch.prob[i].nblk);
        sp.aligned = static_cast<unsigned long long>(sp.waves) * static_cast<unsigned>(nblk_min) >= sp.total &&
                     static_cast<uint32_t>(sp.waves) <= sp.total;
        // a chain phase other than the last adds up its tiles that span
        // workgroups after the next barrier: tile-aligned (a wave adds up
        // at most one tile), and with the three partial-sum buffers
        sp.defer = rotate && k + 1 < n_phases && sp.aligned ? (k + 2 < n_phases ? 2 : 1) : 0;
    }
    ch.n_phases = n_phases;
    ch.slot = slot;
    ch.wait_limit = g_chain_wait_limit.load();
    ch.status = status;
#define TETRA_LAUNCH(B)                                                                                  \
    case B:                                                                                              \
        if (n_phases == 1)                                                                               \
            hipLaunchKernelGGL((tetra_dev::gemv_kernel<B, false>), dim3(grid), dim3(tetra_dev::kGemvThreads), \
                               0, stream, ch);                                                           \
        else                                                                                             \
            hipLaunchKernelGGL((tetra_dev::gemv_kernel<B, true>), dim3(grid), dim3(tetra_dev::kGemvThreads), \
                               0, stream, ch);                                                           \
        break;
    switch (batch) {
        TETRA_LAUNCH(1) TETRA_LAUNCH(2) TETRA_LAUNCH(3) TETRA_LAUNCH(4)
        TETRA_LAUNCH(5) TETRA_LAUNCH(6) TETRA_LAUNCH(7) TETRA_LAUNCH(8)
        default: return TETRA_EINVAL;
    }
#undef TETRA_LAUNCH
    return launch_status();
}

}  // namespace

// ================================================================== C ABI

namespace {

// int4 products with groups of G weights along K (K a positive multiple of G)
template <int G>
int int4_gemv_launch(const void* q, const uint16_t* scale_off, const uint16_t* x, float* y, int M, int K,
                     int batch, hipStream_t stream) {
    if (!q || !scale_off || !x || !y || M < 1 || K < G || K % G) return TETRA_EINVAL;
    if (batch < 1 || batch > TETRA_MAX_BATCH) return TETRA_EINVAL;
    if (!aligned(q, 8) || !aligned(scale_off, 4) || !aligned(x, 16)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    const long long pairs = (static_cast<long long>(M) + tetra_dev::kInt4RowsPerWave - 1) / tetra_dev::kInt4RowsPerWave;
    const long long grid = (pairs + tetra_dev::kInt4Waves - 1) / tetra_dev::kInt4Waves;
    if (grid > 0x7FFFFFFFLL) return TETRA_EINVAL;
    const uint8_t* qb = static_cast<const uint8_t*>(q);
    // a launch of at least one row pair per wave of a full chip of persistent
    // workgroups stages the activations in LDS (when they fit in 64 KB)
    const long long lds_groups = static_cast<long long>(tetra_dev::int4_lds_groups_per_cu(batch)) * ds.cus;
    const size_t lds = tetra_dev::int4_lds_bytes(K, batch);
    const bool use_lds = batch <= tetra_dev::kInt4LdsMaxBatch &&
                         pairs >= lds_groups * tetra_dev::kInt4LdsWaves && lds <= 65536;
#define TETRA_I4(B)                                                                                          \
    case B:                                                                                                  \
        if constexpr (B <= tetra_dev::kInt4LdsMaxBatch) {                                                    \
            if (use_lds) {                                                                                   \
                hipLaunchKernelGGL((tetra_dev::int4_gemv_lds_kernel<B, G>),                                  \
                                   dim3(static_cast<unsigned>(lds_groups)), dim3(tetra_dev::kInt4LdsThreads), \
                                   lds, stream, qb, scale_off, x, y, M, K);                                  \
                break;                                                                                       \
            }                                                                                                \
        }                                                                                                    \
        hipLaunchKernelGGL((tetra_dev::int4_gemv_kernel<B, G>), dim3(static_cast<unsigned>(grid)),           \
                           dim3(tetra_dev::kInt4Waves * 64), 0, stream, qb, scale_off, x, y, M, K);          \
        break;
    switch (batch) {
        TETRA_I4(1) TETRA_I4(2) TETRA_I4(3) TETRA_I4(4) TETRA_I4(5) TETRA_I4(6) TETRA_I4(7) TETRA_I4(8)
        default: return TETRA_EINVAL;
    }
#undef TETRA_I4
    return launch_status();
}

}  // namespace

extern "C" {

const char* tetra_status_string(int status) {
    switch (status) {
        case TETRA_OK: return "ok";
        case TETRA_EINVAL: return "invalid argument";
        case TETRA_EALIGN: return "misaligned device pointer";
        case TETRA_EDEVICE: return "HIP runtime error";
        case TETRA_EUNSUPPORTED: return "unsupported request";
        case TETRA_EBUSY: return "every GEMV workspace slot of the device is held by another stream";
        case TETRA_ETIMEOUT: return "a wait between the phases of a chained product gave up";
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

size_t tetra_row_stride(int K) {
    Shape s;
    return shape_of(1, K, &s) ? static_cast<size_t>(s.nblk) * 6 : 0;
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
    // rows of the last tile beyond M hold the recoded zero word
    const tetra::DeviceWord z = tetra::device_word(0);
    for (int row = 0; row < s.tiles * kTile; ++row) {
        const int tile = row / kTile, r = row % kTile;
        uint8_t* tb = o + static_cast<size_t>(tile) * s.nblk * kChunk;
        for (int b = 0; b < s.nblk; ++b) {
            const tetra::DeviceWord d =
                row < M ? tetra::device_word(words[static_cast<size_t>(row) * s.nblk + b]) : z;
            const tetra::WordLoc at = tetra::word_loc(s.nblk, r, b);
            const uint16_t hi = static_cast<uint16_t>(d.hi);
            std::memcpy(tb + at.lo_off, &d.lo, 4);
            std::memcpy(tb + at.hi_off, &hi, 2);
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
        const uint8_t* tb = c + static_cast<size_t>(tile) * s.nblk * kChunk;
        for (int b = 0; b < s.nblk; ++b) {
            const tetra::WordLoc at = tetra::word_loc(s.nblk, r, b);
            tetra::DeviceWord d;
            uint16_t hi;
            std::memcpy(&d.lo, tb + at.lo_off, 4);
            std::memcpy(&hi, tb + at.hi_off, 2);
            d.hi = hi;
            words[static_cast<size_t>(row) * s.nblk + b] = tetra::canonical_from_device(d);
        }
    }
    if (s.T > 0) std::memcpy(tail, c + s.tail_off, static_cast<size_t>(M) * s.T * 2);
    return TETRA_OK;
}

int tetra_gemv(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M,
               int K, int batch, hipStream_t stream) {
    tetra_gemv_problem p;
    p.codes = codes;
    p.row_scales = row_scales;
    p.x = x;
    p.y = y;
    p.M = M;
    p.K = K;
    return launch_gemv(&p, 1, nullptr, 1, batch, nullptr, stream);
}

int tetra_gemv_grouped(const tetra_gemv_problem* problems, int n, int batch, hipStream_t stream) {
    return launch_gemv(problems, n, nullptr, 1, batch, nullptr, stream);
}

int tetra_gemv_chain(const tetra_gemv_problem* problems, int n, const int* phase_counts, int n_phases, int batch,
                     int* status, hipStream_t stream) {
    if (status && !aligned(status, 4)) return TETRA_EALIGN;
    return launch_gemv(problems, n, phase_counts, n_phases, batch, status, stream);
}

uint32_t tetra_set_chain_wait_limit(uint32_t polls) {
    return g_chain_wait_limit.exchange(polls == 0 ? (1u << 20) : polls);
}

int tetra_decode(const void* words, size_t n, int8_t* y_out, float* blk_scale_out,
                 hipStream_t stream) {
    if (!words || !y_out || n == 0) return TETRA_EINVAL;
    if (!aligned(words, 2) || !aligned(y_out, 4) || (blk_scale_out && !aligned(blk_scale_out, 4)))
        return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    const size_t blocks = std::min<size_t>((n + 255) / 256, static_cast<size_t>(ds.cus) * 8);
    hipLaunchKernelGGL(tetra_dev::decode_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       static_cast<const uint16_t*>(words), n, y_out, blk_scale_out);
    return launch_status();
}

int tetra_dequant(const void* codes, const uint16_t* row_scales, int M, int K, float* w_out,
                  hipStream_t stream) {
    Shape s;
    if (!codes || !row_scales || !w_out || !shape_of(M, K, &s)) return TETRA_EINVAL;
    if (!aligned(codes, 16) || !aligned(w_out, 4)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    const size_t units = static_cast<size_t>(s.tiles) * s.nblk;
    const size_t blocks = std::min<size_t>((units + 3) / 4, static_cast<size_t>(ds.cus) * 2);
    hipLaunchKernelGGL(tetra_dev::dequant_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256),
                       0, stream,
                       static_cast<const uint8_t*>(codes), row_scales, M, K, s.nblk, s.T,
                       s.tail_off, w_out);
    return launch_status();
}

int tetra_int4_gemv(const void* q, const uint16_t* scale_off, const uint16_t* x, float* y, int M, int K,
                    int batch, hipStream_t stream) {
    return int4_gemv_launch<tetra_dev::kInt4Group>(q, scale_off, x, y, M, K, batch, stream);
}

int tetra_head4_gemv(const void* q, const uint16_t* scale_off, const uint16_t* x, float* y, int rows, int dim,
                     int batch, hipStream_t stream) {
    return int4_gemv_launch<tetra_dev::kHead4Group>(q, scale_off, x, y, rows, dim, batch, stream);
}

namespace {

// one launch of the many-token product over tokens n_base .. n_base + N - 1
int gemm_launch(const uint8_t* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M, int K, int N,
                const Shape& s, int max_workers, uint8_t* workspace, hipStream_t stream) {
    const long long token_groups = (static_cast<long long>(N) + tetra_dev::kPfTokens - 1) / tetra_dev::kPfTokens;
    // four token groups per wave (items of two tiles) unless that cuts the
    // average item into more than eight pieces over the launch's workgroups;
    // then two (items of one tile)
    const int upi = s.nblk / tetra::kGroupCols + (s.nblk % tetra::kGroupCols ? 1 : 0);
    long long items = static_cast<long long>((s.tiles + 1) / 2) * token_groups;
    int tg = 4;
    if (std::min<long long>(items * upi, max_workers) > 8 * items) {
        tg = 2;
        items = static_cast<long long>(s.tiles) * token_groups;
    }
    if (items >= (1ll << 31)) return TETRA_EINVAL;
    tetra_dev::GemmArgs a;
    a.codes = codes;
    a.sigma = row_scales;
    a.x = x;
    a.y = y;
    a.tail_off = s.tail_off;
    a.M = M;
    a.K = K;
    a.N = N;
    a.nblk = s.nblk;
    a.T = s.T;
    a.ng = s.nblk / tetra::kGroupCols;
    a.rem = s.nblk % tetra::kGroupCols;
    a.tgroups = static_cast<int>(token_groups);
    a.tiles = s.tiles;
    a.upi = upi;
    a.units = static_cast<unsigned long long>(items) * static_cast<unsigned long long>(a.upi);
    // at most eight workgroups per item on average: past that, a few more
    // chunks per workgroup cost less than the longer reduction
    a.workers = static_cast<int>(std::min<unsigned long long>(
        std::min<unsigned long long>(a.units, static_cast<unsigned long long>(max_workers)),
        static_cast<unsigned long long>(items) * 8));
    if (a.units > ~0ull / static_cast<unsigned long long>(a.workers + 1)) return TETRA_EINVAL;   // range arithmetic
    a.counters = reinterpret_cast<uint32_t*>(workspace);
    a.partials = reinterpret_cast<float*>(workspace + tetra_dev::gemm_counter_bytes(max_workers));
    a.partial_bytes = static_cast<int>(sizeof(float) * 2 * tetra_dev::kPfSlot * static_cast<size_t>(max_workers));
    if (tg == 4)
        hipLaunchKernelGGL(tetra_dev::gemm_kernel<4>, dim3(static_cast<unsigned>(a.workers)),
                           dim3(tetra_dev::kPfThreads), 0, stream, a);
    else
        hipLaunchKernelGGL(tetra_dev::gemm_kernel<2>, dim3(static_cast<unsigned>(a.workers)),
                           dim3(tetra_dev::kPfThreads), 0, stream, a);
    return launch_status();
}

}  // namespace

size_t tetra_gemm_workspace_bytes(void) {
    int dev;
    DeviceState ds;
    if (device_state(&dev, &ds)) return 0;
    return tetra_dev::gemm_workspace_bytes(ds.gemm_workers);
}

int tetra_gemm(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M, int K, int N,
               void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (!codes || !row_scales || !x || !y || !workspace || M < 1 || K < 24 || N < 1 || K % 8) return TETRA_EINVAL;
    if (!aligned(codes, 16) || !aligned(x, 16) || !aligned(row_scales, 2) || !aligned(y, 4) ||
        !aligned(workspace, 256))
        return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    Shape s;
    if (!shape_of(M, K, &s)) return TETRA_EINVAL;
    // as many workgroups as the device holds and the workspace has slots for
    int workers = ds.gemm_workers;
    while (workers > 0 && tetra_dev::gemm_workspace_bytes(workers) > workspace_bytes) --workers;
    if (workers < 1) return TETRA_EINVAL;
    // the kernel addresses a launch's activations with 32-bit byte offsets:
    // prompts longer than that run as several launches of whole token groups
    const long long slice = std::max<long long>(
        tetra_dev::kPfTokens,
        ((0x7FFFFFFFll / (2ll * K)) / tetra_dev::kPfTokens) * tetra_dev::kPfTokens);
    for (long long n = 0; n < N; n += slice) {
        const int cnt = static_cast<int>(std::min<long long>(slice, N - n));
        if (int st = gemm_launch(static_cast<const uint8_t*>(codes), row_scales, x + n * K, y + n * M, M, K, cnt, s,
                                 workers, static_cast<uint8_t*>(workspace), stream))
            return st;
    }
    return TETRA_OK;
}

namespace tetra_dev {

// zeroes n 32-bit words (the counters of a scratch region), so that clearing
// is a kernel node, not a memset, when the caller captures a graph
__global__ __launch_bounds__(256) void zero_words_kernel(uint32_t* p, int n) {
    for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

}  // namespace tetra_dev

int tetra_gemm_noalloc(const void* codes, const uint16_t* row_scales, const uint16_t* x, float* y, int M, int K,
                       int N, hipStream_t stream) {
    static_assert(tetra_dev::kChainTimeout == TETRA_ETIMEOUT, "status value written by the kernel");
    static_assert(tetra_dev::kMaxGroup == TETRA_MAX_GROUP && tetra_dev::kMaxPhases == TETRA_MAX_PHASES,
                  "limits of the boundary");
    static_assert(sizeof(tetra_dev::GemvChain) <= 4096, "kernel arguments");
    static_assert(kScratchBytes >= (sizeof(uint32_t) * kScratchWorkers + 255) / 256 * 256 +
                                       sizeof(float) * static_cast<size_t>(kScratchWorkers) * 2 * tetra_dev::kPfSlot,
                  "scratch holds the counters and pieces of kScratchWorkers workgroups");
    if (!codes || !row_scales || !x || !y || M < 1 || K < 24 || N < 1 || K % 8) return TETRA_EINVAL;
    if (!aligned(codes, 16) || !aligned(x, 16) || !aligned(row_scales, 2) || !aligned(y, 4)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    Shape s;
    if (!shape_of(M, K, &s)) return TETRA_EINVAL;
    // the device's whole grid, as tetra_gemm with a full workspace runs it;
    // a device that holds more workgroups than the scratch has slots for is
    // refused rather than served by a smaller grid with other rounding
    const int workers = ds.gemm_workers;
    if (workers < 1) return TETRA_EDEVICE;
    if (workers > kScratchWorkers || tetra_dev::gemm_workspace_bytes(workers) > kScratchBytes)
        return TETRA_EUNSUPPORTED;
    uint8_t* ws = ds.scratch;
    const int nctr = static_cast<int>(tetra_dev::gemm_counter_bytes(workers) / sizeof(uint32_t));
    hipLaunchKernelGGL(tetra_dev::zero_words_kernel, dim3(static_cast<unsigned>((nctr + 255) / 256)), dim3(256), 0,
                       stream, reinterpret_cast<uint32_t*>(ws), nctr);
    if (int st = launch_status()) return st;
    const long long slice = std::max<long long>(
        tetra_dev::kPfTokens,
        ((0x7FFFFFFFll / (2ll * K)) / tetra_dev::kPfTokens) * tetra_dev::kPfTokens);
    for (long long n = 0; n < N; n += slice) {
        const int cnt = static_cast<int>(std::min<long long>(slice, N - n));
        if (int st = gemm_launch(static_cast<const uint8_t*>(codes), row_scales, x + n * K, y + n * M, M, K, cnt, s,
                                 workers, ws, stream))
            return st;
    }
    return TETRA_OK;
}

int tetra_release_stream(hipStream_t stream) {
    std::lock_guard<std::mutex> lk(g_mu);
    int dev;
    DeviceState* d = nullptr;
    if (int st = device_state_locked(&dev, &d)) return st;
    for (int i = 0; i < tetra_dev::kGemvSlots; ++i)
        if (d->slot_used[i] && same_stream(*d, i, stream)) d->slot_used[i] = false;
    return TETRA_OK;
}

int tetra_encode(const float* w, const float* sigma, size_t n, double radius0, double radius1, void* words_out,
                 hipStream_t stream) {
    if (!w || !sigma || !words_out || n == 0) return TETRA_EINVAL;
    for (double r : {radius0, radius1})
        if (!(r > 0.0 && r <= tetra_dev::kEncMaxRadius)) return TETRA_EINVAL;
    if (!aligned(w, 4) || !aligned(sigma, 4) || !aligned(words_out, 2)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    tetra_dev::EncodeArgs a;
    a.w = w;
    a.sigma = sigma;
    a.words = static_cast<uint16_t*>(words_out);
    a.n = n;
    a.alpha[0] = radius0;
    a.alpha[1] = radius1;
    const size_t grid = std::min<size_t>(n, static_cast<size_t>(ds.cus) * 8);
    hipLaunchKernelGGL(tetra_dev::encode_kernel, dim3(static_cast<unsigned>(grid)), dim3(tetra_dev::kEncThreads), 0,
                       stream, a);
    return launch_status();
}

int tetra_rotate(const uint16_t* x, const uint8_t* sign_bits, uint16_t* out, int K, int n, int rows,
                 hipStream_t stream) {
    if (!x || !sign_bits || !out || n < 4 || n > 4096 || (n & (n - 1)) || K < n || K % n) return TETRA_EINVAL;
    if (rows < 1 || rows > 65535) return TETRA_EINVAL;
    if (!aligned(x, 8) || !aligned(out, 8)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    const float scale = static_cast<float>(1.0 / std::sqrt(static_cast<double>(n)));
    const int T = n <= 1024 ? 256 : n / 4;
    const dim3 grid(static_cast<unsigned>((K + 4 * T - 1) / (4 * T)), static_cast<unsigned>(rows));
    switch (T) {
        case 256:
            hipLaunchKernelGGL(tetra_dev::rotate_kernel<256>, grid, dim3(256), 0, stream, x, sign_bits, out, K, n, scale);
            break;
        case 512:
            hipLaunchKernelGGL(tetra_dev::rotate_kernel<512>, grid, dim3(512), 0, stream, x, sign_bits, out, K, n, scale);
            break;
        default:
            hipLaunchKernelGGL(tetra_dev::rotate_kernel<1024>, grid, dim3(1024), 0, stream, x, sign_bits, out, K, n,
                               scale);
            break;
    }
    return launch_status();
}

int tetra_emb4_gather(const void* q, const uint16_t* scale_off, int rows, int dim, const int* tokens, int n,
                      float* out, hipStream_t stream) {
    if (!q || !scale_off || !tokens || !out || rows < 1 || n < 1 || dim < tetra_dev::kEmbGroup ||
        dim % tetra_dev::kEmbGroup)
        return TETRA_EINVAL;
    if (!aligned(scale_off, 4) || !aligned(tokens, 4) || !aligned(out, 4)) return TETRA_EALIGN;
    int dev;
    DeviceState ds;
    if (int st = device_state(&dev, &ds)) return st;
    const long long bytes = static_cast<long long>(n) * (dim / 2);
    const unsigned grid = static_cast<unsigned>(std::min<long long>((bytes + 255) / 256, 4096));
    hipLaunchKernelGGL(tetra_dev::emb4_gather_kernel, dim3(grid), dim3(256), 0, stream,
                       static_cast<const uint8_t*>(q), scale_off, rows, dim, tokens, n, out);
    return launch_status();
}

}  // extern "C"
