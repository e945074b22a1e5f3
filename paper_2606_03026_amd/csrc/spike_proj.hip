// Host side of the spike-gated INT8 projection library (C ABI in
// include/spike_proj.h).  Validates arguments, owns the per-handle INT32
// workspace, picks a kernel and launch shape, and enqueues on the caller's
// stream.  No host synchronisation, allocation or memset happens on the
// forward path.
#include "spike_proj.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "errors.hpp"
#include "gather.hpp"
#include "mfma.hpp"

struct spike_proj;
struct spike_stream;

namespace {

using spk::fail;
using spk::hip_fail;

int64_t words_per_row(int64_t K) { return (K + 63) / 64; }

// ---------------------------------------------------------------------------
// Launch shapes.  Every instantiated (V, LG, U, BLOCK) combination of the
// gather and stream kernels is listed once; a shape code packs it as
// SPIKE_SHAPE(V, LG, U, BLOCK) from the header.
// ---------------------------------------------------------------------------
using GatherFn = void (*)(const spike_proj*, const uint64_t*, int32_t, int, int, int, int, float*, int32_t*,
                          hipStream_t);
using StreamFn = void (*)(const spike_stream*, int, unsigned, const uint64_t*, float*, hipStream_t);

// Kernels of a shape come in two variants: weight loads through a buffer
// resource (index 1, matrices of at most spk::kBufMaxBytes) and through
// 64-bit addresses (index 0, any size).
struct ShapeEntry {
    int code;
    int vec, lanes, unroll, block;
    GatherFn gather[2];
    GatherFn gather_acc[2];
    StreamFn stream[2];
};

template <class S, bool ACC, bool BUF>
void launch_gather_t(const spike_proj* h, const uint64_t* mask, int32_t B, int sw, int n_slices, int n_tiles,
                     int tpu, float* out, int32_t* acc, hipStream_t st);
template <class S, bool BUF>
void launch_stream_t(const spike_stream* s, int n_tiles, unsigned units, const uint64_t* masks, float* out,
                     hipStream_t st);

template <int V, int LG, int U, int BLOCK, bool NT = false, bool I16 = false>
constexpr ShapeEntry entry()
{
    using S = spk::Shape<V, LG, U, BLOCK, NT, I16>;
    return ShapeEntry{SPIKE_SHAPE(V, LG, U, BLOCK) | (NT ? SPIKE_SHAPE_NT : 0) | (I16 ? SPIKE_SHAPE_I16 : 0),
                      V,
                      LG,
                      U,
                      BLOCK,
                      {&launch_gather_t<S, false, false>, &launch_gather_t<S, false, true>},
                      {&launch_gather_t<S, true, false>, &launch_gather_t<S, true, true>},
                      {&launch_stream_t<S, false>, &launch_stream_t<S, true>}};
}

const ShapeEntry kShapes[] = {
    // half-column tiles, nontemporal weight loads (throughput: streams, batched rows), ring depths
    entry<16, 32, 4, 256, true>(), entry<16, 32, 2, 256, true>(), entry<16, 32, 6, 256, true>(),
    entry<16, 32, 8, 256, true>(), entry<16, 32, 4, 512, true>(), entry<16, 64, 4, 256, true>(),
    entry<8, 64, 4, 256, true>(), entry<8, 32, 4, 256, true>(),
    // exact 16-bit partial sums (buffer-resource kernels; the 64-bit-address ones sum in INT32)
    entry<16, 32, 4, 256, true, true>(),
    // the same with cached loads (weights re-read soon, e.g. warm caches)
    entry<16, 32, 4, 256>(), entry<8, 64, 4, 256>(),
    // narrow tiles (decode latency)
    entry<4, 64, 4, 256>(), entry<4, 16, 8, 256>(), entry<4, 16, 4, 1024>(), entry<4, 16, 16, 256>(),
    // any N, any alignment
    entry<1, 64, 4, 256>(),
};

// The buffer-resource kernels address the weight matrix with 32-bit offsets.
bool fits_buffer(int64_t K, int64_t N) { return K * N <= spk::kBufMaxBytes; }

const ShapeEntry* find_shape(int code)
{
    for (const ShapeEntry& e : kShapes)
        if (e.code == code)
            return &e;
    return nullptr;
}

int shape_tile(const ShapeEntry* e) { return e->vec * e->lanes; }

// The shape's vector loads stay aligned and in range for this matrix.
bool shape_fits(const ShapeEntry* e, const void* W, int64_t N)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(W);
    return N % e->vec == 0 && a % e->vec == 0;
}

// Default throughput shape for a vector width (0: the widest that fits):
// 512-byte tiles with nontemporal loads, four columns in flight per lane
// (16-byte lanes need N to be a multiple of 512 to keep every lane busy).
const ShapeEntry* default_shape(const void* W, int64_t N, int vec)
{
    static const int by_vec[][2] = {{16, SPIKE_SHAPE(16, 32, 4, 256) | SPIKE_SHAPE_NT},
                                    {8, SPIKE_SHAPE(8, 64, 4, 256) | SPIKE_SHAPE_NT},
                                    {4, SPIKE_SHAPE(4, 64, 4, 256)},
                                    {1, SPIKE_SHAPE(1, 64, 4, 256)}};
    for (const auto& bv : by_vec) {
        if (vec != 0 && bv[0] != vec)
            continue;
        if (vec == 0 && bv[0] == 16 && N % 512 != 0)
            continue;
        const ShapeEntry* e = find_shape(bv[1]);
        if (shape_fits(e, W, N))
            return e;
    }
    return nullptr;
}

// Decode-latency plan for one or a few rows (measured on the 1536-wide
// stack): 64-byte tiles so that enough workgroups share the active columns;
// short rows (<= 32 mask words) in 256-thread workgroups without a K-split,
// long rows in 1024-thread workgroups with K-slices of 24 words.
const ShapeEntry* latency_shape(const void* W, int64_t N, int wpr)
{
    const int code = wpr <= 32 ? SPIKE_SHAPE(4, 16, 8, 256) : SPIKE_SHAPE(4, 16, 4, 1024);
    const ShapeEntry* e = find_shape(code);
    return shape_fits(e, W, N) ? e : nullptr;
}
constexpr int kLatencySliceWords = 24;

constexpr int kMinTile = 32;  // smallest tile of any shape: sizes the counter array

// Smallest batch that AUTO sends to the matrix cores: every batch.  Measured
// per dependent call on the 1536 -> 1536 and 6144 -> 1536 shapes, the dense
// contraction is faster than the gather at every B up to 64 and every
// density from 0.02 to 0.40 (a batch-1 call is latency-bound: reading all of
// W at HBM rate costs less than the gather's compaction and K-split
// hand-off).
constexpr int kDefaultMfmaMinB = 1;

}  // namespace

struct spike_proj {
    const int8_t* W = nullptr;
    const float* scale = nullptr;
    int32_t K = 0, N = 0, wpr = 0;
    int device = 0;
    int32_t max_B = 0;
    int32_t* ws = nullptr;         // [max_B][N] INT32, zero between calls
    uint32_t* counters = nullptr;  // [max_B][counter_stride], zero between calls
    int32_t counter_stride = 0;
    int8_t* packed = nullptr;      // matrix-core operand copy of W (null: no matrix-core path)
    bool gather_only = false;      // created with SPIKE_CREATE_GATHER_ONLY: never holds the copy
    int path = SPIKE_PATH_AUTO;
    int slice_words = 0;  // 0 = automatic
    int max_slices = 16;
    const ShapeEntry* shape = nullptr;  // throughput shape (B above the latency range)
    bool shape_pinned = false;          // set by SPIKE_TUNE_SHAPE / _VEC: used for every B
    int tiles_per_unit = 1;
    int mfma_min_b = kDefaultMfmaMinB;
    int mfma_waves = 0;      // 0 = automatic
    int mfma_depth = 0;      // 0 = automatic
    int mfma_row_tile = 0;   // 16-row subtiles per workgroup, 0 = automatic
    int mfma_col_sets = 0;   // 16-channel sets per workgroup, 0 = automatic
};

struct spike_stream {
    int32_t n_proj = 0, n_sets = 0, n_tokens = 0, N = 0;
    const ShapeEntry* shape = nullptr;
    int tiles_per_unit = 1;
    int xcd_spread = 8;  // contiguous unit ranges per XCD (see k_stream)
    int max_wpr = 0;
    int device = 0;
    int64_t mask_stride = 0, out_stride = 0;
    bool buf = true;  // every weight matrix fits the buffer-resource kernels
    spk::StreamOperands* d_ops = nullptr;  // device operand table [n_sets][n_proj]
    spk::StreamLayout layout{};
    std::vector<const void*> weights;  // to re-check alignment when the shape changes
};

namespace {

template <class S, bool ACC, bool BUF>
void launch_gather_t(const spike_proj* h, const uint64_t* mask, int32_t B, int sw, int n_slices, int n_tiles,
                     int tpu, float* out, int32_t* acc, hipStream_t st)
{
    const size_t dyn = spk::unit_dyn_lds<S>(sw, tpu);
    const int64_t groups = (n_tiles + tpu - 1) / tpu;
    const int64_t units = (int64_t)B * groups * n_slices;
    hipLaunchKernelGGL((spk::k_gather<S, ACC, BUF>), dim3((unsigned)units), dim3(S::BLOCK), dyn, st, h->W, h->scale,
                       h->K, h->N, mask, h->wpr, sw, n_slices, n_tiles, tpu, h->ws, h->counters, h->counter_stride,
                       out, acc);
}

template <class S, bool BUF>
void launch_stream_t(const spike_stream* s, int n_tiles, unsigned units, const uint64_t* masks, float* out,
                     hipStream_t st)
{
    const size_t dyn = spk::unit_dyn_lds<S>(s->max_wpr, s->tiles_per_unit);
    const int n_items = s->n_tokens * s->n_proj;
    hipLaunchKernelGGL((spk::k_stream<S, BUF>), dim3(units), dim3(S::BLOCK), dyn, st, s->d_ops, s->layout, s->n_proj,
                       s->n_sets, s->N, n_tiles, s->tiles_per_unit, n_items, s->xcd_spread, masks, s->mask_stride,
                       out, s->out_stride);
}

int alloc_workspace(spike_proj* h, int32_t max_B)
{
    const size_t ws_bytes = (size_t)max_B * h->N * sizeof(int32_t);
    const int32_t stride = (int32_t)((h->N + kMinTile - 1) / kMinTile);
    const size_t ctr_bytes = (size_t)max_B * stride * sizeof(uint32_t);
    int32_t* ws = nullptr;
    uint32_t* ctr = nullptr;
    hipError_t e = hipMalloc(&ws, ws_bytes);
    if (e != hipSuccess)
        return fail(SPIKE_ENOMEM, "workspace allocation of %zu bytes failed: %s", ws_bytes, hipGetErrorString(e));
    e = hipMalloc(&ctr, ctr_bytes);
    if (e != hipSuccess) {
        (void)hipFree(ws);
        return fail(SPIKE_ENOMEM, "workspace allocation failed: %s", hipGetErrorString(e));
    }
    // Zeroed once here; the kernels leave both zeroed after every call.
    if ((e = hipMemset(ws, 0, ws_bytes)) != hipSuccess || (e = hipMemset(ctr, 0, ctr_bytes)) != hipSuccess ||
        (e = hipDeviceSynchronize()) != hipSuccess) {
        (void)hipFree(ws);
        (void)hipFree(ctr);
        return hip_fail(e, "workspace initialisation");
    }
    if (h->ws)
        (void)hipFree(h->ws);
    if (h->counters)
        (void)hipFree(h->counters);
    h->ws = ws;
    h->counters = ctr;
    h->counter_stride = stride;
    h->max_B = max_B;
    return SPIKE_OK;
}

int check_device(int want)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    if (dev != want)
        return fail(SPIKE_EINVAL, "handle was created on device %d but device %d is current", want, dev);
    return SPIKE_OK;
}

// K-slices for a gather over B rows: enough units to spread one row over the
// chip, capped so that the atomic traffic (slices * N * 4 bytes per row)
// stays a small fraction of the weight bytes.
int choose_slice_words(const spike_proj* h, int32_t B, int n_groups)
{
    int sw;
    if (h->slice_words > 0) {
        sw = h->slice_words;
    } else {
        const int64_t target_units = 2 * 256;
        const int64_t per_slice = (int64_t)B * n_groups;
        int64_t slices = (target_units + per_slice - 1) / per_slice;
        slices = std::max<int64_t>(1, std::min<int64_t>(slices, h->max_slices));
        sw = (int)((h->wpr + slices - 1) / slices);
    }
    return std::max(1, std::min(sw, std::min(h->wpr, spk::kMaxSliceWords)));
}

// Launch plan of the gather for B rows: shape, mask words per K-slice and
// tiles per workgroup.  Tuning knobs override the automatic choices.
struct GatherPlan {
    const ShapeEntry* shape;
    int sw, n_slices, n_tiles, tpu;
};

constexpr int kLatencyRows = 4;  // up to this many rows use the decode-latency plan

GatherPlan plan_gather(const spike_proj* h, int32_t B)
{
    GatherPlan p{};
    p.shape = h->shape;
    bool latency = false;
    if (!h->shape_pinned && B <= kLatencyRows && h->wpr <= spk::kMaxSliceWords) {
        if (const ShapeEntry* e = latency_shape(h->W, h->N, h->wpr)) {
            p.shape = e;
            latency = true;
        }
    }
    const int tile = shape_tile(p.shape);
    p.n_tiles = (int)((h->N + tile - 1) / tile);
    p.tpu = std::min(h->tiles_per_unit, p.n_tiles);
    const int n_groups = (p.n_tiles + p.tpu - 1) / p.tpu;
    if (h->slice_words > 0)
        p.sw = std::min(h->slice_words, std::min(h->wpr, spk::kMaxSliceWords));
    else if (latency)
        p.sw = h->wpr <= 32 ? h->wpr : kLatencySliceWords;
    else if (h->wpr <= spk::kMaxSliceWords)
        p.sw = h->wpr;  // enough rows x tiles to fill the chip without a K-split
    else
        p.sw = choose_slice_words(h, B, n_groups);
    p.n_slices = (int)((h->wpr + p.sw - 1) / p.sw);
    return p;
}

template <bool ACC>
int launch_gather(const spike_proj* h, const uint64_t* mask, int32_t B, float* out, int32_t* acc, hipStream_t st)
{
    const GatherPlan p = plan_gather(h, B);
    const int n_groups = (p.n_tiles + p.tpu - 1) / p.tpu;
    const int64_t units = (int64_t)B * n_groups * p.n_slices;
    if (units > 0x7fffffff)
        return fail(SPIKE_EUNSUPPORTED, "launch of %lld workgroups is too large", (long long)units);
    const int buf = fits_buffer(h->K, h->N) ? 1 : 0;
    (ACC ? p.shape->gather_acc[buf] : p.shape->gather[buf])(h, mask, B, p.sw, p.n_slices, p.n_tiles, p.tpu, out, acc,
                                                             st);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "gather launch");
}

spk::MfmaPlan mfma_plan_of(const spike_proj* h, int32_t B)
{
    return spk::mfma_plan(h->K, h->N, B, h->mfma_row_tile, h->mfma_col_sets, h->mfma_waves, h->mfma_depth);
}

// Why the matrix-core path cannot serve B rows of a K x N projection with
// plan p (null: it can).  The kernel addresses the spike words of its row
// tiles (including the padding rows of the last one) with 31-bit offsets.
const char* mfma_refusal(int32_t K, int32_t N, bool has_copy, int32_t B, const spk::MfmaPlan& p)
{
    if (!has_copy)
        return "the handle has no matrix-core copy of W (it needs N % 16 == 0, fewer than 2^31 packed bytes, "
               "a reserved batch of at least the matrix-core minimum and the memory for the copy)";
    if (const char* why = spk::mfma_plan_check(p, K, N))
        return why;
    const int64_t tile = 16ll * p.rt;
    const int64_t rows = ((int64_t)B + tile - 1) / tile * tile;
    if (rows * words_per_row(K) * (int64_t)sizeof(uint64_t) >= (1ll << 31))
        return "the spike rows exceed 31-bit offsets";
    return nullptr;
}

// AUTO sends batches from mfma_min_b rows to the matrix cores whenever
// their plan can run, and everything else to the gather.
bool auto_uses_mfma(int32_t K, int32_t N, bool has_copy, int32_t B, int min_b, const spk::MfmaPlan& p)
{
    return B >= min_b && mfma_refusal(K, N, has_copy, B, p) == nullptr;
}

bool use_mfma(const spike_proj* h, int32_t B)
{
    if (h->path == SPIKE_PATH_MFMA)
        return true;
    if (h->path == SPIKE_PATH_GATHER)
        return false;
    return auto_uses_mfma(h->K, h->N, h->packed != nullptr, B, h->mfma_min_b, mfma_plan_of(h, B));
}

// Packed operand copy of W for the matrix cores (layout in mfma.hpp), made
// once; null where the shape has no matrix-core path or memory is short.
int make_packed(spike_proj* h)
{
    if (!spk::mfma_supported(h->K, h->N))
        return SPIKE_OK;
    const int64_t bytes = spk::mfma_packed_bytes(h->K, h->N);
    int8_t* P = nullptr;
    if (hipMalloc(&P, (size_t)bytes) != hipSuccess) {
        (void)hipGetLastError();  // no matrix-core path for this handle; the gather serves every B
        return SPIKE_OK;
    }
    const int64_t chunks = bytes / 16;
    const int64_t blocks = (chunks + spk::kPackBlock - 1) / spk::kPackBlock;
    hipError_t e = hipDeviceSynchronize();  // W may still be in flight on any stream
    if (e == hipSuccess) {
        hipLaunchKernelGGL(spk::k_mfma_pack, dim3((unsigned)blocks), dim3(spk::kPackBlock), 0, nullptr, h->W, h->K,
                           h->N, h->wpr, P, chunks);
        e = hipGetLastError();
    }
    if (e == hipSuccess)
        e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        (void)hipFree(P);
        return hip_fail(e, "packing the matrix-core copy of W");
    }
    h->packed = P;
    return SPIKE_OK;
}

template <bool ACC>
int forward_impl(spike_proj* h, const uint64_t* mask, int32_t B, float* out, int32_t* acc, void* stream)
{
    if (!h)
        return fail(SPIKE_EINVAL, "null handle");
    if (B < 0 || B > h->max_B)
        return fail(SPIKE_EINVAL, "B = %d outside [0, %d] (reserve more rows with spike_proj_reserve)", B, h->max_B);
    if (B == 0)
        return SPIKE_OK;
    if (!mask || (ACC ? !acc : !out))
        return fail(SPIKE_EINVAL, "null mask or output pointer");
    if (int rc = check_device(h->device))
        return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (use_mfma(h, B)) {
        const spk::MfmaPlan p = mfma_plan_of(h, B);
        if (const char* why = mfma_refusal(h->K, h->N, h->packed != nullptr, B, p))
            return fail(SPIKE_EUNSUPPORTED, "matrix-core path for B = %d, K = %d, N = %d (row tile %d, channel sets "
                        "%d, waves %d, depth %d): %s", B, h->K, h->N, p.rt, p.cs, p.kw, p.d, why);
        const hipError_t e = spk::launch_mfma(p, h->packed, h->scale, h->K, h->N, mask, B, out, acc, ACC, st);
        return e == hipSuccess ? SPIKE_OK : hip_fail(e, "matrix-core launch");
    }
    return launch_gather<ACC>(h, mask, B, out, acc, st);
}

// Shape codes accepted by the tuning calls: 0 = automatic.
int parse_shape(int value, const void* W, int64_t N, const ShapeEntry** out)
{
    const ShapeEntry* e = value == 0 ? default_shape(W, N, 0) : find_shape(value);
    if (!e)
        return fail(SPIKE_EINVAL, "shape code 0x%x is not instantiated", value);
    if (!shape_fits(e, W, N))
        return fail(SPIKE_EINVAL, "shape with %d-byte loads does not fit N = %lld and the weight alignment", e->vec,
                    (long long)N);
    *out = e;
    return SPIKE_OK;
}

}  // namespace

// Device memory of spike_proj_forward_noalloc: the INT32 partial sums and
// completion counters of a K-split gather, [B][N] words followed by
// [B][ceil(N/32)] counters.  One copy per GPU, held until the process ends.
// In host code `scratch` is only a symbol: its device address comes from
// hipGetSymbolAddress (per device, see static_scratch below).
static __device__ __align__(256) uint32_t scratch[SPIKE_STATIC_SCRATCH_WORDS];

__global__ __launch_bounds__(256) void k_zero_words(uint32_t* __restrict__ p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
        p[i] = 0u;
}

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
uint32_t* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device (null: not looked up yet)
bool g_scratch_clean[kMaxDevices];     // a clearing kernel has been enqueued outside graph capture

// Device address of the current device's scratch array.  The first call on a
// device looks it up; until one call has run outside graph capture, every
// call also enqueues a kernel on `st` that clears the array (captured calls
// then clear it on every replay).  After that the gather's own protocol
// leaves the array zeroed at the end of every call.
int static_scratch(int dev, hipStream_t st, uint32_t** out)
{
    if (dev < 0 || dev >= kMaxDevices)
        return fail(SPIKE_EUNSUPPORTED, "device ordinal %d is beyond the %d devices this library tracks", dev,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return hip_fail(e, "hipGetSymbolAddress(scratch)");
        g_scratch_ptr[dev] = static_cast<uint32_t*>(p);
    }
    if (!g_scratch_clean[dev]) {
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(st, &cs);
        if (e != hipSuccess)
            return hip_fail(e, "hipStreamIsCapturing");
        hipLaunchKernelGGL(k_zero_words, dim3(256), dim3(256), 0, st, g_scratch_ptr[dev],
                           (int64_t)SPIKE_STATIC_SCRATCH_WORDS);
        if ((e = hipGetLastError()) != hipSuccess)
            return hip_fail(e, "scratch clearing launch");
        if (cs == hipStreamCaptureStatusNone)
            g_scratch_clean[dev] = true;
    }
    *out = g_scratch_ptr[dev];
    return SPIKE_OK;
}

}  // namespace

extern "C" {

int spike_proj_create_reserved(const int8_t* W, const float* scale, int32_t K, int32_t N, int32_t max_B,
                               int32_t flags, spike_proj_t* out_handle)
{
    spk::last_error.clear();
    if (!out_handle)
        return fail(SPIKE_EINVAL, "null out_handle");
    *out_handle = nullptr;
    if (!W || !scale)
        return fail(SPIKE_EINVAL, "null weight or scale pointer");
    if (K < 1 || K > SPIKE_MAX_K)
        return fail(SPIKE_EINVAL, "K = %d outside [1, %d]", K, SPIKE_MAX_K);
    if (N < 1 || N > SPIKE_MAX_N)
        return fail(SPIKE_EINVAL, "N = %d outside [1, %d]", N, SPIKE_MAX_N);
    if (max_B < 1 || max_B > 65535)
        return fail(SPIKE_EINVAL, "max_B = %d outside [1, 65535]", max_B);
    if (flags & ~SPIKE_CREATE_GATHER_ONLY)
        return fail(SPIKE_EINVAL, "unknown create flags 0x%x", flags);
    spike_proj* h = new (std::nothrow) spike_proj;
    if (!h)
        return fail(SPIKE_ENOMEM, "handle allocation failed");
    h->W = W;
    h->scale = scale;
    h->K = K;
    h->N = N;
    h->wpr = (int32_t)words_per_row(K);
    h->shape = default_shape(W, N, 0);
    h->gather_only = (flags & SPIKE_CREATE_GATHER_ONLY) != 0;
    hipError_t e = hipGetDevice(&h->device);
    if (e != hipSuccess) {
        delete h;
        return hip_fail(e, "hipGetDevice");
    }
    if (int rc = alloc_workspace(h, max_B)) {
        delete h;
        return rc;
    }
    // the matrix-core copy of W only where batches that use it can be run
    if (!h->gather_only && max_B >= h->mfma_min_b) {
        if (int rc = make_packed(h)) {
            (void)hipFree(h->ws);
            (void)hipFree(h->counters);
            delete h;
            return rc;
        }
    }
    *out_handle = h;
    return SPIKE_OK;
}

int spike_proj_create(const int8_t* W, const float* scale, int32_t K, int32_t N, spike_proj_t* out_handle)
{
    return spike_proj_create_reserved(W, scale, K, N, SPIKE_DEFAULT_MAX_B, 0, out_handle);
}

int spike_proj_reserve(spike_proj_t h, int32_t max_B)
{
    spk::last_error.clear();
    if (!h)
        return fail(SPIKE_EINVAL, "null handle");
    if (max_B < 1 || max_B > 65535)
        return fail(SPIKE_EINVAL, "max_B = %d outside [1, 65535]", max_B);
    if (max_B == h->max_B &&
        (h->gather_only || max_B < h->mfma_min_b || h->packed || !spk::mfma_supported(h->K, h->N)))
        return SPIKE_OK;
    if (int rc = check_device(h->device))
        return rc;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess)
        return hip_fail(e, "hipDeviceSynchronize");
    if (int rc = alloc_workspace(h, max_B))
        return rc;
    // The matrix-core copy of W is kept only while batches that would use it
    // can be run: fewer reserved rows than the matrix-core minimum free it.
    if (h->gather_only || max_B < h->mfma_min_b) {
        if (h->packed)
            (void)hipFree(h->packed);
        h->packed = nullptr;
        return SPIKE_OK;
    }
    return h->packed ? SPIKE_OK : make_packed(h);
}

int spike_proj_forward(spike_proj_t h, const uint64_t* mask, int32_t B, float* out, void* stream)
{
    return forward_impl<false>(h, mask, B, out, nullptr, stream);
}

int spike_proj_forward_acc(spike_proj_t h, const uint64_t* mask, int32_t B, int32_t* acc, void* stream)
{
    return forward_impl<true>(h, mask, B, nullptr, acc, stream);
}

int spike_proj_forward_noalloc(const int8_t* W, const float* scale, int32_t K, int32_t N, const uint64_t* mask,
                               int32_t B, float* out, void* stream)
{
    spk::last_error.clear();
    if (K < 1 || K > SPIKE_MAX_K)
        return fail(SPIKE_EINVAL, "K = %d outside [1, %d]", K, SPIKE_MAX_K);
    if (N < 1 || N > SPIKE_MAX_N)
        return fail(SPIKE_EINVAL, "N = %d outside [1, %d]", N, SPIKE_MAX_N);
    if (B < 0)
        return fail(SPIKE_EINVAL, "B = %d < 0", B);
    const int64_t stride = (N + kMinTile - 1) / kMinTile;
    const int64_t words = (int64_t)B * ((int64_t)N + stride);
    if (words > SPIKE_STATIC_SCRATCH_WORDS)
        return fail(SPIKE_EINVAL,
                    "B * (N + ceil(N/32)) = %lld words exceeds the %d-word static scratch (B = %d, N = %d)",
                    (long long)words, SPIKE_STATIC_SCRATCH_WORDS, B, N);
    if (B == 0)
        return SPIKE_OK;
    if (!W || !scale || !mask || !out)
        return fail(SPIKE_EINVAL, "null weight, scale, mask or output pointer");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipGetDevice");
    hipStream_t st = static_cast<hipStream_t>(stream);
    uint32_t* ws = nullptr;
    if (int rc = static_scratch(dev, st, &ws))
        return rc;
    // A handle on the stack over the borrowed operands and the static
    // scratch: the gather's planner and kernels are those of spike_proj_forward.
    spike_proj h;
    h.W = W;
    h.scale = scale;
    h.K = K;
    h.N = N;
    h.wpr = (int32_t)words_per_row(K);
    h.device = dev;
    h.max_B = B;
    h.ws = reinterpret_cast<int32_t*>(ws);
    h.counters = ws + (int64_t)B * N;
    h.counter_stride = (int32_t)stride;
    h.path = SPIKE_PATH_GATHER;
    h.shape = default_shape(W, N, 0);
    return launch_gather<false>(&h, mask, B, out, nullptr, st);
}

int spike_proj_destroy(spike_proj_t h)
{
    if (!h)
        return SPIKE_OK;
    int rc = SPIKE_OK;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess)
        rc = hip_fail(e, "hipDeviceSynchronize");
    if (h->ws)
        (void)hipFree(h->ws);
    if (h->counters)
        (void)hipFree(h->counters);
    if (h->packed)
        (void)hipFree(h->packed);
    delete h;
    return rc;
}

int spike_proj_tune(spike_proj_t h, int32_t key, int32_t value)
{
    spk::last_error.clear();
    if (!h)
        return fail(SPIKE_EINVAL, "null handle");
    switch (key) {
    case SPIKE_TUNE_PATH:
        if (value != SPIKE_PATH_AUTO && value != SPIKE_PATH_GATHER && value != SPIKE_PATH_MFMA)
            return fail(SPIKE_EINVAL, "unknown path %d", value);
        h->path = value;
        return SPIKE_OK;
    case SPIKE_TUNE_SLICE_WORDS:
        if (value < 0 || value > spk::kMaxSliceWords)
            return fail(SPIKE_EINVAL, "slice words %d outside [0, %d]", value, spk::kMaxSliceWords);
        h->slice_words = value;
        return SPIKE_OK;
    case SPIKE_TUNE_MFMA_MIN_B:
        if (value < 1)
            return fail(SPIKE_EINVAL, "matrix-core minimum batch must be >= 1");
        h->mfma_min_b = value;
        return SPIKE_OK;
    case SPIKE_TUNE_VEC: {
        if (value != 0 && value != 1 && value != 4 && value != 8 && value != 16)
            return fail(SPIKE_EINVAL, "vector width %d is not 0, 1, 4, 8 or 16", value);
        const ShapeEntry* e = default_shape(h->W, h->N, value);
        if (!e)
            return fail(SPIKE_EINVAL, "vector width %d does not fit N = %d and the weight alignment", value, h->N);
        h->shape = e;
        h->shape_pinned = value != 0;
        return SPIKE_OK;
    }
    case SPIKE_TUNE_MAX_SLICES:
        if (value < 1 || value > 4096)
            return fail(SPIKE_EINVAL, "max slices %d outside [1, 4096]", value);
        h->max_slices = value;
        return SPIKE_OK;
    case SPIKE_TUNE_SHAPE:
        if (int rc = parse_shape(value, h->W, h->N, &h->shape))
            return rc;
        h->shape_pinned = value != 0;
        return SPIKE_OK;
    case SPIKE_TUNE_TILES_PER_UNIT:
        if (value < 1 || value > 4096)
            return fail(SPIKE_EINVAL, "tiles per unit %d outside [1, 4096]", value);
        h->tiles_per_unit = value;
        return SPIKE_OK;
    case SPIKE_TUNE_MFMA_DEPTH:
        if (value != 0 && value != 2 && value != 3 && value != 4 && value != 6 && value != 8 && value != 12)
            return fail(SPIKE_EINVAL, "matrix-core depth must be 0, 2, 3, 4, 6, 8 or 12, got %d", value);
        h->mfma_depth = value;
        return SPIKE_OK;
    case SPIKE_TUNE_MFMA_WAVES:
        if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8 && value != 16)
            return fail(SPIKE_EINVAL, "matrix-core waves per workgroup must be 0, 1, 2, 4, 8 or 16, got %d", value);
        h->mfma_waves = value;
        return SPIKE_OK;
    case SPIKE_TUNE_MFMA_ROW_TILE:
        if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8)
            return fail(SPIKE_EINVAL, "matrix-core row subtiles must be 0, 1, 2, 4 or 8, got %d", value);
        h->mfma_row_tile = value;
        return SPIKE_OK;
    case SPIKE_TUNE_MFMA_COL_SETS:
        if (value < 0 || value > 6 || value == 5)
            return fail(SPIKE_EINVAL, "matrix-core channel sets must be 0, 1, 2, 3, 4 or 6, got %d", value);
        h->mfma_col_sets = value;
        return SPIKE_OK;
    default:
        return fail(SPIKE_EINVAL, "unknown tuning key %d", key);
    }
}

int spike_compact(const uint64_t* mask, int32_t B, int32_t K, int32_t* active_idx, int32_t* active_count,
                  void* stream)
{
    spk::last_error.clear();
    if (B < 0 || K < 1 || K > SPIKE_MAX_K)
        return fail(SPIKE_EINVAL, "B = %d or K = %d out of range", B, K);
    if (B == 0)
        return SPIKE_OK;
    if (!mask || !active_idx || !active_count)
        return fail(SPIKE_EINVAL, "null pointer");
    hipLaunchKernelGGL(spk::k_compact, dim3((unsigned)B), dim3(spk::kCompactBlock), 0,
                       static_cast<hipStream_t>(stream), mask, K, (int)words_per_row(K), active_idx, active_count);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "compaction launch");
}

int spike_stack_forward(const spike_proj_t* projs, int32_t n_proj, const uint64_t* masks, int32_t B, float* out,
                        void* stream)
{
    spk::last_error.clear();
    if (!projs || n_proj < 1)
        return fail(SPIKE_EINVAL, "need at least one projection");
    if (B < 0)
        return fail(SPIKE_EINVAL, "B = %d < 0", B);
    for (int j = 0; j < n_proj; ++j) {
        if (!projs[j])
            return fail(SPIKE_EINVAL, "projection %d is null", j);
        if (B > projs[j]->max_B)
            return fail(SPIKE_EINVAL, "B = %d exceeds projection %d's reserved %d rows", B, j, projs[j]->max_B);
    }
    if (B == 0)
        return SPIKE_OK;
    if (!masks || !out)
        return fail(SPIKE_EINVAL, "null mask or output pointer");
    int64_t moff = 0, ooff = 0;
    for (int j = 0; j < n_proj; ++j) {
        if (int rc = spike_proj_forward(projs[j], masks + moff, B, out + ooff, stream))
            return rc;
        moff += (int64_t)B * projs[j]->wpr;
        ooff += (int64_t)B * projs[j]->N;
    }
    return SPIKE_OK;
}

int spike_stack_forward_fused(const spike_proj_t* projs, int32_t n_proj, const uint64_t* masks, int32_t B,
                              float* out, void* stream)
{
    spk::last_error.clear();
    if (!projs || n_proj < 1)
        return fail(SPIKE_EINVAL, "need at least one projection");
    if (n_proj > spk::kMfmaMaxItems)
        return fail(SPIKE_EUNSUPPORTED, "a fused launch holds at most %d projections", spk::kMfmaMaxItems);
    if (B < 0)
        return fail(SPIKE_EINVAL, "B = %d < 0", B);
    for (int j = 0; j < n_proj; ++j) {
        if (!projs[j])
            return fail(SPIKE_EINVAL, "projection %d is null", j);
        if (B > projs[j]->max_B)
            return fail(SPIKE_EINVAL, "B = %d exceeds projection %d's reserved %d rows", B, j, projs[j]->max_B);
    }
    if (B == 0)
        return SPIKE_OK;
    if (!masks || !out)
        return fail(SPIKE_EINVAL, "null mask or output pointer");
    const int32_t N = projs[0]->N;
    int32_t min_K = projs[0]->K;
    int max_wpr = 0;
    for (int j = 0; j < n_proj; ++j) {
        if (projs[j]->N != N)
            return fail(SPIKE_EUNSUPPORTED, "all projections of a fused launch must share N (%d vs %d)", projs[j]->N, N);
        if (projs[j]->device != projs[0]->device)
            return fail(SPIKE_EINVAL, "projections live on different devices");
        min_K = std::min(min_K, projs[j]->K);
        max_wpr = std::max(max_wpr, projs[j]->wpr);
    }
    if (int rc = check_device(projs[0]->device))
        return rc;
    // one ring plan for all items, chosen for the shortest K (every wave needs a k-step)
    // Tiles of up to 64 rows by 48 channels, two k-steps in flight per wave;
    // 8 waves for 64-row tiles (measured on the 64-row decode stack, 1408
    // workgroups over 44 projections: 49 us per step against 57 us with 16
    // waves, 53 with 4), 16 for the narrower tiles of smaller batches; the
    // first handle's matrix-core tuning knobs override it for the whole
    // launch.
    const spike_proj* h0 = projs[0];
    const int sets = N / spk::kMfmaNAlign;
    spk::MfmaPlan p{};
    p.rt = B <= 16 ? 1 : B <= 32 ? 2 : 4;
    p.cs = sets % 3 == 0 ? 3 : sets % 2 == 0 ? 2 : 1;
    p.kw = p.rt >= 4 ? 8 : 16;
    p.d = 2;
    if (h0->mfma_row_tile > 0)
        p.rt = h0->mfma_row_tile;
    if (h0->mfma_col_sets > 0)
        p.cs = h0->mfma_col_sets;
    if (h0->mfma_waves > 0)
        p.kw = h0->mfma_waves;
    if (h0->mfma_depth > 0)
        p.d = h0->mfma_depth;
    if (N % spk::kMfmaNAlign != 0 || !spk::mfma_ring_plan(p, (int)words_per_row(min_K), N))
        return fail(SPIKE_EUNSUPPORTED, "no matrix-core plan serves N = %d, K >= %d, B = %d in one launch", N, min_K, B);
    spk::MfmaItems items{};
    int64_t moff = 0, ooff = 0;
    for (int j = 0; j < n_proj; ++j) {
        const spike_proj* h = projs[j];
        if (const char* why = mfma_refusal(h->K, N, h->packed != nullptr, B, p))
            return fail(SPIKE_EUNSUPPORTED, "projection %d (K = %d) cannot run on the matrix cores with B = %d: %s", j,
                        h->K, B, why);
        items.P[j] = h->packed;
        items.scale[j] = h->scale;
        items.mask_off[j] = moff;
        items.out_off[j] = ooff;
        items.wpr[j] = h->wpr;
        moff += (int64_t)B * h->wpr;
        ooff += (int64_t)B * N;
    }
    if (spk::mfma_lds_bytes(p.rt, p.cs, max_wpr) > spk::kMfmaMaxLds)
        return fail(SPIKE_EUNSUPPORTED, "the staged spike words of the longest projection exceed the LDS budget");
    const hipError_t e = spk::launch_mfma_items(p, items, n_proj, max_wpr, N, masks, B, out,
                                                static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "fused matrix-core launch");
}

int spike_stream_create(const spike_proj_t* projs, int32_t n_proj, int32_t n_sets, int32_t n_tokens,
                        spike_stream_t* out_stream)
{
    spk::last_error.clear();
    if (!out_stream)
        return fail(SPIKE_EINVAL, "null out_stream");
    *out_stream = nullptr;
    if (!projs || n_proj < 1 || n_sets < 1 || n_tokens < 1)
        return fail(SPIKE_EINVAL, "n_proj, n_sets and n_tokens must be >= 1");
    if (n_proj > spk::kStreamMaxProj)
        return fail(SPIKE_EUNSUPPORTED, "a stream holds at most %d projections per token", spk::kStreamMaxProj);
    const int64_t n_handles = (int64_t)n_proj * n_sets;
    if (!projs[0])
        return fail(SPIKE_EINVAL, "projection 0 is null");
    const int32_t N = projs[0]->N;
    int max_wpr = 0;
    bool buf = true;
    std::vector<const void*> weights;
    for (int64_t i = 0; i < n_handles; ++i) {
        const spike_proj* p = projs[i];
        if (!p)
            return fail(SPIKE_EINVAL, "projection %lld is null", (long long)i);
        if (p->N != N)
            return fail(SPIKE_EUNSUPPORTED, "all projections of a stream must share N (%d vs %d)", p->N, N);
        const spike_proj* first = projs[i % n_proj];
        if (!first || p->K != first->K)
            return fail(SPIKE_EINVAL, "set %lld projection %lld has a different K from set 0", (long long)(i / n_proj),
                        (long long)(i % n_proj));
        if (p->wpr > spk::kMaxSliceWords)
            return fail(SPIKE_EUNSUPPORTED, "stream projections need K <= %d", 64 * spk::kMaxSliceWords);
        max_wpr = std::max(max_wpr, p->wpr);
        buf = buf && fits_buffer(p->K, p->N);
        weights.push_back(p->W);
    }
    // the widest default shape whose loads fit every weight matrix
    const ShapeEntry* shape = nullptr;
    for (int vec : {16, 8, 4, 1}) {
        const ShapeEntry* e = default_shape(weights[0], N, vec);
        if (!e || (vec == 16 && N % 512 != 0))
            continue;
        bool ok = true;
        for (const void* w : weights)
            ok = ok && shape_fits(e, w, N);
        if (ok) {
            shape = e;
            break;
        }
    }
    const int tile = shape_tile(shape);
    const int64_t n_tiles = (N + tile - 1) / tile;
    if (((int64_t)n_tokens * n_proj + 8) * n_tiles > 0x7fffffff)
        return fail(SPIKE_EUNSUPPORTED, "stream of %d tokens is too large for one launch", n_tokens);
    std::vector<spk::StreamOperands> ops((size_t)n_handles);
    int64_t moff = 0;
    spike_stream* s = new (std::nothrow) spike_stream;
    if (!s)
        return fail(SPIKE_ENOMEM, "stream allocation failed");
    for (int j = 0; j < n_proj; ++j) {
        for (int set = 0; set < n_sets; ++set) {
            const spike_proj* p = projs[(int64_t)set * n_proj + j];
            ops[(size_t)set * n_proj + j] = spk::StreamOperands{p->W, p->scale};
        }
        s->layout.K[j] = projs[j]->K;
        s->layout.mask_off[j] = (int32_t)std::min<int64_t>(moff, 0x7fffffff);
        moff += projs[j]->wpr;
    }
    if (moff > 0x7fffffff) {
        delete s;
        return fail(SPIKE_EUNSUPPORTED, "token mask stride too large");
    }
    s->n_proj = n_proj;
    s->n_sets = n_sets;
    s->n_tokens = n_tokens;
    s->N = N;
    s->shape = shape;
    s->max_wpr = max_wpr;
    s->buf = buf;
    s->mask_stride = moff;
    s->out_stride = (int64_t)n_proj * N;
    s->weights = std::move(weights);
    const size_t ops_bytes = ops.size() * sizeof(spk::StreamOperands);
    hipError_t e = hipGetDevice(&s->device);
    if (e == hipSuccess)
        e = hipMalloc(&s->d_ops, ops_bytes);
    if (e == hipSuccess)
        e = hipMemcpy(s->d_ops, ops.data(), ops_bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        if (s->d_ops)
            (void)hipFree(s->d_ops);
        delete s;
        return hip_fail(e, "stream operand table upload");
    }
    *out_stream = s;
    return SPIKE_OK;
}

int spike_stream_tune(spike_stream_t s, int32_t key, int32_t value)
{
    spk::last_error.clear();
    if (!s)
        return fail(SPIKE_EINVAL, "null stream handle");
    switch (key) {
    case SPIKE_TUNE_SHAPE: {
        const ShapeEntry* e = nullptr;
        for (const void* w : s->weights)
            if (int rc = parse_shape(value, w, s->N, &e))
                return rc;
        const int64_t n_tiles = (s->N + shape_tile(e) - 1) / shape_tile(e);
        if (((int64_t)s->n_tokens * s->n_proj + 8) * n_tiles > 0x7fffffff)
            return fail(SPIKE_EUNSUPPORTED, "shape makes the launch too large");
        s->shape = e;
        return SPIKE_OK;
    }
    case SPIKE_TUNE_TILES_PER_UNIT:
        if (value < 1 || value > 4096)
            return fail(SPIKE_EINVAL, "tiles per unit %d outside [1, 4096]", value);
        s->tiles_per_unit = value;
        return SPIKE_OK;
    case SPIKE_TUNE_XCD_SPREAD:
        if (value != 1 && value != 8)
            return fail(SPIKE_EINVAL, "xcd spread must be 1 or 8, got %d", value);
        s->xcd_spread = value;
        return SPIKE_OK;

    default:
        return fail(SPIKE_EINVAL, "key %d does not apply to a stream", key);
    }
}

int spike_stream_forward(spike_stream_t s, const uint64_t* masks, float* out, void* stream)
{
    spk::last_error.clear();
    if (!s)
        return fail(SPIKE_EINVAL, "null stream handle");
    if (!masks || !out)
        return fail(SPIKE_EINVAL, "null mask or output pointer");
    if (int rc = check_device(s->device))
        return rc;
    const int tile = shape_tile(s->shape);
    const int n_tiles = (s->N + tile - 1) / tile;
    const int tpu = std::min(s->tiles_per_unit, n_tiles);
    const int n_groups = (n_tiles + tpu - 1) / tpu;
    const int64_t n_items = (int64_t)s->n_tokens * s->n_proj;
    const int64_t n_units = n_items * n_groups;
    const unsigned units = (unsigned)((n_units + s->xcd_spread - 1) / s->xcd_spread * s->xcd_spread);
    const int saved = s->tiles_per_unit;
    s->tiles_per_unit = tpu;  // launch with the clamped value
    s->shape->stream[s->buf ? 1 : 0](s, n_tiles, units, masks, out, static_cast<hipStream_t>(stream));
    s->tiles_per_unit = saved;
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "stream launch");
}

int spike_stream_destroy(spike_stream_t s)
{
    if (!s)
        return SPIKE_OK;
    int rc = SPIKE_OK;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess)
        rc = hip_fail(e, "hipDeviceSynchronize");
    if (s->d_ops)
        (void)hipFree(s->d_ops);
    delete s;
    return rc;
}

int spike_proj_shapes(int32_t* codes, int32_t cap)
{
    const int n = (int)(sizeof kShapes / sizeof kShapes[0]);
    for (int i = 0; i < n && i < cap && codes; ++i)
        codes[i] = kShapes[i].code;
    return n;
}

int spike_mfma_plans(int32_t* codes, int32_t cap) { return spk::mfma_plan_codes(codes, cap); }

int spike_proj_plan_query(int32_t K, int32_t N, int32_t B, int32_t* path, int32_t* plan)
{
    spk::last_error.clear();
    if (!path || !plan)
        return fail(SPIKE_EINVAL, "null output pointer");
    if (K < 1 || K > SPIKE_MAX_K || N < 1 || N > SPIKE_MAX_N || B < 0)
        return fail(SPIKE_EINVAL, "K = %d, N = %d or B = %d out of range", K, N, B);
    const spk::MfmaPlan p = spk::mfma_plan(K, N, B, 0, 0, 0, 0);
    const bool mf = auto_uses_mfma(K, N, spk::mfma_supported(K, N), B, kDefaultMfmaMinB, p);
    *path = mf ? SPIKE_PATH_MFMA : SPIKE_PATH_GATHER;
    *plan = mf ? spk::mfma_plan_code(p) : 0;
    return SPIKE_OK;
}

const char* spike_proj_last_error(void) { return spk::last_error.c_str(); }

int spike_proj_abi_version(void) { return SPIKE_PROJ_ABI_VERSION; }

}  // extern "C"
