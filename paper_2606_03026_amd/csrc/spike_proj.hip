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
#include <new>
#include <string>
#include <vector>

#include "gather.hpp"
#include "mfma.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

int hip_fail(hipError_t e, const char* what)
{
    return fail(SPIKE_EHIP, "%s: %s", what, hipGetErrorString(e));
}

int64_t words_per_row(int64_t K) { return (K + 63) / 64; }

// Launch shapes of the gather: V bytes per lane, LG lanes per column group.
enum GatherShape { SHAPE_V16_LG32 = 16, SHAPE_V8_LG64 = 8, SHAPE_V4_LG64 = 4, SHAPE_V1_LG64 = 1 };

int shape_tile(int shape)
{
    switch (shape) {
    case SHAPE_V16_LG32: return 16 * 32;
    case SHAPE_V8_LG64: return 8 * 64;
    case SHAPE_V4_LG64: return 4 * 64;
    default: return 64;
    }
}

// Widest vector whose loads stay aligned and in range for this matrix.
int pick_shape(const void* W, int64_t N, int requested)
{
    const uintptr_t a = reinterpret_cast<uintptr_t>(W);
    auto ok = [&](int v) { return N % v == 0 && a % v == 0; };
    if (requested == 16 || requested == 8 || requested == 4 || requested == 1)
        return ok(requested) ? requested : -1;
    if (requested != 0)
        return -1;
    if (ok(16) && N % 512 == 0)
        return SHAPE_V16_LG32;
    if (ok(8))
        return SHAPE_V8_LG64;
    if (ok(4))
        return SHAPE_V4_LG64;
    return SHAPE_V1_LG64;
}

constexpr int kMinTile = 64;  // smallest gather tile: sizes the counter array

}  // namespace

struct spike_proj {
    const int8_t* W = nullptr;
    const float* scale = nullptr;
    int32_t K = 0, N = 0, wpr = 0;
    int device = 0;
    int32_t max_B = 0;
    int32_t* ws = nullptr;          // [max_B][N] INT32, zero between calls
    uint32_t* counters = nullptr;   // [max_B][counter_stride], zero between calls
    int32_t counter_stride = 0;
    int path = SPIKE_PATH_AUTO;
    int slice_words = 0;            // 0 = automatic
    int max_slices = 16;
    int vec_request = 0;            // 0 = automatic
    int shape = SHAPE_V1_LG64;
    int mfma_min_b = 64;
};

struct spike_stream {
    int32_t n_proj = 0, n_sets = 0, n_tokens = 0, N = 0;
    int shape = SHAPE_V1_LG64;
    int max_wpr = 0;
    int device = 0;
    int64_t mask_stride = 0, out_stride = 0;
    spk::StreamDesc* d_desc = nullptr;
};

namespace {

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
        return fail(SPIKE_ENOMEM, "counter allocation of %zu bytes failed: %s", ctr_bytes, hipGetErrorString(e));
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
int choose_slice_words(const spike_proj* h, int32_t B, int n_tiles)
{
    int sw;
    if (h->slice_words > 0) {
        sw = h->slice_words;
    } else {
        const int64_t target_units = 2 * 256;
        int64_t slices = (target_units + (int64_t)B * n_tiles - 1) / ((int64_t)B * n_tiles);
        slices = std::max<int64_t>(1, std::min<int64_t>(slices, h->max_slices));
        sw = (int)((h->wpr + slices - 1) / slices);
    }
    sw = std::max(1, std::min(sw, std::min(h->wpr, spk::kMaxSliceWords)));
    return sw;
}

template <int V, int LG, bool ACC>
void launch_gather_t(const spike_proj* h, const uint64_t* mask, int32_t B, int sw, int n_slices, int n_tiles,
                     float* out, int32_t* acc, hipStream_t st)
{
    const size_t dyn = spk::unit_dyn_lds<V, LG>(sw);
    const int64_t units = (int64_t)B * n_tiles * n_slices;
    hipLaunchKernelGGL((spk::k_gather<V, LG, ACC>), dim3((unsigned)units), dim3(spk::kBlock), dyn, st, h->W,
                       h->scale, h->K, h->N, mask, h->wpr, sw, n_slices, n_tiles, h->ws, h->counters,
                       h->counter_stride, out, acc);
}

template <bool ACC>
int launch_gather(const spike_proj* h, const uint64_t* mask, int32_t B, float* out, int32_t* acc, hipStream_t st)
{
    const int n_tiles = (int)((h->N + shape_tile(h->shape) - 1) / shape_tile(h->shape));
    const int sw = choose_slice_words(h, B, n_tiles);
    const int n_slices = (int)((h->wpr + sw - 1) / sw);
    const int64_t units = (int64_t)B * n_tiles * n_slices;
    if (units > 0x7fffffff)
        return fail(SPIKE_EUNSUPPORTED, "launch of %lld workgroups is too large", (long long)units);
    switch (h->shape) {
    case SHAPE_V16_LG32: launch_gather_t<16, 32, ACC>(h, mask, B, sw, n_slices, n_tiles, out, acc, st); break;
    case SHAPE_V8_LG64: launch_gather_t<8, 64, ACC>(h, mask, B, sw, n_slices, n_tiles, out, acc, st); break;
    case SHAPE_V4_LG64: launch_gather_t<4, 64, ACC>(h, mask, B, sw, n_slices, n_tiles, out, acc, st); break;
    default: launch_gather_t<1, 64, ACC>(h, mask, B, sw, n_slices, n_tiles, out, acc, st); break;
    }
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "gather launch");
}

int use_mfma(const spike_proj* h, int32_t B)
{
    if (h->path == SPIKE_PATH_MFMA)
        return 1;
    if (h->path == SPIKE_PATH_GATHER)
        return 0;
    return spk::mfma_supported(h->K, h->N, h->W) && B >= h->mfma_min_b;
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
        if (!spk::mfma_supported(h->K, h->N, h->W))
            return fail(SPIKE_EUNSUPPORTED, "matrix-core path needs N %% %d == 0 and a %d-byte aligned W",
                        spk::kMfmaNAlign, spk::kMfmaNAlign);
        const hipError_t e = spk::launch_mfma(h->W, h->scale, h->K, h->N, mask, B, out, acc, ACC, st);
        return e == hipSuccess ? SPIKE_OK : hip_fail(e, "matrix-core launch");
    }
    return launch_gather<ACC>(h, mask, B, out, acc, st);
}

template <int V, int LG>
void launch_stream_t(const spike_stream* s, int n_tiles, unsigned units, const uint64_t* masks, float* out,
                     hipStream_t st)
{
    const size_t dyn = spk::unit_dyn_lds<V, LG>(s->max_wpr);
    hipLaunchKernelGGL((spk::k_stream<V, LG>), dim3(units), dim3(spk::kBlock), dyn, st, s->d_desc, s->n_proj, s->n_sets, s->N, n_tiles, masks, s->mask_stride, out,
                       s->out_stride);
}

}  // namespace

extern "C" {

int spike_proj_create(const int8_t* W, const float* scale, int32_t K, int32_t N, spike_proj_t* out_handle)
{
    g_last_error.clear();
    if (!out_handle)
        return fail(SPIKE_EINVAL, "null out_handle");
    *out_handle = nullptr;
    if (!W || !scale)
        return fail(SPIKE_EINVAL, "null weight or scale pointer");
    if (K < 1 || K > SPIKE_MAX_K)
        return fail(SPIKE_EINVAL, "K = %d outside [1, %d]", K, SPIKE_MAX_K);
    if (N < 1 || N > SPIKE_MAX_N)
        return fail(SPIKE_EINVAL, "N = %d outside [1, %d]", N, SPIKE_MAX_N);
    spike_proj* h = new (std::nothrow) spike_proj;
    if (!h)
        return fail(SPIKE_ENOMEM, "handle allocation failed");
    h->W = W;
    h->scale = scale;
    h->K = K;
    h->N = N;
    h->wpr = (int32_t)words_per_row(K);
    h->shape = pick_shape(W, N, 0);
    hipError_t e = hipGetDevice(&h->device);
    if (e != hipSuccess) {
        delete h;
        return hip_fail(e, "hipGetDevice");
    }
    if (int rc = alloc_workspace(h, SPIKE_DEFAULT_MAX_B)) {
        delete h;
        return rc;
    }
    *out_handle = h;
    return SPIKE_OK;
}

int spike_proj_reserve(spike_proj_t h, int32_t max_B)
{
    g_last_error.clear();
    if (!h)
        return fail(SPIKE_EINVAL, "null handle");
    if (max_B < 1 || max_B > 65535)
        return fail(SPIKE_EINVAL, "max_B = %d outside [1, 65535]", max_B);
    if (max_B == h->max_B)
        return SPIKE_OK;
    if (int rc = check_device(h->device))
        return rc;
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess)
        return hip_fail(e, "hipDeviceSynchronize");
    return alloc_workspace(h, max_B);
}

int spike_proj_forward(spike_proj_t h, const uint64_t* mask, int32_t B, float* out, void* stream)
{
    return forward_impl<false>(h, mask, B, out, nullptr, stream);
}

int spike_proj_forward_acc(spike_proj_t h, const uint64_t* mask, int32_t B, int32_t* acc, void* stream)
{
    return forward_impl<true>(h, mask, B, nullptr, acc, stream);
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
    delete h;
    return rc;
}

int spike_proj_tune(spike_proj_t h, int32_t key, int32_t value)
{
    g_last_error.clear();
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
        const int shape = pick_shape(h->W, h->N, value);
        if (shape < 0)
            return fail(SPIKE_EINVAL, "vector width %d does not fit N = %d and the weight alignment", value, h->N);
        h->vec_request = value;
        h->shape = shape;
        return SPIKE_OK;
    }
    case SPIKE_TUNE_MAX_SLICES:
        if (value < 1 || value > 4096)
            return fail(SPIKE_EINVAL, "max slices %d outside [1, 4096]", value);
        h->max_slices = value;
        return SPIKE_OK;
    default:
        return fail(SPIKE_EINVAL, "unknown tuning key %d", key);
    }
}

int spike_compact(const uint64_t* mask, int32_t B, int32_t K, int32_t* active_idx, int32_t* active_count,
                  void* stream)
{
    g_last_error.clear();
    if (B < 0 || K < 1 || K > SPIKE_MAX_K)
        return fail(SPIKE_EINVAL, "B = %d or K = %d out of range", B, K);
    if (B == 0)
        return SPIKE_OK;
    if (!mask || !active_idx || !active_count)
        return fail(SPIKE_EINVAL, "null pointer");
    if (B > 0x7fffffff / 1)
        return fail(SPIKE_EINVAL, "B too large");
    hipLaunchKernelGGL(spk::k_compact, dim3((unsigned)B), dim3(spk::kBlock), 0, static_cast<hipStream_t>(stream),
                       mask, K, (int)words_per_row(K), active_idx, active_count);
    const hipError_t e = hipGetLastError();
    return e == hipSuccess ? SPIKE_OK : hip_fail(e, "compaction launch");
}

int spike_stack_forward(const spike_proj_t* projs, int32_t n_proj, const uint64_t* masks, int32_t B, float* out,
                        void* stream)
{
    g_last_error.clear();
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

int spike_stream_create(const spike_proj_t* projs, int32_t n_proj, int32_t n_sets, int32_t n_tokens,
                        spike_stream_t* out_stream)
{
    g_last_error.clear();
    if (!out_stream)
        return fail(SPIKE_EINVAL, "null out_stream");
    *out_stream = nullptr;
    if (!projs || n_proj < 1 || n_sets < 1 || n_tokens < 1)
        return fail(SPIKE_EINVAL, "n_proj, n_sets and n_tokens must be >= 1");
    const int64_t n_handles = (int64_t)n_proj * n_sets;
    const int32_t N = projs[0] ? projs[0]->N : 0;
    int shape = SHAPE_V16_LG32;
    int max_wpr = 0;
    for (int64_t i = 0; i < n_handles; ++i) {
        const spike_proj* p = projs[i];
        if (!p)
            return fail(SPIKE_EINVAL, "projection %lld is null", (long long)i);
        if (p->N != N)
            return fail(SPIKE_EUNSUPPORTED, "all projections of a stream must share N (%d vs %d)", p->N, N);
        const spike_proj* first = projs[i % n_proj];
        if (p->K != first->K)
            return fail(SPIKE_EINVAL, "set %lld projection %lld has K = %d, set 0 has %d", (long long)(i / n_proj),
                        (long long)(i % n_proj), p->K, first->K);
        if (p->wpr > spk::kMaxSliceWords)
            return fail(SPIKE_EUNSUPPORTED, "stream projections need K <= %d", 64 * spk::kMaxSliceWords);
        shape = std::min(shape, pick_shape(p->W, N, 0));
        max_wpr = std::max(max_wpr, p->wpr);
    }
    const int tile = shape_tile(shape);
    const int64_t n_tiles = (N + tile - 1) / tile;
    if ((int64_t)n_tokens * n_proj * n_tiles > 0x7fffffff)
        return fail(SPIKE_EUNSUPPORTED, "stream of %d tokens is too large for one launch", n_tokens);
    std::vector<spk::StreamDesc> desc((size_t)n_handles);
    int64_t moff = 0;
    for (int j = 0; j < n_proj; ++j) {
        for (int set = 0; set < n_sets; ++set) {
            const spike_proj* p = projs[(int64_t)set * n_proj + j];
            spk::StreamDesc& d = desc[(size_t)set * n_proj + j];
            d.W = p->W;
            d.scale = p->scale;
            d.K = p->K;
            d.wpr = p->wpr;
            d.mask_off = moff;
            d.out_off = (int64_t)j * N;
        }
        moff += projs[j]->wpr;
    }
    spike_stream* s = new (std::nothrow) spike_stream;
    if (!s)
        return fail(SPIKE_ENOMEM, "stream allocation failed");
    s->n_proj = n_proj;
    s->n_sets = n_sets;
    s->n_tokens = n_tokens;
    s->N = N;
    s->shape = shape;
    s->max_wpr = max_wpr;
    s->mask_stride = moff;
    s->out_stride = (int64_t)n_proj * N;
    hipError_t e = hipGetDevice(&s->device);
    if (e == hipSuccess)
        e = hipMalloc(&s->d_desc, desc.size() * sizeof(spk::StreamDesc));
    if (e == hipSuccess)
        e = hipMemcpy(s->d_desc, desc.data(), desc.size() * sizeof(spk::StreamDesc), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        if (s->d_desc)
            (void)hipFree(s->d_desc);
        delete s;
        return hip_fail(e, "stream descriptor upload");
    }
    *out_stream = s;
    return SPIKE_OK;
}

int spike_stream_forward(spike_stream_t s, const uint64_t* masks, float* out, void* stream)
{
    g_last_error.clear();
    if (!s)
        return fail(SPIKE_EINVAL, "null stream handle");
    if (!masks || !out)
        return fail(SPIKE_EINVAL, "null mask or output pointer");
    if (int rc = check_device(s->device))
        return rc;
    const int tile = shape_tile(s->shape);
    const int n_tiles = (s->N + tile - 1) / tile;
    const unsigned units = (unsigned)((int64_t)s->n_tokens * s->n_proj * n_tiles);
    hipStream_t st = static_cast<hipStream_t>(stream);
    switch (s->shape) {
    case SHAPE_V16_LG32: launch_stream_t<16, 32>(s, n_tiles, units, masks, out, st); break;
    case SHAPE_V8_LG64: launch_stream_t<8, 64>(s, n_tiles, units, masks, out, st); break;
    case SHAPE_V4_LG64: launch_stream_t<4, 64>(s, n_tiles, units, masks, out, st); break;
    default: launch_stream_t<1, 64>(s, n_tiles, units, masks, out, st); break;
    }
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
    if (s->d_desc)
        (void)hipFree(s->d_desc);
    delete s;
    return rc;
}

const char* spike_proj_last_error(void) { return g_last_error.c_str(); }

int spike_proj_abi_version(void) { return SPIKE_PROJ_ABI_VERSION; }

}  // extern "C"
