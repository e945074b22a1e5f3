// Host side of the dense continuous-input INT8 projection (C ABI in
// include/dense_proj.h): validates arguments, picks the load width, batch
// rows per launch and rows per lane group, and enqueues k_dense on the
// caller's stream.  No allocation and no synchronisation.
#include "dense_proj.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdint>

#include "dense.hpp"
#include "errors.hpp"

static_assert(spk::dense_lds_floats(DENSE_MAX_K, 16, 1, 8) <= spk::kDenseMaxLdsFloats, "one row of the largest K fits");

namespace {

using spk::fail;
using spk::hip_fail;

using DenseFn = void (*)(const int8_t*, const float*, int, int, const float*, int, float*, int);
using RegFn = void (*)(const int8_t*, const float*, int, int, const float*, int, float*);

// Staged-activation kernels: load width V (16, 4, 1) x batch rows BC (1, 2,
// 4, 8).  Ring depth: four 16-byte loads or eight narrower ones per lane.
template <int V>
constexpr int ring_of() { return V == 16 ? 4 : 8; }

template <int V>
DenseFn dense_fn(int bc)
{
    constexpr int U = ring_of<V>();
    switch (bc) {
    case 1: return spk::k_dense<V, 1, U>;
    case 2: return spk::k_dense<V, 2, U>;
    case 4: return spk::k_dense<V, 4, U>;
    default: return spk::k_dense<V, 8, U>;
    }
}

DenseFn pick_fn(int v, int bc)
{
    if (v == 16)
        return dense_fn<16>(bc);
    if (v == 4)
        return dense_fn<4>(bc);
    return dense_fn<1>(bc);
}

// Register kernels: NPL 16-byte chunks per lane and row (K <= 512 NPL).  The
// activations held per lane, 16 NPL BC floats, stay at or below 96; rows in
// flight per lane: U = 8 / NPL rounded, at least 2.
constexpr int kRegMaxNpl = 8;
constexpr int reg_max_bc(int npl) { return npl <= 1 ? 4 : npl <= 3 ? 2 : 1; }
template <int NPL>
constexpr int reg_ring() { return NPL >= 4 ? 2 : 8 / NPL; }

template <int NPL>
RegFn reg_fn_npl(int bc)
{
    constexpr int U = reg_ring<NPL>();
    if constexpr (reg_max_bc(NPL) >= 4)
        if (bc == 4)
            return spk::k_dense_reg<NPL, 4, U>;
    if constexpr (reg_max_bc(NPL) >= 2)
        if (bc == 2)
            return spk::k_dense_reg<NPL, 2, U>;
    return spk::k_dense_reg<NPL, 1, U>;
}

RegFn reg_fn(int npl, int bc)
{
    switch (npl) {
    case 1: return reg_fn_npl<1>(bc);
    case 2: return reg_fn_npl<2>(bc);
    case 3: return reg_fn_npl<3>(bc);
    case 4: return reg_fn_npl<4>(bc);
    case 5: return reg_fn_npl<5>(bc);
    case 6: return reg_fn_npl<6>(bc);
    case 7: return reg_fn_npl<7>(bc);
    default: return reg_fn_npl<8>(bc);
    }
}

// Workgroups of a register kernel one CU holds at once (its VGPR use sets
// it), asked of the runtime once per kernel; 2 while the query fails (no
// device), without caching that.
int reg_resident(int npl, int bc)
{
    static std::atomic<int> cache[kRegMaxNpl + 1][5];
    std::atomic<int>& c = cache[std::min(npl, kRegMaxNpl)][std::min(bc, 4)];
    int v = c.load(std::memory_order_relaxed);
    if (v > 0)
        return v;
    int n = 0;
    const RegFn fn = reg_fn(npl, bc);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, reinterpret_cast<const void*>(fn), spk::kRegBlock, 0) !=
            hipSuccess ||
        n < 1) {
        (void)hipGetLastError();
        return 2;
    }
    c.store(n, std::memory_order_relaxed);
    return n;
}

// Process-wide launch-shape overrides (dense_proj_tune); 0 = automatic.
std::atomic<int> g_tune_kernel{0};
std::atomic<int> g_tune_wg_per_cu{0};

struct DensePlan {
    int kernel;    // DENSE_KERNEL_STAGED or DENSE_KERNEL_REGISTER
    int v;         // bytes per weight load
    int bc;        // batch rows per launch
    int npl;       // register kernel: 16-byte chunks per lane and row
    int rpg;       // rows per lane group (register kernel: the most any group takes)
    int64_t wgs;   // workgroups per launch
    size_t lds;    // dynamic LDS bytes
};

constexpr int kCUs = 256;

// q_align: the largest power of two (up to 16) dividing Q's address.  The
// kernel and load width depend on K and q_align only, never on B, so a row's
// summation order is the same in every batch.
DensePlan make_plan(int32_t K, int32_t M, int32_t B, int q_align)
{
    DensePlan p{};
    p.v = (K % 16 == 0 && q_align >= 16) ? 16 : (K % 4 == 0 && q_align >= 4 ? 4 : 1);
    const int npl = (K + 32 * 16 - 1) / (32 * 16);
    const bool reg_ok = p.v == 16 && npl <= kRegMaxNpl;
    const int tk = g_tune_kernel.load();
    p.kernel = (tk == DENSE_KERNEL_STAGED || !reg_ok) ? DENSE_KERNEL_STAGED : DENSE_KERNEL_REGISTER;
    const int wpc = g_tune_wg_per_cu.load();
    if (p.kernel == DENSE_KERNEL_REGISTER) {
        p.npl = npl;
        p.bc = 1;
        while (p.bc < reg_max_bc(npl) && p.bc < B)
            p.bc *= 2;
        // One row per group when the matrix is small; otherwise two
        // workgroups per CU (fewer if the kernel's occupancy allows only one),
        // each group then walking several rows.  Longer walks keep the ring
        // full for longer: measured on the 1536 -> 57344 head, two per CU
        // beat the four that fit by 5%.
        const int64_t groups = (M + 1) / 2 * 2;  // whole waves
        const int64_t cap =
            (int64_t)kCUs * (wpc > 0 ? wpc : std::min(2, reg_resident(npl, p.bc))) * spk::kRegGroups;
        const int64_t g = std::min(groups, cap);
        p.wgs = (g + spk::kRegGroups - 1) / spk::kRegGroups;
        const int64_t gq = p.wgs * spk::kRegGroups;
        p.rpg = (int)((M + gq - 1) / gq);
        p.lds = 0;
        return p;
    }
    // Every launch streams all of Q, so a launch takes as many batch rows as
    // it can: the smallest instantiated count covering B, at most 8, within
    // the LDS budget (which K <= DENSE_MAX_K meets for one row).
    p.bc = 1;
    while (p.bc < 8 && p.bc < B && spk::dense_lds_floats(K, p.v, 2 * p.bc, 8) <= spk::kDenseMaxLdsFloats)
        p.bc *= 2;
    // Rows per lane group: whole ring rounds per group where that still
    // leaves a thousand or more workgroups to spread over the chip.
    const int u = p.v == 16 ? ring_of<16>() : ring_of<4>();
    const int64_t n_chunks = K / p.v;
    const int64_t n_pl = (n_chunks + spk::kDenseLanes - 1) / spk::kDenseLanes;
    const int64_t groups16 = (M + spk::kDenseGroups - 1) / spk::kDenseGroups;
    p.rpg = 1;
    for (int r = 1; r <= 8; ++r) {
        if (r > 1 && (groups16 + r - 1) / r < 1024)
            break;
        if ((r * n_pl) % u == 0) {
            p.rpg = r;
            break;
        }
    }
    p.wgs = (groups16 + p.rpg - 1) / p.rpg;
    p.lds = (size_t)spk::dense_lds_floats(K, p.v, p.bc, p.rpg) * sizeof(float);
    return p;
}

int check_sizes(int32_t K, int32_t M, int32_t B)
{
    if (K < 1 || K > DENSE_MAX_K)
        return fail(SPIKE_EINVAL, "K = %d outside [1, %d]", K, DENSE_MAX_K);
    if (M < 1)
        return fail(SPIKE_EINVAL, "M = %d < 1", M);
    if ((int64_t)M * K > spk::kBufMaxBytes)
        return fail(SPIKE_EUNSUPPORTED, "M * K = %lld bytes exceeds %lld", (long long)M * K,
                    (long long)spk::kBufMaxBytes);
    if (B < 0 || B > DENSE_MAX_B)
        return fail(SPIKE_EINVAL, "B = %d outside [0, %d]", B, DENSE_MAX_B);
    return SPIKE_OK;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

int align_of(const void* p) { return aligned(p, 16) ? 16 : aligned(p, 4) ? 4 : 1; }

}  // namespace

extern "C" {

int dense_proj_plan(int32_t K, int32_t M, int32_t B, int32_t q_align, int32_t* kernel, int32_t* vec,
                    int32_t* rows_per_launch, int32_t* workgroups)
{
    spk::last_error.clear();
    if (int rc = check_sizes(K, M, B))
        return rc;
    if (q_align != 1 && q_align != 2 && q_align != 4 && q_align != 8 && q_align != 16)
        return fail(SPIKE_EINVAL, "q_align = %d is not 1, 2, 4, 8 or 16", q_align);
    const DensePlan p = make_plan(K, M, B, q_align);
    if (kernel)
        *kernel = p.kernel;
    if (vec)
        *vec = p.v;
    if (rows_per_launch)
        *rows_per_launch = p.bc;
    if (workgroups)
        *workgroups = (int32_t)p.wgs;
    return SPIKE_OK;
}

int dense_proj_tune(int32_t key, int32_t value)
{
    spk::last_error.clear();
    switch (key) {
    case DENSE_TUNE_KERNEL:
        if (value != 0 && value != DENSE_KERNEL_STAGED && value != DENSE_KERNEL_REGISTER)
            return fail(SPIKE_EINVAL, "kernel %d is not 0, DENSE_KERNEL_STAGED or DENSE_KERNEL_REGISTER", value);
        g_tune_kernel.store(value);
        return SPIKE_OK;
    case DENSE_TUNE_WG_PER_CU:
        if (value < 0 || value > 64)
            return fail(SPIKE_EINVAL, "workgroups per CU %d outside [0, 64]", value);
        g_tune_wg_per_cu.store(value);
        return SPIKE_OK;
    default:
        return fail(SPIKE_EINVAL, "unknown dense tuning key %d", key);
    }
}

int dense_proj_forward(const int8_t* Q, const float* scale, int32_t K, int32_t M, const float* x, int32_t B,
                       float* y, void* stream)
{
    spk::last_error.clear();
    if (int rc = check_sizes(K, M, B))
        return rc;
    if (B == 0)
        return SPIKE_OK;
    if (!Q || !scale || !x || !y)
        return fail(SPIKE_EINVAL, "null pointer (Q %p, scale %p, x %p, y %p)", (const void*)Q, (const void*)scale,
                    (const void*)x, (const void*)y);
    if (!aligned(scale, 4) || !aligned(x, 4) || !aligned(y, 4))
        return fail(SPIKE_EINVAL, "scale, x and y must be 4-byte aligned");
    const hipStream_t st = static_cast<hipStream_t>(stream);
    for (int32_t b0 = 0; b0 < B;) {
        const DensePlan p = make_plan(K, M, B - b0, align_of(Q));
        const int32_t nb = std::min<int32_t>(p.bc, B - b0);
        const float* xb = x + (int64_t)b0 * K;
        float* yb = y + (int64_t)b0 * M;
        if (p.kernel == DENSE_KERNEL_REGISTER)
            hipLaunchKernelGGL(reg_fn(p.npl, p.bc), dim3((unsigned)p.wgs), dim3(spk::kRegBlock), 0, st, Q, scale, K,
                               M, xb, nb, yb);
        else
            hipLaunchKernelGGL(pick_fn(p.v, p.bc), dim3((unsigned)p.wgs), dim3(spk::kDenseBlock), p.lds, st, Q,
                               scale, K, M, xb, nb, yb, p.rpg);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return hip_fail(e, "dense projection launch");
        b0 += nb;
    }
    return SPIKE_OK;
}

}  // extern "C"
