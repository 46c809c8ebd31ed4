// Allocation-free variant of the bias-gradient operator [baob / baib]:
// the per-block column partial sums, which bias_grad takes from the
// caller's workspace, live in a fixed device array of this library instead.
// For callers that cannot allocate (code under stream capture, tight
// serving loops).  Every call on one GPU uses that GPU's one copy of the
// array, so calls that overlap on a GPU race; the array needs no clearing,
// since the partial kernel writes every partial row before the finish
// kernel reads it.
#include <mutex>

#include "internal.hpp"

namespace {

// 8 MiB: room for the partial rows of up to 2048 columns at any row count
// (at most 512 partial rows), or 4096 columns up to 4096 rows.
constexpr size_t SCRATCH_FLOATS = (size_t)2 << 20;
static __device__ __align__(256) float scratch[SCRATCH_FLOATS];

constexpr int MAX_DEVICES = 64;
std::mutex g_setup_mu;
float* g_scratch[MAX_DEVICES] = {};  // device address of `scratch`, per device

// Device address of this library's scratch array on the current device,
// fetched once per device (the host-side name of the array is not a device
// address).  Returns DM_OK or an error code (message set).
int scratch_on_current_device(float** out) {
    *out = nullptr;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return dm::set_error(DM_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= MAX_DEVICES)
        return dm::set_error(DM_ERR_UNSUPPORTED, "device %d beyond the %d this library tracks", dev, MAX_DEVICES);
    std::lock_guard<std::mutex> lk(g_setup_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return dm::set_error(DM_ERR_DEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch[dev] = static_cast<float*>(p);
    }
    *out = g_scratch[dev];
    return DM_OK;
}

}  // namespace

using namespace dm;

extern "C" {

int bias_grad_noalloc(int32_t dtype, int64_t rows, int32_t cols, const void* x, float* db, void* stream) {
    if (dtype != DM_F32 && dtype != DM_F16 && dtype != DM_BF16)
        return set_error(DM_ERR_UNSUPPORTED, "unsupported dtype %d", dtype);
    if (rows <= 0 || cols <= 0) return set_error(DM_ERR_ARG, "bad shape rows=%lld cols=%d", (long long)rows, cols);
    if (cols % 8) return set_error(DM_ERR_UNSUPPORTED, "row length %d is not a multiple of 8", cols);
    if (cols > 16384) return set_error(DM_ERR_UNSUPPORTED, "row length %d above 16384", cols);
    if (rows > (int64_t)INT32_MAX * 8) return set_error(DM_ERR_UNSUPPORTED, "too many rows");
    if (!x || ((uintptr_t)x & 15u)) return set_error(DM_ERR_ARG, "x is NULL or not 16-byte aligned");
    if (!db || ((uintptr_t)db & 15u)) return set_error(DM_ERR_ARG, "db is NULL or not 16-byte aligned");
    const size_t need = (size_t)colsum_blocks(rows) * (size_t)cols;
    if (need > SCRATCH_FLOATS)
        return set_error(DM_ERR_UNSUPPORTED,
                         "bias_grad_noalloc: %lld rows x %d columns need %zu bytes of partial sums, above the "
                         "fixed %zu-byte scratch (use bias_grad with a workspace)",
                         (long long)rows, cols, need * sizeof(float), SCRATCH_FLOATS * sizeof(float));
    float* part = nullptr;
    if (int rc = scratch_on_current_device(&part)) return rc;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    run_colsum_partial(dtype, rows, cols, x, part, st);
    run_colsum_finish(colsum_blocks(rows), cols, part, db, st);
    return check_launch("bias_grad_noalloc");
}

}  // extern "C"
