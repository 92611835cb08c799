// rmm_linear_noalloc: rmm_linear with its workspace in a fixed device array
// of this library, for callers that cannot allocate device memory (code
// under HIP graph capture, serving loops that forbid allocation).
//
// The array below is one per GPU: every device this library runs on holds
// its own copy at its own address, from the first call on that device until
// the process ends.  In host code its name is only a stand-in for the
// device symbol, never a device address, so host code uses the address that
// hipGetSymbolAddress returns for the current device and nothing else.
#include <mutex>

#include <hip/hip_runtime.h>

#include "../../include/rmm.h"

namespace {

constexpr size_t kScratchBytes = size_t(64) << 20;      // RMM_NOALLOC_SCRATCH_BYTES
constexpr int kMaxDevices = 64;

static __device__ __attribute__((aligned(256))) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];          // device address per device id, or null

// The scratch address on the current device, looked up once per device
// (with that device current) and kept for the rest of the process.
rmm_status_t scratch_on_current_device(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return RMM_ERR_HIP;
    if (dev < 0 || dev >= kMaxDevices) return RMM_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return RMM_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return RMM_OK;
}

}  // namespace

extern "C" {

size_t rmm_noalloc_scratch_bytes(void) { return kScratchBytes; }

rmm_status_t rmm_linear_noalloc(const void *X, const void *W, double r, rmm_dtype_t dtype,
                                int64_t B, int64_t M, int64_t N, int64_t K, int64_t ldx,
                                int64_t ldw, void *Y, int64_t ldy, int32_t *idx_out,
                                hipStream_t stream) {
    // argument errors first, exactly as rmm_linear reports them
    const int64_t k = rmm_retained_count(r, K);
    if (k < 0) return RMM_ERR_INVALID_ARGUMENT;
    if (!X || !W || !Y) return RMM_ERR_INVALID_ARGUMENT;
    if (dtype != RMM_F32 && dtype != RMM_BF16) return RMM_ERR_INVALID_ARGUMENT;
    if (B < 1 || M < 1 || N < 1 || ldx < K || ldw < N || ldy < N) return RMM_ERR_INVALID_ARGUMENT;
    const size_t need = rmm_workspace_size(RMM_OP_LINEAR, B, M, K, k);
    if (need == 0 || need > kScratchBytes) return RMM_ERR_TOO_LARGE;
    // the scratch of the device the stream runs on
    if (stream != nullptr) {
        int sdev = -1, cur = -1;
        if (hipStreamGetDevice(stream, &sdev) != hipSuccess || hipGetDevice(&cur) != hipSuccess)
            return RMM_ERR_HIP;
        if (sdev != cur) return RMM_ERR_INVALID_ARGUMENT;
    }
    void *ws = nullptr;
    const rmm_status_t st = scratch_on_current_device(&ws);
    if (st != RMM_OK) return st;
    return rmm_linear(X, W, r, dtype, B, M, N, K, ldx, ldw, Y, ldy, idx_out, ws, kScratchBytes,
                      stream);
}

}  // extern "C"
