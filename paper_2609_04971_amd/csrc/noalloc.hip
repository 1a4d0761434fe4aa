// bkv_evict_noalloc: the whole eviction of one layer (bkv_evict_ex) with
// its workspace in a fixed device array of this library instead of a
// caller-allocated buffer, for callers that cannot allocate device memory
// (code under HIP graph capture, serving loops, harnesses that forbid it).
//
// The array is a file-scope __device__ variable.  In host code its name is
// only a host-side stand-in, so its device address is looked up once per
// device with hipGetSymbolAddress (with that device current) and only that
// address is ever passed to kernels.  Each GPU holds its own copy until the
// process ends; every call on a GPU reuses it, so calls on one GPU that
// overlap in time race (order them on one stream).
#include <mutex>

#include "bkv.h"
#include "internal.h"

namespace bkv {
namespace {

constexpr size_t kScratchBytes = BKV_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices];  // device address of `scratch` per device, once looked up

// Device address of this device's scratch array; nullptr on failure.
void* scratch_ptr(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_ptr[dev] = p;
    }
    return g_ptr[dev];
}

// Copy the workspace's sticky device-error word to the caller's status word.
__global__ void report_error_kernel(const int* hdr, int32_t* out) {
    if (threadIdx.x == 0) *out = hdr[kHdrErr] ? (int32_t)BKV_ERR_DEVICE : (int32_t)BKV_OK;
}

}  // namespace
}  // namespace bkv

extern "C" bkv_status bkv_evict_noalloc(const bkv_dims* d, int32_t flags, void* K, void* V, const void* q_win,
                                        const float* beacons, const int32_t* counts, const float* rope_cos,
                                        const float* rope_sin, float scale, int32_t* kept, float* scores,
                                        float* row_lse, int32_t* device_status, hipStream_t stream) {
    using namespace bkv;
    bkv_status st = evict_check(d, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale);
    if (st != BKV_OK) return st;
    if (bkv_workspace_bytes(d, BKV_OP_EVICT) > kScratchBytes) return BKV_ERR_WORKSPACE;
    if (d->B == 0 || d->N == 0) return BKV_OK;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return BKV_ERR_HIP;
    void* ws = scratch_ptr(dev);
    if (!ws) return BKV_ERR_HIP;
    // the array keeps the previous call's contents: re-stamp and clear its
    // control block first (a fill kernel; graph-capturable)
    st = bkv_workspace_init(d, ws, kScratchBytes, stream);
    if (st != BKV_OK) return st;
    st = evict_enqueue(d, flags, K, V, q_win, beacons, counts, rope_cos, rope_sin, scale, kept, scores, row_lse, ws,
                       stream);
    if (st != BKV_OK || !device_status) return st;
    hipLaunchKernelGGL(report_error_kernel, dim3(1), dim3(64), 0, stream, static_cast<const int*>(ws), device_status);
    return hipGetLastError() == hipSuccess ? BKV_OK : BKV_ERR_HIP;
}
