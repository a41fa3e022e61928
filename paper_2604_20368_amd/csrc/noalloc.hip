// noalloc.hip -- lapattn_forward_noalloc: the forward pass with its workspace in a static device
// array of the library instead of caller memory, for callers that cannot allocate device memory.
//
// `scratch` is a file-scope __device__ array: every GPU the library runs on holds its own copy
// (kScratchBytes) from the loading of the code object until the process ends.  Host code never
// uses the name as an address (on the host it is only a stand-in for the symbol): the device
// address of each GPU's copy is looked up once per device, with that device current, by
// hipGetSymbolAddress, and kept per device.  The entry point then runs lapattn_forward on that
// address, so it shares every kernel and every check of the forward and allocates nothing.
//
// The forward overwrites every workspace slice it reads (the reused-workspace tests hold it to
// that), so nothing in the array needs clearing between calls.  All calls on one GPU share the
// array: calls that overlap on one GPU (different streams, or different host threads without
// ordering) race on it and must be serialised by the caller.
#include <hip/hip_runtime.h>

#include <mutex>

#include "lapattn.h"

static constexpr size_t kScratchBytes = size_t(32) << 20;   // 32 MiB per GPU

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];   // per device: the device address of its `scratch`

// The current device's copy of `scratch`: looked up on the first call on each device.
int scratch_of_current_device(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return LAPATTN_ERR_HIP;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return LAPATTN_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return LAPATTN_OK;
}

}  // namespace

extern "C" {

int lapattn_forward_noalloc(const void* Q, const void* K, const void* V, void* Out, int B, int H, int n, int d,
                            int m, float lambda, int ns_iters, int dtype, const lapattn_opts* opts,
                            lapattn_stream_t stream) {
    try {
        if (opts && opts->save) return LAPATTN_ERR_PARAM;   // the saved state would live in the shared array
        // Every argument check of the forward, with no workspace given: a valid call reports only
        // the missing workspace, and nothing is enqueued either way.
        const int rc = lapattn_forward(Q, K, V, Out, B, H, n, d, m, lambda, ns_iters, dtype, opts, nullptr, 0,
                                       stream);
        if (rc != LAPATTN_ERR_WORKSPACE) return rc;
        const int flags = (opts && opts->dwc_k) ? LAPATTN_WS_DWC : 0;
        const size_t need = lapattn_workspace_size(B, H, n, d, m, ns_iters, dtype, flags);
        if (need == 0) return LAPATTN_ERR_SHAPE;
        if (need > kScratchBytes) return LAPATTN_ERR_SCRATCH;
        void* ws = nullptr;
        const int sr = scratch_of_current_device(&ws);
        if (sr != LAPATTN_OK) return sr;
        return lapattn_forward(Q, K, V, Out, B, H, n, d, m, lambda, ns_iters, dtype, opts, ws, kScratchBytes,
                               stream);
    } catch (...) {
        return LAPATTN_ERR_HIP;
    }
}

}  // extern "C"
