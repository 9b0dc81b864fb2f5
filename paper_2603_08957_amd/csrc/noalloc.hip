// tre_execute_noalloc: tre_execute with its workspace in a static device
// array instead of a caller-supplied buffer, for callers that cannot
// allocate device memory (code under stream capture, tight serving loops,
// harnesses that forbid allocation).
//
// The array lives in this module's device data: every GPU the library runs
// on holds its own copy, at its own address, from module load to process
// end.  Host code never passes the array's name to a kernel -- on the host
// that name is a stand-in, not a device address -- but the address
// hipGetSymbolAddress returns for the current device, looked up once per
// device on the first call there and kept.  Calls on one GPU share its
// array: each call clears what it needs zeroed (the header, the pacing
// counters) with fill kernels, and calls that overlap on one GPU (several
// streams or threads) race on it and must be serialised by the caller.
#include <mutex>

#include "tre_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t(256) << 20;  // the documented maximum workspace
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of `scratch` on the current device (nullptr on failure,
// with the error recorded).
void* scratch_ptr() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        tre::set_error(std::string("tre_execute_noalloc: no usable current device: ") + hipGetErrorString(e));
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            tre::set_error(std::string("tre_execute_noalloc: hipGetSymbolAddress: ") + hipGetErrorString(e));
            return nullptr;
        }
        g_ptr[dev] = p;
    }
    return g_ptr[dev];
}

}  // namespace

extern "C" {

size_t tre_noalloc_scratch_bytes(void) { return kScratchBytes; }

tre_status tre_execute_noalloc(tre_plan_t plan, const int32_t* u_keys, int64_t n_u, const void* u_tiles,
                               const int32_t* v_keys, int64_t n_v, const void* v_tiles, int32_t* w_keys,
                               void* w_tiles, int64_t w_cap, int64_t* n_w, int32_t* pairs_out, int64_t pair_cap,
                               int64_t* n_pairs, void* stream) {
    if (n_w) *n_w = 0;
    if (n_pairs) *n_pairs = 0;
    if (!plan || n_u < 0 || n_v < 0) {
        tre::set_error("tre_execute_noalloc: null plan or negative size");
        return TRE_E_ARG;
    }
    // the inputs' fixed part of the workspace (no pairs yet) must fit
    if (tre_workspace_max_pairs(plan, n_u, n_v, kScratchBytes) < 0) {
        tre::set_error("tre_execute_noalloc: inputs need more workspace than the " +
                       std::to_string(kScratchBytes >> 20) + " MiB static scratch array");
        return TRE_E_WORKSPACE;
    }
    void* ws = scratch_ptr();
    if (!ws) return TRE_E_DEVICE;
    const tre_status st = tre_execute(plan, u_keys, n_u, u_tiles, v_keys, n_v, v_tiles, w_keys, w_tiles, w_cap, n_w,
                                      pairs_out, pair_cap, n_pairs, ws, kScratchBytes, stream, nullptr);
    if (st == TRE_E_WORKSPACE)
        tre::set_error("tre_execute_noalloc: the matched pairs (n_pairs) need more workspace than the " +
                       std::to_string(kScratchBytes >> 20) + " MiB static scratch array holds");
    return st;
}

}  // extern "C"
