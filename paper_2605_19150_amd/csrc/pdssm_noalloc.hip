// pdssm_noalloc.hip -- the forward scan for callers that cannot allocate
// (code under HIP graph capture, tight serving loops): the same kernels as
// pdssm_scan_fwd, with the workspace in a device array of the library.
#include <hip/hip_runtime.h>

#include <mutex>

#include "pdssm.h"

namespace {

// The workspace of every pdssm_scan_fwd_noalloc call on a device: the
// dictionary tables and the segment aggregates.  Each GPU the library runs
// on holds one copy until the process ends.
constexpr size_t kScratchBytes = (size_t)PDSSM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of each device's copy, taken once per device with that
// device current (the array's host-side name is no device address).
constexpr int kMaxDevices = 64;
void* g_scratch[kMaxDevices];
hipError_t g_status[kMaxDevices];
std::once_flag g_once[kMaxDevices];

void* scratch_on(int dev) {
    std::call_once(g_once[dev], [dev] {
        void* p = nullptr;
        g_status[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_scratch[dev] = g_status[dev] == hipSuccess ? p : nullptr;
    });
    return g_scratch[dev];
}

}  // namespace

extern "C" int pdssm_scan_fwd_noalloc(const pdssm_desc* desc, const int32_t* idx, const int32_t* pi,
                                      const pdssm_c64* D, const pdssm_c64* b, const pdssm_c64* c,
                                      const pdssm_c64* h0, float* y, pdssm_c64* h_final, pdssm_c64* saved,
                                      int* dev_status, void* stream) {
    const int C = pdssm_num_chunks(desc);
    if (C < 0) return C;
    // the tables of another call may sit in the array: always rebuild them
    if (desc->flags & PDSSM_FLAG_PREPARED) return PDSSM_ERR_INVALID_ARG;
    const size_t need = pdssm_workspace_size(desc, PDSSM_OP_FWD);
    if (need > kScratchBytes) return PDSSM_ERR_WORKSPACE;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PDSSM_ERR_HIP;
    void* ws = scratch_on(dev);
    if (!ws) return PDSSM_ERR_HIP;
    return pdssm_scan_fwd(desc, idx, pi, D, b, c, h0, y, h_final, saved, ws, kScratchBytes, dev_status, stream);
}
