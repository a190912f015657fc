// k_gate_noalloc.hip -- mg_margin_gate_noalloc: the margin gate for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  It runs the same two top-2 kernels as mg_margin_gate, with their
// per-slice partial states kept in a file-scope device array instead of a context's
// workspace, so it needs no context and no allocation.
#include <mutex>

#include "../../include/mg.h"
#include "mg_kernels.h"

namespace {

// Largest partial-state buffer a gate launch uses: the slice count times the rows never
// exceeds 2048 states of 16 bytes (top2_ws_bytes).
constexpr size_t GATE_SCRATCH_BYTES = 2048 * 16;
constexpr int MAX_DEVICES = 64;

// One copy per GPU the library runs on, held until the process ends.  In host code this
// name is only a stand-in for the device symbol: kernels get the address looked up below.
static __device__ __align__(256) unsigned char scratch[GATE_SCRATCH_BYTES];

std::mutex g_mu;
void* g_scratch_ptr[MAX_DEVICES];

// The device address of `scratch` on the current device, looked up once per device (with
// that device current) and kept.
hipError_t scratch_on_current_device(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return hipSuccess;
}

}  // namespace

extern "C" mg_status mg_margin_gate_noalloc(int B, int V, const float* logits, const uint8_t* protected_mask,
                                            float tau, int32_t* top1, float* margin, uint8_t* gate,
                                            int32_t* gated_rows, int32_t* n_gated, void* stream) {
    if (!logits || !top1 || !margin || !gate || !gated_rows || !n_gated) return MG_ERR_ARG;
    if (B < 0 || B > 256 || V < 2) return MG_ERR_ARG;
    if (B == 0) return MG_OK;
    if (mg::top2_ws_bytes(B, V) > GATE_SCRATCH_BYTES) return MG_ERR_WORKSPACE;
    void* ws = nullptr;
    if (scratch_on_current_device(&ws) != hipSuccess) return MG_ERR_HIP;
    // every partial state the second kernel reads is written by the first one in the same
    // call, so the array needs no clearing between calls
    if (mg::launch_top2(B, V, logits, protected_mask, tau, top1, margin, gate, gated_rows, n_gated, nullptr, ws,
                        nullptr, static_cast<hipStream_t>(stream)) != hipSuccess)
        return MG_ERR_HIP;
    return MG_OK;
}
