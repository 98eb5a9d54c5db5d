// The log-likelihood evaluation on a workspace that the library holds itself,
// for callers that cannot allocate device memory (code under HIP graph
// capture, serving loops, harnesses that forbid hipMalloc).
//
// `scratch` is a file-scope device array: every GPU the library runs on holds
// its own copy, at its own address, from the time the code object is loaded
// until the process ends. In host code the array's name is only a stand-in, so
// the first call on each device looks up that device's address with
// hipGetSymbolAddress and keeps it; kernels only ever receive that address.
// Every call on a device shares the device's array: calls that overlap on one
// device (other streams, other threads) race on it and must be serialised by
// the caller. Nothing in it needs to start at zero: the sampling and
// evaluation kernels write every word they later read.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>

#include "w2v_internal.h"

static constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace w2v {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The calling thread's current device's address of `scratch` (looked up once per device).
int scratch_address(void **ptr) {
    int d = 0;
    W2V_HIP(hipGetDevice(&d));
    if (d < 0 || d >= kMaxDevices) return fail(W2V_E_DEVICE, "device index out of range");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[d]) {
        void *p = nullptr;
        W2V_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
        if (!p) return fail(W2V_E_DEVICE, "hipGetSymbolAddress returned no address for the scratch array");
        g_scratch_ptr[d] = p;
    }
    *ptr = g_scratch_ptr[d];
    return W2V_OK;
}

}  // namespace
}  // namespace w2v

using namespace w2v;

extern "C" {

size_t w2v_noalloc_scratch_bytes(void) { return kScratchBytes; }

int w2v_hs_loglik_noalloc(const w2v_model *m, const int32_t *tokens, int64_t n_tokens, const w2v_params *p,
                          double *sum_ll_host, int64_t *n_pairs_host, int64_t *n_nodes_host, void *hip_stream) {
    set_error("");
    if (int rc = check_loglik_args(m, tokens, n_tokens, p, sum_ll_host, n_pairs_host)) return rc;
    const size_t need = w2v_hs_loglik_workspace_bytes(m, n_tokens, p);
    if (need > kScratchBytes)
        return fail(W2V_E_RANGE, "this evaluation needs " + std::to_string(need) + " bytes of workspace; the static "
                                 "scratch holds " + std::to_string(kScratchBytes) + " (use w2v_hs_loglik)");
    void *ws = nullptr;
    if (int rc = scratch_address(&ws)) return rc;
    return loglik_run(m, tokens, n_tokens, p, sum_ll_host, n_pairs_host, n_nodes_host, ws,
                      static_cast<hipStream_t>(hip_stream));
}

}  // extern "C"
