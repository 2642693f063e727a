// Decode attention for callers that cannot allocate device memory (code under
// HIP graph capture, serving loops that forbid allocation): the split partials
// and the row page prefix live in a file-scope device array instead of a
// caller's workspace.  Each GPU the library runs on holds its own copy of the
// array until the process ends.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is taken once per device with hipGetSymbolAddress (at pool
// creation, with the pool's device current) and only that address is handed to
// kernels.

#include "hotcold_kv.h"
#include "kernels.h"

#include <mutex>

namespace {

constexpr size_t kScratchBytes = size_t(KV_DECODE_SCRATCH_BYTES);
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch`, per device

}  // namespace

namespace hck {

hipError_t scratch_address(int device, void** out) {
    *out = nullptr;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch[device] = p;
    }
    *out = g_scratch[device];
    return hipSuccess;
}

}  // namespace hck

extern "C" int paged_decode_attention_noalloc(kv_pool* pool, int32_t layer, const void* q,
                                              const int32_t* page_table, int64_t pt_stride,
                                              const int32_t* seq_lens, int32_t batch, int32_t num_q_heads,
                                              float scale, void* out, kv_stream_t stream) {
    void* ws = nullptr;
    const int rc = hck::pool_scratch(pool, &ws);
    if (rc != KV_OK) return rc;
    return hck::decode_impl(pool, layer, q, page_table, pt_stride, seq_lens, batch, num_q_heads, scale, out,
                            ws, kScratchBytes, stream, /*no_alloc=*/true);
}
