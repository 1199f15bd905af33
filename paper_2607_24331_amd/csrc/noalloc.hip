// Decode with no caller workspace, for callers that cannot allocate device
// memory (code under HIP graph capture, tight serving loops, harnesses that
// forbid hipMalloc).  The decode's scratch (folded queries, split partials,
// merged rows) lives in one fixed array in device memory instead of a
// caller-provided workspace; the kernels are those of dckv_decode.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace dckv {
namespace {

// Each GPU the library runs on holds its own copy of this array until the
// process ends.  Host code never uses the name as an address: it takes the
// device address from hipGetSymbolAddress, once per device.
static __device__ __align__(256) unsigned char scratch[DCKV_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up on the first call on
// that device (with that device current).
hipError_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace
}  // namespace dckv

extern "C" int dckv_decode_noalloc(const dckv_plan* p, const float* q, int32_t batch,
                                   const void* pool, int64_t num_pages, const int32_t* page_table,
                                   int32_t max_pages, const int32_t* seq_lens, int32_t max_context,
                                   const void* R_keys, const void* R_value, float* out,
                                   void* stream) {
  dckv::DecodeShape shape;
  int st = dckv::check_decode("decode_noalloc", p, q, batch, pool, num_pages, page_table,
                              max_pages, seq_lens, max_context, R_keys, R_value, out, &shape);
  if (st != DCKV_OK || batch == 0) return st;
  if (shape.bytes > size_t(DCKV_NOALLOC_SCRATCH_BYTES))
    return dckv::fail(DCKV_EWORKSPACE,
                      "decode_noalloc: this call needs %zu bytes of scratch; the fixed device "
                      "array holds %zu (use dckv_decode with a workspace)",
                      shape.bytes, size_t(DCKV_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  hipError_t e = dckv::scratch_address(&ws);
  if (e != hipSuccess)
    return dckv::fail(DCKV_EHIP, "decode_noalloc: scratch address: %s", hipGetErrorString(e));
  e = dckv::launch_decode(*p, shape, q, pool, num_pages, page_table, max_pages, seq_lens, R_keys,
                          R_value, out, ws, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return dckv::fail(DCKV_EHIP, "decode_noalloc: %s", hipGetErrorString(e));
  return DCKV_OK;
}
