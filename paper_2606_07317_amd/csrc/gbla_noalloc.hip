// gbla_noalloc.hip -- gbla_forward_noalloc: gbla_forward for callers that
// cannot allocate device memory (code under graph capture, tight serving
// loops, harnesses that forbid allocation).  Its scratch is a file-scope
// device array instead of a caller's workspace; everything else -- the
// checks, the kernels, the results -- is gbla_forward's.
#include <hip/hip_runtime.h>

#include <mutex>

#include "gbla.h"
#include "gbla_plan.h"

namespace {

// Each GPU that the library runs on holds its own copy of this array until
// the process ends.  In host code `scratch` only names the symbol: its
// device address is looked up per device with hipGetSymbolAddress.
constexpr size_t kScratchBytes = size_t(16) << 20;
static_assert(kScratchBytes == GBLA_NOALLOC_SCRATCH_BYTES, "the header's figure");
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::once_flag g_once[kMaxDevices];
void* g_scratch[kMaxDevices];
hipError_t g_lookup[kMaxDevices];

// The address of `scratch` on `device`, looked up once with that device
// current (the caller's current device is restored afterwards).
gbla_status scratch_of(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices) return GBLA_ERR_UNSUPPORTED;
  std::call_once(g_once[device], [device] {
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e == hipSuccess && prev != device) e = hipSetDevice(device);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (prev >= 0 && prev != device) {
      const hipError_t r = hipSetDevice(prev);
      if (e == hipSuccess) e = r;
    }
    g_lookup[device] = e;
    g_scratch[device] = e == hipSuccess ? p : nullptr;
  });
  if (g_lookup[device] != hipSuccess || !g_scratch[device]) return GBLA_ERR_HIP;
  *ptr = g_scratch[device];
  return GBLA_OK;
}

}  // namespace

extern "C" gbla_status gbla_forward_noalloc(const gbla_shape* shape, const void* q, const void* k,
                                            const void* v, const void* gate_logits,
                                            const void* out_gate, const float* conv_w,
                                            const float* norm_w, const int32_t* cu_seqlens,
                                            float* out, void* stream) {
  // Shapes whose scratch exceeds the array are refused before any HIP call.
  gbla::Plan p;
  const gbla_status planned = gbla::make_plan(shape, cu_seqlens != nullptr, &p);
  if (planned != GBLA_OK) return planned;
  if (p.total_bytes > kScratchBytes) return GBLA_ERR_WORKSPACE;
  int device = -1;
  if (hipStreamGetDevice(static_cast<hipStream_t>(stream), &device) != hipSuccess)
    return GBLA_ERR_HIP;
  void* ws = nullptr;
  const gbla_status found = scratch_of(device, &ws);
  if (found != GBLA_OK) return found;
  return gbla::forward_entry(shape, q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens,
                             ws, kScratchBytes, out, stream, {});
}
