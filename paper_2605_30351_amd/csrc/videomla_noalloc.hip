// videomla_attend_noalloc: videomla_attend for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc). The
// attention workspace is a static device array of this file, `scratch`, of kScratchBytes: every
// device the library runs on holds its own copy from the code object's load until the process
// ends. Its device address is looked up once per device with hipGetSymbolAddress, with that
// device current, and kept in g_scratch_ptr; host code passes only that address, never the
// array's own name (which in host code is a host-side stand-in, not a device address).
#include <hip/hip_runtime.h>

#include <mutex>

#include "videomla.h"
#include "vmla_internal.h"

namespace {

constexpr size_t kScratchBytes = VIDEOMLA_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once looked up

// The current device's copy of the scratch array (looked up on its first use on that device).
int current_scratch(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess)
    return vmla::report_error(VIDEOMLA_EHIP, "hipGetDevice failed: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return vmla::report_error(VIDEOMLA_EUNSUPPORTED, "device %d beyond the %d the library tracks",
                              dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return vmla::report_error(VIDEOMLA_EHIP, "hipGetSymbolAddress(scratch) failed: %s",
                                hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return VIDEOMLA_OK;
}

}  // namespace

extern "C" {

int videomla_attend_noalloc(const videomla_dims* dims, const videomla_window* win, int32_t batch,
                            const uint16_t* q_nope, const uint16_t* q_r, const uint16_t* w_uk,
                            const uint16_t* w_uv, const uint16_t* c_kv, const uint16_t* k_r,
                            uint16_t* out, void* stream) {
  const size_t need = videomla_attend_workspace_bytes(dims, batch);
  if (need == 0)  // invalid or unsupported arguments: videomla_attend reports which
    return videomla_attend(dims, win, batch, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, nullptr,
                           0, stream);
  if (need > kScratchBytes)
    return vmla::report_error(VIDEOMLA_EWORKSPACE,
                              "this shape needs %zu bytes of workspace; the static scratch of "
                              "videomla_attend_noalloc holds %zu (use videomla_attend)",
                              need, kScratchBytes);
  void* ws = nullptr;
  if (int e = current_scratch(&ws)) return e;
  return videomla_attend(dims, win, batch, q_nope, q_r, w_uk, w_uv, c_kv, k_r, out, ws,
                         kScratchBytes, stream);
}

}  // extern "C"
