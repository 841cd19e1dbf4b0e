// retro_step with its workspace in a static device array instead of a caller's
// buffer: for callers that cannot allocate (code under HIP graph capture, tight
// serving loops, harnesses that forbid allocation).
//
// The array `scratch` lives in the library's code object, one copy per GPU,
// held until the process ends.  Host code never passes the array's name to a
// kernel: its device address comes from hipGetSymbolAddress, once per device
// (with that device current), and is kept per device.  Every call on a GPU
// shares its array, which keeps the last call's contents; the step's protocol
// needs the workspace zero-filled once per geometry, so a call whose dims
// differ from the previous call's on that device first clears the part it
// uses with a fill kernel on the call's stream (not while the stream is being
// captured: a replayed clear would reset the launch epochs and let words of an
// earlier replay pass for current ones, so such a call is refused).  Calls that
// overlap on one GPU (other streams, other host threads) race on the array.
#include <mutex>

#include "internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct DeviceScratch {
  void* ptr = nullptr;   // the device address of `scratch` on this device
  bool used = false;     // a call ran here: `last` holds its dims
  retro_dims last{};
};
DeviceScratch g_dev[kMaxDevices];
std::mutex g_mutex;

__global__ void __launch_bounds__(256) clear_kernel(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16;
       i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// dims that give the same workspace layout and geometry (flags aside)
bool same_geometry(const retro_dims& a, const retro_dims& b) {
  return a.batch == b.batch && a.num_kv_heads == b.num_kv_heads && a.group == b.group &&
         a.head_dim == b.head_dim && a.page_size == b.page_size &&
         a.budget_tokens == b.budget_tokens && a.window == b.window &&
         a.max_pages == b.max_pages && a.num_phys_pages == b.num_phys_pages &&
         a.dtype == b.dtype && a.sm_scale == b.sm_scale && a.budget_permille == b.budget_permille;
}

}  // namespace

extern "C" retro_status retro_step_noalloc(const retro_dims* dims, int32_t step,
                                           const void* q_window, const void* k_new,
                                           const void* v_new, const retro_kv_cache* cache,
                                           const retro_selection* sel,
                                           const retro_output_cache* ocache, float* o_out,
                                           float* lse_out, void* stream) {
  if (!dims) return RETRO_EINVAL;
  size_t need = 0;
  retro_status st = retro_workspace_size(dims, &need);
  if (st != RETRO_OK) return st;
  if (need > kScratchBytes) return RETRO_ESCRATCH;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return RETRO_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return RETRO_EUNSUPPORTED;
  hipStream_t s = (hipStream_t)stream;
  void* ptr = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceScratch& d = g_dev[dev];
    if (!d.ptr) {  // first call on this device (it is current)
      void* p = nullptr;
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return RETRO_EHIP;
      d.ptr = p;
    }
    if (!d.used || !same_geometry(d.last, *dims)) {
      hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
      if (hipStreamIsCapturing(s, &cap) != hipSuccess) return RETRO_EHIP;
      if (cap != hipStreamCaptureStatusNone) return RETRO_ESCRATCH;
      const size_t n16 = (need + 15) / 16;
      const unsigned blocks = (unsigned)std::min<size_t>((n16 + 255) / 256, 4096);
      clear_kernel<<<blocks, 256, 0, s>>>(reinterpret_cast<uint4*>(d.ptr), n16);
      if (hipGetLastError() != hipSuccess) return RETRO_EHIP;
      d.last = *dims;
      d.used = true;
    }
    ptr = d.ptr;
  }
  return retro_step(dims, step, q_window, k_new, v_new, cache, sel, ocache, o_out, lse_out, ptr,
                    kScratchBytes, stream);
}
