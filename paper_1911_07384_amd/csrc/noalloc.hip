// The weight gradient for callers that cannot allocate device memory (code
// under HIP graph capture, serving loops, harnesses that forbid hipMalloc):
// fp16_conv_wgrad with its workspace -- the float32 split-K partial sums and,
// for the stem, the space-to-depth staging of the image -- in a fixed,
// library-owned device array instead of a caller's buffer.
//
// The array is a file-scope __device__ variable: every GPU the library runs
// on holds its own copy, at its own address, from the first use on that GPU
// until the process ends.  Host code never passes the variable's name to a
// kernel (on the host it names a stand-in, not device memory); it asks the
// runtime once per device for the device address and passes that.  Nothing
// in the array has to start at zero: every partial sum the reduction reads is
// written earlier in the same call.  Calls that overlap in time on one GPU
// (two streams, two host threads) share the array and race.

#include "../../include/fp16train.h"

#include <hip/hip_runtime.h>

#include <mutex>

namespace {

constexpr size_t kScratchBytes = (size_t)32 << 20;  // FP16_NOALLOC_SCRATCH_BYTES
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

// Device address of this GPU's array; looked up once per device, with that
// device current.
fp16_status scratch_ptr(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return FP16_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return FP16_ERR_HIP;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return FP16_ERR_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return FP16_ERR_HIP;
    if (e != hipSuccess || !p) return FP16_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return FP16_OK;
}

}  // namespace

extern "C" {

size_t fp16_noalloc_scratch_bytes(void) { return kScratchBytes; }

fp16_status fp16_conv_wgrad_noalloc(const fp16_conv_desc* desc, const fp16_t* x,
                                    const fp16_t* dy, fp16_t* dw, fp16_stream_t stream) {
  int32_t p = 0, q = 0;
  const fp16_status sd = fp16_conv_out_dims(desc, &p, &q);  // validates the descriptor
  if (sd != FP16_OK) return sd;
  if (fp16_conv_workspace_bytes(desc, FP16_PASS_WGRAD) > kScratchBytes) return FP16_ERR_WORKSPACE;
  if (!x || !dy || !dw) return FP16_ERR_NULL;
  int dev = -1;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (st) {
    if (hipStreamGetDevice(st, &dev) != hipSuccess) return FP16_ERR_HIP;
  } else if (hipGetDevice(&dev) != hipSuccess) {
    return FP16_ERR_HIP;
  }
  void* ws = nullptr;
  const fp16_status s = scratch_ptr(dev, &ws);
  if (s != FP16_OK) return s;
  return fp16_conv_wgrad(desc, x, dy, dw, ws, kScratchBytes, stream);
}

}  // extern "C"
