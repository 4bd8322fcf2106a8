// af_packed_forward_noalloc: the packed step for callers that cannot allocate device memory.
//
// Every device workspace of the step (normalized rows, queries, attention output, the MLP
// activation, split-K partial sums, the step tables, the rotary table) lives in `scratch`, one
// file-scope device array per GPU that the loader reserves with the library's code object and
// that stays until the process ends.  In host code `scratch` names a host-side stand-in; the
// array's device address comes from hipGetSymbolAddress, looked up once per device (with that
// device current) on the first call there, and only that address is handed to kernels and copies.
#include <hip/hip_runtime.h>

#include <mutex>

#include "af_internal.h"

static __device__ __align__(256) unsigned char scratch[AF_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kScratchBytes = (size_t)AF_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

struct DeviceScratch {
  void* ptr = nullptr;  // device address of `scratch` on this device
  af::BufferRope rope;  // rotary table the array holds
};

std::mutex g_mu;
DeviceScratch g_dev[kMaxDevices];

}  // namespace

extern "C" af_status af_packed_forward_noalloc(af_weights* w, const int32_t* token_ids, const void* embeds,
                                               int32_t M, const af_segment* segs, int32_t n_seg, af_ring* ring,
                                               void* out_hidden, float* out_logits, int32_t* out_tokens,
                                               void* hip_stream) {
  af::clear_error();
  int device = -1;
  AF_HIP(hipGetDevice(&device));
  if (device < 0 || device >= kMaxDevices) {
    af::set_error("af_packed_forward_noalloc: device %d outside [0, %d)", device, kMaxDevices);
    return AF_ERR_UNSUPPORTED;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceScratch& ds = g_dev[device];
  if (!ds.ptr) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      af::set_error("af_packed_forward_noalloc: hipGetSymbolAddress of the scratch array failed on device %d: %s",
                    device, hipGetErrorString(e));
      return AF_ERR_DEVICE;
    }
    ds.ptr = p;
  }
  return af::packed_forward_in_buffer(w, token_ids, embeds, M, segs, n_seg, ring, out_hidden, out_logits, out_tokens,
                                      (hipStream_t)hip_stream, ds.ptr, kScratchBytes, &ds.rope);
}
