// ckv_noalloc.hip -- ckv_compress_layer for callers that cannot allocate.
//
// The workspace is a file-scope device array instead of a caller buffer. Every
// GPU the library runs on holds its own copy (allocated when this code object
// is first loaded on that GPU, kept until the process ends), so its device
// address is looked up per GPU, with that GPU current, on the entry point's
// first call there. The host-side name `scratch` is only a handle for that
// lookup: its address is never passed to a kernel or a copy.
//
// The kernels behind ckv_compress_layer clear the selection control words and
// histograms they use at the start of every call, so the previous call's
// contents are harmless; calls that overlap on one GPU share the array and
// race (see the header).
#include <hip/hip_runtime.h>

#include <mutex>

#include "ckv.h"
#include "ckv_internal.h"

static __device__ __align__(256) unsigned char scratch[CKV_NOALLOC_MAX_WORKSPACE_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];  // scratch's device address on each GPU, once looked up

// This GPU's scratch address in *p, looked up on the first call (dev current).
hipError_t scratch_ptr(int dev, void** p) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* q = nullptr;
    const hipError_t e = hipGetSymbolAddress(&q, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!q) return hipErrorInvalidSymbol;
    g_ptr[dev] = q;
  }
  *p = g_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" int ckv_compress_layer_noalloc(const ckv_layer_desc* desc, const uint8_t* head_mask,
                                          const ckv_seq* seqs, int32_t num_seqs, void* stream) {
  const size_t need = ckv_workspace_bytes(desc, seqs, num_seqs);
  // invalid descriptors and prompt lists get ckv_compress_layer's own status
  if (need == 0) return ckv_compress_layer(desc, head_mask, seqs, num_seqs, nullptr, 0, stream);
  if (need > CKV_NOALLOC_MAX_WORKSPACE_BYTES) return CKV_ERR_WORKSPACE;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess && stream) {
    int sdev = 0;
    e = hipStreamGetDevice((hipStream_t)stream, &sdev);
    if (e == hipSuccess && sdev != dev) return CKV_ERR_INVALID_ARG;
  }
  if (e != hipSuccess) return ckv::record_hip_error((int)e);
  if (dev < 0 || dev >= kMaxDevices) return CKV_ERR_UNSUPPORTED;
  void* ws = nullptr;
  if ((e = scratch_ptr(dev, &ws)) != hipSuccess) return ckv::record_hip_error((int)e);
  return ckv_compress_layer(desc, head_mask, seqs, num_seqs, ws, CKV_NOALLOC_MAX_WORKSPACE_BYTES,
                            stream);
}
