// The box backward for callers that cannot allocate device memory (code under
// graph capture, tight serving loops, harnesses that forbid allocation): the
// workspace of box_conv_bwd -- the boxes' tap records, the per-wave partial
// edge gradients and, for maps whose table does not fit in LDS, the upstream
// gradient's tables -- lives in a fixed device array owned by the library.
#include <mutex>

#include "../../include/boxconv.h"
#include "bc_internal.hpp"

namespace {

// The library's scratch array: one copy per GPU, held until the process ends.
constexpr size_t kScratchBytes = BC_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each GPU, looked up once per device (with
// that device current) by hipGetSymbolAddress: in host code the array's name
// is a host-side stand-in, never a device address.
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};

bc_status scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return BC_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return BC_ERR_HIP;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return BC_OK;
}

}  // namespace

extern "C" {

size_t bc_noalloc_scratch_bytes(void) { return kScratchBytes; }

bc_status box_conv_bwd_noalloc(const float* x, const float* boxes, const float* grad_y, int N, int C, int H, int W,
                               int B, float* grad_x, float* grad_boxes, unsigned flags, hipStream_t stream) {
  // the workspace box_conv_bwd needs for this request; 0 means the sizes
  // themselves are invalid, which box_conv_bwd reports below
  const size_t need = bc_box_workspace_bytes(1, N, C, H, W, B, flags);
  if (need > kScratchBytes) return BC_ERR_WORKSPACE;
  if (!x || !boxes || !grad_y) return BC_ERR_NULL;
  void* ws = nullptr;
  if (need > 0 && (grad_x || grad_boxes)) {
    const bc_status st = scratch_ptr(&ws);
    if (st != BC_OK) return st;
  }
  // every word of the workspace that the backward reads it writes first in
  // the same call (tap records, partial sums, tables), so nothing is cleared
  return box_conv_bwd(x, boxes, grad_y, N, C, H, W, B, grad_x, grad_boxes, flags, ws, ws ? kScratchBytes : 0,
                      stream);
}

}  // extern "C"
