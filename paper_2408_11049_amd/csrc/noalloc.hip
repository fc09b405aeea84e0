// noalloc.hip -- md_attn_noalloc: md_verify_attn / md_draft_attn with the
// library's own device scratch in place of a caller workspace, for callers
// that cannot allocate (code under graph capture, tight serving loops).
//
// The scratch holds what a split-range call keeps in its workspace: the
// tagged arrival counters and the chunks' partial O and lse.  It is a
// file-scope device array, so every GPU the library runs on holds one copy
// until the process ends.  Host code never passes the array's name to a
// kernel (on the host it is only a stand-in symbol): its device address is
// looked up once per device with hipGetSymbolAddress, with that device
// current, and that address is what the kernels receive.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

#include "internal.h"
#include "kernels.h"
#include "magicdec.h"

namespace md {

namespace {

__device__ __align__(256) unsigned char scratch[MD_NOALLOC_SCRATCH_BYTES];
static_assert(kBalMaxWorkspace <= MD_NOALLOC_SCRATCH_BYTES,
              "every balanced verify plan must fit the static scratch");

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// The device address of the current device's scratch (looked up once per
// device), or nullptr with *err set.
void* scratch_address(int dev, hipError_t* err) {
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch[dev].load(std::memory_order_relaxed);
  if (p) return p;
  void* addr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !addr) {
    *err = e != hipSuccess ? e : hipErrorInvalidSymbol;
    return nullptr;
  }
  g_scratch[dev].store(addr, std::memory_order_release);
  return addr;
}

}  // namespace

}  // namespace md

extern "C" int md_attn_noalloc(const md_attn_args* a, int32_t mode, int32_t n_sink,
                               int32_t window, void* stream) {
  if (!a || (mode != MD_MODE_VERIFY && mode != MD_MODE_DRAFT)) return MD_ERR_INVALID_ARG;
  // Sizes first (host arithmetic only; 0 for malformed sizes, which the call
  // itself then reports): a plan whose workspace exceeds the scratch is
  // refused before any HIP call.
  if (md_workspace_bytes(a, mode, n_sink, window) > MD_NOALLOC_SCRATCH_BYTES)
    return MD_ERR_WORKSPACE;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return md::hip_fail(e);
  if (dev < 0 || dev >= md::kMaxDevices) return MD_ERR_UNSUPPORTED;
  if (stream) {
    // The scratch address belongs to the current device: the stream must too.
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess) return md::hip_fail(e);
    if (sdev != dev) return MD_ERR_INVALID_ARG;
  }
  void* ws = md::scratch_address(dev, &e);
  if (!ws) return md::hip_fail(e);
  return md::run_attention(a, mode, n_sink, window, stream, nullptr, nullptr, ws,
                           MD_NOALLOC_SCRATCH_BYTES, nullptr);
}
