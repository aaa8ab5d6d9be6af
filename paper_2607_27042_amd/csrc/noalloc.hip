// gptq2d_round without any allocation: the sweep's workspace (deferred
// feedback, errors, C = L E, per-tile objective partials) lives in a
// file-scope device array instead of caller memory, for callers that cannot
// allocate (code under graph capture, tight serving loops).
#include <mutex>
#include <string>

#include "device.hpp"
#include "internal.hpp"

namespace g2d {

// Maximum workspace of the entry point. Every device the library runs on
// holds one copy of `scratch` from the module's load until the process ends.
constexpr size_t kScratchBytes = (size_t)64 << 20;

// Never passed to a kernel or a copy by name: in host code the name is a
// stand-in, not a device address. Host code uses the per-device address that
// hipGetSymbolAddress returns.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

// Address of this device's copy of `scratch`, looked up once per device with
// that device current (the caller has checked that `dev` is current).
static gptq2d_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("device index out of range of the no-allocation scratch table");
    return GPTQ2D_ERR_INVALID_ARG;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) {
      set_error("hipGetSymbolAddress(scratch) returned NULL");
      return GPTQ2D_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return GPTQ2D_OK;
}

}  // namespace g2d

using namespace g2d;

extern "C" gptq2d_status gptq2d_round_noalloc(gptq2d_factors_t f, gptq2d_dtype dt, const void* X,
                                              int64_t ldx, int32_t* Z, int64_t ldz, void* Y,
                                              int64_t ldy, double* objective, int32_t* status_word,
                                              void* stream) {
  const gptq2d_status sa = check_round_args(f, dt, X, ldx, Z, ldz, Y, ldy);
  if (sa != GPTQ2D_OK) return sa;
  if (!status_word) {
    set_error("status_word is NULL");
    return GPTQ2D_ERR_INVALID_ARG;
  }
  const size_t need = workspace_bytes(*f);
  if (need > kScratchBytes) {
    set_error("gptq2d_round_noalloc: an " + std::to_string(f->m) + " x " + std::to_string(f->n) +
              " problem needs " + std::to_string(need) + " bytes of workspace, more than the " +
              std::to_string(kScratchBytes >> 20) +
              " MiB it holds (4 x 8 bytes per entry of the 64-padded matrix); use gptq2d_round");
    return GPTQ2D_ERR_WORKSPACE;
  }
  gptq2d_status st = check_device(f);
  if (st != GPTQ2D_OK) return st;
  void* base = nullptr;
  st = scratch_address(f->device, &base);
  if (st != GPTQ2D_OK) return st;
  // the sweep's buffers in this device's scratch; the error word is the
  // caller's (the sweep clears it with a kernel before its first stage)
  Workspace ws = workspace_carve(*f, base);
  ws.flags = status_word;
  return launch_round(*f, dt, X, ldx, Z, ldz, Y, ldy, objective, ws, (hipStream_t)stream,
                      /*allow_timing=*/false);
}
