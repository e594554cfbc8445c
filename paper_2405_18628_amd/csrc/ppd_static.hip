// The verification step without a caller workspace: its scratch (residual
// stream, activations, attention and GEMM partial sums, tile counters,
// status word) lives in a device array of this library, so the call
// allocates nothing.  Each GPU the library runs on holds its own copy of the
// array until the process ends; its device address is looked up once per
// device (hipGetSymbolAddress) and used for every kernel argument.
#include <mutex>

#include "ppd_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[PPD_STATIC_WS_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices] = {nullptr};

__global__ void copy_status_kernel(const uint32_t *status, uint32_t *out) { *out = *status; }

}  // namespace

extern "C" ppd_status ppd_verify_step_static(const ppd_model *model, const ppd_kv *kv, int32_t L,
                                             int32_t T, const int32_t *ids, const int32_t *depth,
                                             const uint64_t *mask, float *logits, int32_t *pred,
                                             uint32_t *status_out, void *stream) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return ppd_fail(PPD_EDEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return ppd_fail(PPD_EDEVICE, "device %d out of range", dev);
  void *ws = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
      // the array's address on the current device (its host-side name is not
      // a device address)
      e = hipGetSymbolAddress(&g_scratch[dev], HIP_SYMBOL(scratch));
      if (e != hipSuccess) {
        g_scratch[dev] = nullptr;
        return ppd_fail(PPD_EDEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
      }
    }
    ws = g_scratch[dev];
  }
  if (!kv) return ppd_fail(PPD_EINVAL, "kv cache pointers must be set");
  if (T < 1 || T > PPD_T_MAX) return ppd_fail(PPD_EINVAL, "T=%d outside [1, %d]", T, PPD_T_MAX);
  const size_t need = ppd_workspace_bytes(model, T, kv->capacity);
  if (need == 0) return PPD_EINVAL;  // message set by ppd_workspace_bytes
  if (need > (size_t)PPD_STATIC_WS_BYTES)
    return ppd_fail(PPD_EWORKSPACE,
                    "the step needs %zu bytes of workspace, more than the static %zu-byte array",
                    need, (size_t)PPD_STATIC_WS_BYTES);
  // the header (status word, line of zeros) starts at zero for every call:
  // the array keeps whatever the previous call on this GPU left
  ppd_status st = ppd_workspace_init(ws, need, stream);
  if (st != PPD_OK) return st;
  st = ppd_verify_step(model, kv, L, T, ids, depth, mask, ws, need, logits, pred, stream);
  if (st != PPD_OK) return st;
  if (status_out) {
    hipLaunchKernelGGL(copy_status_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream,
                       (const uint32_t *)ws, status_out);
    e = hipGetLastError();
    if (e != hipSuccess) return ppd_fail(PPD_EDEVICE, "status copy: %s", hipGetErrorString(e));
  }
  return PPD_OK;
}
