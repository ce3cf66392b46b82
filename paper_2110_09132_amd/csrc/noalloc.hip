// The owner-major coalesce for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid
// allocation): emb_grad_coalesce_by_owner with its workspace held by the
// library in a static device array, `scratch`, of EMB_NOALLOC_SCRATCH_BYTES.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up once per device, with that device current, at
// the first call on it (hipGetSymbolAddress), and kept per device; only that
// address is ever handed to the kernels.  Each device holds its own copy of
// the array, at its own address, until the process ends.  Calls on one device
// share the array and race if they can overlap (different streams without
// ordering); the kernels clear what must start at zero themselves, so the
// array's contents on entry do not matter.
#include <mutex>

#include "common.h"
#include "launch.h"

namespace {

constexpr size_t kScratchBytes = EMB_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];  // device address of `scratch` on each device (null: not looked up yet)

// The device address of `scratch` on the current device.
int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return EMB_ERR_LAUNCH;
  if (dev < 0 || dev >= kMaxDevices) return EMB_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_dev[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return EMB_ERR_LAUNCH;
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return EMB_OK;
}

}  // namespace

extern "C" int emb_grad_coalesce_by_owner_noalloc(const int32_t* ids, int32_t T, const void* grad,
                                                  int32_t grad_dtype, int32_t D, int64_t V,
                                                  const int32_t* row_owner, int32_t P, int32_t* send_ids,
                                                  int32_t* seg_offsets, float* send_rows, int32_t* send_counts,
                                                  int32_t* send_offsets, int32_t* num_unique, int32_t* dev_status,
                                                  void* stream) {
  // the size limit first, on the host, before anything touches the device
  if (emb_grad_coalesce_workspace_bytes(T, V, D, grad_dtype) > kScratchBytes) return EMB_ERR_WORKSPACE;
  void* ws = nullptr;
  const int sst = scratch_address(&ws);
  if (sst != EMB_OK) return sst;
  const int st = emb::coalesce_by_owner_args_status(ids, T, grad, grad_dtype, D, V, row_owner, P, nullptr, -1,
                                                    send_ids, seg_offsets, send_rows, send_counts, send_offsets,
                                                    num_unique, ws, kScratchBytes);
  if (st != EMB_OK) return st;
  emb::CoalesceVariant var;
  var.row_owner = row_owner;
  var.P = P;
  const hipError_t e = emb::launch_coalesce(ids, T, grad, grad_dtype == EMB_BF16, D, V, var, send_ids, seg_offsets,
                                            send_rows, num_unique, send_counts, send_offsets, ws, dev_status,
                                            static_cast<hipStream_t>(stream));
  return e == hipSuccess ? EMB_OK : EMB_ERR_LAUNCH;
}
