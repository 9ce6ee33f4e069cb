// layer_noalloc.hip - eqb_layer for callers that cannot allocate device
// memory: the layer's working buffers live in one file-scope device array
// instead of a caller-owned workspace.
//
// The array is a host-side symbol in host code, not a device address: host
// code reaches it only through the pointer hipGetSymbolAddress returns, taken
// once per device with that device current and kept per device.
#include <mutex>

#include "eqb_internal.hpp"

namespace eqb {
namespace {

constexpr size_t kScratchBytes = EQB_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::once_flag g_once[kMaxDevices];
void* g_ptr[kMaxDevices];
hipError_t g_err[kMaxDevices];

// The scratch array's device address on the current device.
eqb_status scratch_ptr(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return EQB_ERR_HIP;
  std::call_once(g_once[dev], [dev] {
    void* p = nullptr;
    g_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_ptr[dev] = (g_err[dev] == hipSuccess) ? p : nullptr;
  });
  if (g_err[dev] != hipSuccess || g_ptr[dev] == nullptr) return EQB_ERR_HIP;
  *out = g_ptr[dev];
  return EQB_OK;
}

// Zeroes n bytes (a multiple of 16) at p with 16-byte vector stores.  A
// kernel rather than hipMemsetAsync, so that a caller may capture the call in
// a graph.
__global__ __launch_bounds__(256) void zero_kernel(uint4* __restrict__ p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x)
    p[i] = make_uint4(0, 0, 0, 0);
}

}  // namespace
}  // namespace eqb

using namespace eqb;

extern "C" eqb_status eqb_layer_noalloc(const uint16_t* z, const float* b, int64_t T, int32_t E, int32_t K,
                                        const int64_t* part_off, int32_t P, int32_t* topk_idx,
                                        float* topk_score, float* tau, int32_t* load, uint16_t* q_bf16,
                                        float* b_next, int32_t* hist_hi_sum, int32_t* hist_lo_sum,
                                        int32_t* dev_status, void* stream) {
  // the argument checks of eqb_layer, except the workspace's.  The array
  // holds the layer's counters only: the fine pass adds its counts to the
  // partition slabs instead of storing per-block images.
  size_t need = 0;
  if (eqb_layer_workspace_size(E, part_off ? P : 1) != 0)
    need = layer_workspace(nullptr, E, part_off ? P : 1, nullptr, false);
  if (need > kScratchBytes) return EQB_ERR_SCRATCH;
  if (T < 0 || T > INT32_MAX || K < 1 || K >= E) return EQB_ERR_INVALID_ARG;
  if (need == 0) return (E == 8 || E == 16 || E == 32 || E == 64 || E == 128 || E == 256) ?
                        EQB_ERR_INVALID_ARG : EQB_ERR_UNSUPPORTED;
  if (eqb_rank(T, K, E) < 1) return EQB_ERR_RANK;
  if (!z || !b || !topk_idx || !topk_score || !tau || !load || !q_bf16 || !b_next || !dev_status)
    return EQB_ERR_INVALID_ARG;
  void* ws = nullptr;
  const eqb_status st = scratch_ptr(&ws);
  if (st != EQB_OK) return st;
  // Calls on one device share the array and find the last call's contents:
  // the part this layer uses is cleared before it runs.  (A layer leaves its
  // workspace zeroed, but one that failed part-way may not have.)
  const hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t n16 = need / 16;
  const int blocks = (int)((n16 + 255) / 256 < 1024 ? (n16 + 255) / 256 : 1024);
  zero_kernel<<<blocks, 256, 0, s>>>(static_cast<uint4*>(ws), n16);
  if (launch_status() != EQB_OK) return EQB_ERR_HIP;
  return layer_call(z, b, T, E, K, part_off, P, topk_idx, topk_score, tau, load, q_bf16, b_next, hist_hi_sum,
                    hist_lo_sum, dev_status, ws, need, false, nullptr, stream);
}
