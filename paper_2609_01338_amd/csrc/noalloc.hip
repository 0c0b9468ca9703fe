// mz_q4_gemm_split_noalloc: the split-K Q4_0 GEMM (mz_q4_gemm_split) for
// callers that cannot allocate -- code under HIP graph capture, tight serving
// loops, hosts that forbid device allocation.  Its fp32 partials live in one
// fixed device array of this file instead of a caller or library buffer, so
// the call allocates nothing: no hipMalloc, hipFree or allocating library
// routine, on any path.
//
// The array's address on a device is looked up once per device (with that
// device current) on the first call there, and kept; the kernels take that
// address as their workspace argument, exactly as mz_q4_gemm_split passes its
// caller's buffer, so both entry points run the same kernels on the same
// inputs and give the same bits.  Every call on one GPU shares its array: the
// partial kernels write every element the reduce reads within the same call,
// so nothing needs clearing, but calls that overlap on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/mz.h"
#include "mz_internal.h"
#include "mz_kernels.h"

namespace {

static_assert(MZ_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
static __device__ __align__(256) uint8_t scratch[MZ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];   // the array's device address per device, once looked up

// Address of `scratch` on the current device (looked up on its first call).
mz_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    mzrt::set_error("no usable current HIP device");
    return MZ_EHIP;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      mzrt::set_error("hipGetSymbolAddress of the scratch array failed");
      return MZ_EHIP;
    }
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MZ_OK;
}

}  // namespace

extern "C" mz_status mz_q4_gemm_split_noalloc(const void* x_f16, int32_t m, int32_t n_pad, int32_t k,
                                               const void* w_packed, int32_t epilogue, void* y, int32_t n_split,
                                               void* stream) {
  if (!x_f16 || !w_packed || !y) {
    mzrt::set_error("NULL pointer");
    return MZ_EINVAL;
  }
  if (m < 1 || n_pad < 1 || k < 1 || n_pad % mzk::kGemmTileN || k % mzk::kGemmTileK || epilogue < 0 ||
      epilogue > 2 || n_split < 1 || n_split > 1024) {
    mzrt::set_error("bad sizes, epilogue or n_split (as mz_q4_gemm_split)");
    return MZ_EINVAL;
  }
  if (mzk::gemm_splitk_ws_bytes(m, n_pad, n_split) > (int64_t)MZ_NOALLOC_SCRATCH_BYTES) {
    mzrt::set_error("n_split * m * n_pad * 4 bytes of partials exceed the fixed scratch of this entry point");
    return MZ_EINVAL;
  }
  hipStream_t s = (hipStream_t)stream;
  if (s) {
    int cur = -1;
    hipDevice_t sdev = -1;
    if (hipGetDevice(&cur) != hipSuccess || hipStreamGetDevice(s, &sdev) != hipSuccess || sdev != cur) {
      mzrt::set_error("the stream must belong to the current device");
      return MZ_EINVAL;
    }
  }
  void* ws = nullptr;
  const mz_status st = scratch_address(&ws);
  if (st != MZ_OK) return st;
  mzk::launch_gemm_q4_splitk(x_f16, m, n_pad, k, w_packed, epilogue, y, n_split, ws, s);
  if (hipGetLastError() != hipSuccess) {
    mzrt::set_error("kernel launch failed");
    return MZ_EHIP;
  }
  return MZ_OK;
}
