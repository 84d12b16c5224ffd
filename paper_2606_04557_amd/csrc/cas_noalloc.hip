// The forward without allocation: a static device scratch per GPU replaces
// the caller's workspace, and the launch tables travel as kernel arguments.
#include <hip/hip_runtime.h>

#include <map>
#include <mutex>

#include "../../include/cas.h"
#include "cas_internal.h"

// Workspace of cas_prefix_attn_fwd_noalloc: launch tables, exact-pass flags
// and split partials. Every GPU holds its own copy at its own address; host
// code uses only the address hipGetSymbolAddress returns for the current
// device (this name on the host is a stand-in, not a device address).
static __device__ __align__(256) char scratch[CAS_NOALLOC_SCRATCH_BYTES];

namespace {

std::mutex g_scratch_mu;
std::map<int, void *> g_scratch_ptr;   // device ordinal -> its copy of `scratch`

// Device address of `scratch` on the current device, looked up once per device.
hipError_t scratch_address(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void *ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (!ptr) return hipErrorInvalidSymbol;
  g_scratch_ptr.emplace(dev, ptr);
  *out = ptr;
  return hipSuccess;
}

// One kernel-argument load of table bytes: 16-byte pieces, one per lane.
struct TableChunk {
  uint4 data[cas::kTableArgChunk / 16];
  uint4 *dst;
  uint32_t pieces;
};

__global__ __launch_bounds__(cas::kTableArgChunk / 16) void table_args_kernel(TableChunk c) {
  const uint32_t i = threadIdx.x;
  if (i < c.pieces) c.dst[i] = c.data[i];
}

}  // namespace

namespace cas {

hipError_t launch_table_args_upload(const void *host, size_t bytes, void *dst, hipStream_t s) {
  const char *src = (const char *)host;
  for (size_t off = 0; off < bytes; off += kTableArgChunk) {
    const size_t n = bytes - off < (size_t)kTableArgChunk ? bytes - off : (size_t)kTableArgChunk;
    TableChunk c;
    __builtin_memcpy(c.data, src + off, n);
    c.dst = (uint4 *)((char *)dst + off);
    c.pieces = (uint32_t)(n / 16);
    hipLaunchKernelGGL(table_args_kernel, dim3(1), dim3(kTableArgChunk / 16), 0, s, c);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace cas

extern "C" cas_status_t cas_prefix_attn_fwd_noalloc(const cas_problem_t *p, const void *q,
                                                    const void *k_self, const void *v_self, void *o,
                                                    float *lse, void *hip_stream) {
  return cas::prefix_attn_fwd_run(p, q, k_self, v_self, o, lse, nullptr, CAS_NOALLOC_SCRATCH_BYTES,
                                  (hipStream_t)hip_stream, scratch_address);
}
