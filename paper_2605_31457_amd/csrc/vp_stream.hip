// Streaming-read ceiling of the GPU: one read of a device buffer through the
// two access paths the decode-step kernels could use, so a benchmark can hold
// their bandwidth against what a plain read reaches on the same GPU. Not part
// of the method.
//   mode 0  16-byte vector loads into registers, 8 per lane in flight
//           (256-lane work-groups, a grid-stride over 32 KB blocks);
//   mode 1  HBM -> LDS copies (global_load_lds_dwordx4, 1 KB of consecutive
//           bytes per wave instruction), 16 KB per one-wave work-group in
//           flight, the copy path of the context and kept passes.
// Both carry the non-temporal cache policy of those kernels.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "vp_internal.h"

namespace vp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kRegLanes = 256;
constexpr int kRegLoads = 8;           // loads in flight per lane
constexpr int kLdsChunk = 16 * 1024;   // bytes in flight per one-wave work-group
constexpr uint32_t kNever = 0x9e3779b9u;

__global__ __launch_bounds__(kRegLanes) void read_regs_kernel(const u32x4* __restrict__ src, size_t n16,
                                                               uint32_t* sink) {
  uint32_t acc = 0;
  const size_t stride = static_cast<size_t>(gridDim.x) * kRegLanes * kRegLoads;
  for (size_t base = static_cast<size_t>(blockIdx.x) * kRegLanes * kRegLoads + threadIdx.x; base < n16;
       base += stride) {
    u32x4 v[kRegLoads];
#pragma unroll
    for (int u = 0; u < kRegLoads; ++u) {
      const size_t i = base + static_cast<size_t>(u) * kRegLanes;
      v[u] = i < n16 ? __builtin_nontemporal_load(src + i) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kRegLoads; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  // keeps the loads (the data decides; a write, if any, is one word)
  if (acc == kNever) atomicOr(sink, 1u);
}

__global__ __launch_bounds__(64) void read_lds_kernel(const char* __restrict__ src, size_t nchunks) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsChunk];
  const int lane = threadIdx.x;
  for (size_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
    const char* p = src + c * kLdsChunk + 16 * lane;
#pragma unroll
    for (int j = 0; j < kLdsChunk / 1024; ++j)
      __builtin_amdgcn_global_load_lds((global_void*)(p + 1024 * j), (lds_void*)(lds + 1024 * j), 16, 0, 2);
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the copies have landed before the slots are reused
  }
}

}  // namespace

hipError_t launch_stream_read(const void* src, size_t bytes, int mode, uint32_t* sink, hipStream_t st) {
  if (mode == 0) {
    const size_t n16 = bytes / 16;
    const size_t per = static_cast<size_t>(kRegLanes) * kRegLoads;
    size_t grid = (n16 + per - 1) / per;
    if (grid > 4096) grid = 4096;  // 16 work-groups per CU, then a grid-stride
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(read_regs_kernel, dim3(static_cast<unsigned>(grid)), dim3(kRegLanes), 0, st,
                       static_cast<const u32x4*>(src), n16, sink);
  } else {
    const size_t nchunks = bytes / kLdsChunk;
    size_t grid = nchunks < 2048 ? nchunks : 2048;  // 8 one-wave work-groups per CU
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(read_lds_kernel, dim3(static_cast<unsigned>(grid)), dim3(64), 0, st,
                       static_cast<const char*>(src), nchunks);
  }
  return hipGetLastError();
}

}  // namespace vp
