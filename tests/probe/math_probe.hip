// math_probe.hip -- test infrastructure: evaluates the library's device exp,
// SiLU and exp2 (paper_2609_11356_amd/csrc/dg_device.h, the functions the
// fused epilogue, the softmax and the attention kernels call) on a
// contiguous range of binary32 bit patterns, so that the tests can compare
// every binary32 input with the CPU oracle's versions.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../paper_2609_11356_amd/csrc/dg_device.h"

__global__ __launch_bounds__(256) void exp_silu_range(uint64_t start, int64_t count, float* e, float* s) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) {
    const float x = dg::bits_f32((uint32_t)(start + (uint64_t)i));
    e[i] = dg::exp_f32(x);
    s[i] = dg::silu_f32(x);
  }
}

// e[i] = exp_f32(x), s[i] = silu_f32(x) for the binary32 value x with bits
// start + i, i < count (start + count <= 2^32); e and s are device buffers of
// count floats.  Returns a hipError_t.
extern "C" int math_probe_exp_silu(uint64_t start, int64_t count, float* e, float* s, void* stream) {
  if (count <= 0) return 0;
  if (start + (uint64_t)count > ((uint64_t)1 << 32) || !e || !s) return (int)hipErrorInvalidValue;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(exp_silu_range, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, start, count, e, s);
  return (int)hipGetLastError();
}

__global__ __launch_bounds__(256) void exp2_range(uint64_t start, int64_t count, float* e) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256)
    e[i] = dg::exp2_f32(dg::bits_f32((uint32_t)(start + (uint64_t)i)));
}

// e[i] = exp2_f32(x) for the binary32 x with bits start + i, i < count.
extern "C" int math_probe_exp2(uint64_t start, int64_t count, float* e, void* stream) {
  if (count <= 0) return 0;
  if (start + (uint64_t)count > ((uint64_t)1 << 32) || !e) return (int)hipErrorInvalidValue;
  int64_t blocks = (count + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(exp2_range, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, start, count, e);
  return (int)hipGetLastError();
}
