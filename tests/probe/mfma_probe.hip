// mfma_probe.hip -- test infrastructure: issues raw gfx950 bf16 / fp16 MFMAs on
// operand slots the host supplies, so that the CPU oracle's model of one
// instruction can be checked against the hardware (paper Sec. 4: numerical
// experiments on crafted inputs read the arithmetic off the instruction).
// One wave per case; case c reads operands [c][lane][0..7] and the
// accumulator [c][lane][..] and writes the result in the same slot layout.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef short shortx8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef int intx8 __attribute__((ext_vector_type(8)));

__global__ __launch_bounds__(64) void probe16(const shortx8* A, const shortx8* B, const floatx4* C,
                                              floatx4* D, int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, A[i]),
                                                 __builtin_bit_cast(bf16x8, B[i]), C[i], 0, 0, 0);
}

__global__ __launch_bounds__(64) void probe32(const shortx8* A, const shortx8* B, const floatx16* C,
                                              floatx16* D, int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, A[i]),
                                                 __builtin_bit_cast(bf16x8, B[i]), C[i], 0, 0, 0);
}

__global__ __launch_bounds__(64) void probe16h(const shortx8* A, const shortx8* B, const floatx4* C,
                                               floatx4* D, int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, A[i]),
                                                __builtin_bit_cast(f16x8, B[i]), C[i], 0, 0, 0);
}

__global__ __launch_bounds__(64) void probe32h(const shortx8* A, const shortx8* B, const floatx16* C,
                                               floatx16* D, int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, A[i]),
                                                __builtin_bit_cast(f16x8, B[i]), C[i], 0, 0, 0);
}

// The fp8 instruction of the same shape (OCP e4m3 operands, 8 bytes per lane:
// lane l holds A[l%16][8(l/16)+e], B[8(l/16)+e][l%16], byte e).
__global__ __launch_bounds__(64) void probe16f8(const long* A, const long* B, const floatx4* C, floatx4* D,
                                                int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_16x16x32_fp8_fp8(A[i], B[i], C[i], 0, 0, 0);
}

// 32x32x16 with e4m3 operands: lane l holds A[l%32][8(l/32)+e], B[8(l/32)+e][l%32].
__global__ __launch_bounds__(64) void probe32f8(const long* A, const long* B, const floatx16* C, floatx16* D,
                                                int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_f32_32x32x16_fp8_fp8(A[i], B[i], C[i], 0, 0, 0);
}

// The block-scaled f8f6f4 instructions with both operands e4m3 (format code 0)
// and both E8M0 scales 127 (= 1.0): 32 bytes per lane.  16x16x128: lane l's
// bytes 0..15 hold k = 16(l/16) + e, bytes 16..31 hold k = 64 + 16(l/16) + e;
// 32x32x64: bytes 0..15 hold k = 16(l/32) + e, bytes 16..31 k = 32 + 16(l/32) + e.
__global__ __launch_bounds__(64) void probe16f8s(const intx8* A, const intx8* B, const floatx4* C, floatx4* D,
                                                 int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(A[i], B[i], C[i], 0, 0, 0, 127, 0, 127);
}

__global__ __launch_bounds__(64) void probe32f8s(const intx8* A, const intx8* B, const floatx16* C,
                                                 floatx16* D, int ncases) {
  const int c = blockIdx.x, l = threadIdx.x;
  if (c >= ncases) return;
  const size_t i = (size_t)c * 64 + l;
  D[i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(A[i], B[i], C[i], 0, 0, 0, 127, 0, 127);
}

// instr 0: 16x16x32 bf16 (4 accumulator floats per lane), 1: 32x32x16 bf16
// (16); 2 and 3: the same shapes with fp16 operands; 4: 16x16x32 with e4m3
// operands (8 bytes per lane, not 16); 5: 32x32x16 e4m3 (8 bytes, 16
// floats); 6: 16x16x128 and 7: 32x32x64 block-scaled e4m3 at scale 1 (32
// bytes per lane; 4 and 16 floats).
// All pointers are device pointers sized for ncases.
extern "C" int mfma_probe(int instr, int ncases, const void* A, const void* B, const void* C,
                          void* D, void* stream) {
  if (ncases <= 0) return 0;
  (void)hipGetLastError();   // an error left by an earlier call is not this launch's
  hipStream_t s = (hipStream_t)stream;
  if (instr == 0)
    hipLaunchKernelGGL(probe16, dim3(ncases), dim3(64), 0, s, (const shortx8*)A, (const shortx8*)B,
                       (const floatx4*)C, (floatx4*)D, ncases);
  else if (instr == 1)
    hipLaunchKernelGGL(probe32, dim3(ncases), dim3(64), 0, s, (const shortx8*)A, (const shortx8*)B,
                       (const floatx16*)C, (floatx16*)D, ncases);
  else if (instr == 2)
    hipLaunchKernelGGL(probe16h, dim3(ncases), dim3(64), 0, s, (const shortx8*)A, (const shortx8*)B,
                       (const floatx4*)C, (floatx4*)D, ncases);
  else if (instr == 3)
    hipLaunchKernelGGL(probe32h, dim3(ncases), dim3(64), 0, s, (const shortx8*)A, (const shortx8*)B,
                       (const floatx16*)C, (floatx16*)D, ncases);
  else if (instr == 4)
    hipLaunchKernelGGL(probe16f8, dim3(ncases), dim3(64), 0, s, (const long*)A, (const long*)B,
                       (const floatx4*)C, (floatx4*)D, ncases);
  else if (instr == 5)
    hipLaunchKernelGGL(probe32f8, dim3(ncases), dim3(64), 0, s, (const long*)A, (const long*)B,
                       (const floatx16*)C, (floatx16*)D, ncases);
  else if (instr == 6)
    hipLaunchKernelGGL(probe16f8s, dim3(ncases), dim3(64), 0, s, (const intx8*)A, (const intx8*)B,
                       (const floatx4*)C, (floatx4*)D, ncases);
  else if (instr == 7)
    hipLaunchKernelGGL(probe32f8s, dim3(ncases), dim3(64), 0, s, (const intx8*)A, (const intx8*)B,
                       (const floatx16*)C, (floatx16*)D, ncases);
  else
    return -1;
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? 0 : -1000 - (int)e;   // -1000 - the HIP error code
}
