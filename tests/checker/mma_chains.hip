// One wave's 16 x 16 fp32 tile C = A (16 x K, bf16, row-major) . B (given as
// B^T, 16 x K, bf16, row-major) on v_mfma_f32_16x16x32_bf16, written several
// ways, for the static order checker.  Compiled to gfx950 assembly only;
// never launched.
#include <hip/hip_runtime.h>

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short shortx8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;

#define KERNEL extern "C" __global__ void __launch_bounds__(64)

__device__ __forceinline__ floatx4 step(const short* A, const short* Bt, int K, int k0, floatx4 acc) {
  const int l = threadIdx.x, r = l & 15, g = l >> 4;
  const shortx8 a = *(const shortx8*)&A[r * K + k0 + 8 * g];
  const shortx8 b = *(const shortx8*)&Bt[r * K + k0 + 8 * g];
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}

__device__ __forceinline__ void store(float* C, floatx4 acc) {
  const int l = threadIdx.x, r = l & 15, g = l >> 4;
  for (int i = 0; i < 4; ++i) C[(4 * g + i) * 16 + r] = acc[i];
}

// K = 64 in two instructions, unrolled
KERNEL mma_unrolled(const short* __restrict__ A, const short* __restrict__ Bt, float* __restrict__ C) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  acc = step(A, Bt, 64, 0, acc);
  acc = step(A, Bt, 64, 32, acc);
  store(C, acc);
}

// a K loop of step 32 (K bound by the caller)
KERNEL mma_loop32(const short* __restrict__ A, const short* __restrict__ Bt, float* __restrict__ C, int K) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma nounroll
  for (int k0 = 0; k0 < K; k0 += 32) acc = step(A, Bt, K, k0, acc);
  store(C, acc);
}

// a K loop of step 64, two instructions per iteration
KERNEL mma_loop64(const short* __restrict__ A, const short* __restrict__ Bt, float* __restrict__ C, int K) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma nounroll
  for (int k0 = 0; k0 < K; k0 += 64) {
    acc = step(A, Bt, K, k0, acc);
    acc = step(A, Bt, K, k0 + 32, acc);
  }
  store(C, acc);
}

// two accumulators (k 0-31 and 32-63) added at the end: another tree
KERNEL mma_two_acc(const short* __restrict__ A, const short* __restrict__ Bt, float* __restrict__ C) {
  floatx4 z = {0.f, 0.f, 0.f, 0.f};
  const floatx4 a0 = step(A, Bt, 64, 0, z), a1 = step(A, Bt, 64, 32, z);
  floatx4 acc;
  for (int i = 0; i < 4; ++i) acc[i] = a0[i] + a1[i];
  store(C, acc);
}

// k 32-63 first, then 0-31: another chain
KERNEL mma_reversed(const short* __restrict__ A, const short* __restrict__ Bt, float* __restrict__ C) {
  floatx4 acc = {0.f, 0.f, 0.f, 0.f};
  acc = step(A, Bt, 64, 32, acc);
  acc = step(A, Bt, 64, 0, acc);
  store(C, acc);
}
