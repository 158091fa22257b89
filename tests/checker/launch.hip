// Host launchers for the order checker's fixture kernels (test
// infrastructure): the same sources the checker reads, built with the same
// floating-point flags, so that a GPU test can confirm on the part that
// kernels the checker puts in one class give the same bits and kernels in
// different classes do not.
#include <cstring>

#include "lane_trees.hip"
#include "mma_chains.hip"

// x: at least 512 floats (n <= 512 for the strided folds), y: 64 floats
extern "C" int run_lane(const char* name, const float* x, float* y, int n) {
  struct K { const char* name; void (*f2)(const float*, float*); void (*f3)(const float*, float*, int); int threads; };
  static const K ks[] = {
      {"up_library", up_library, nullptr, 64},       {"up_shfl", up_shfl, nullptr, 64},
      {"up_four", up_four, nullptr, 64},             {"up_two", up_two, nullptr, 64},
      {"up_reversed", up_reversed, nullptr, 64},     {"down_library", down_library, nullptr, 64},
      {"down_shfl", down_shfl, nullptr, 64},         {"up_steps_swapped", up_steps_swapped, nullptr, 64},
      {"chain", chain, nullptr, 64},                 {"groups16", groups16, nullptr, 64},
      {"block_256", block_256, nullptr, 256},        {"block_128x2", block_128x2, nullptr, 128},
      {"block_256_chain", block_256_chain, nullptr, 256},
      {"strided_fold", nullptr, strided_fold, 64},   {"strided_fold_unroll2", nullptr, strided_fold_unroll2, 64},
      {"strided_fold_two_acc", nullptr, strided_fold_two_acc, 64}};
  if (n < 128 || n > 512) return -2;              // the strided folds read x[l] and x[l + 64] at least
  for (const K& k : ks) {
    if (std::strcmp(k.name, name) != 0) continue;
    if (k.f2) hipLaunchKernelGGL(k.f2, dim3(1), dim3(k.threads), 0, 0, x, y);
    else hipLaunchKernelGGL(k.f3, dim3(1), dim3(k.threads), 0, 0, x, y, n);
    return hipDeviceSynchronize() == hipSuccess ? 0 : -3;
  }
  return -1;
}

// A, Bt: 16 x K bf16 each; C: 16 x 16 floats; K a multiple of 64, at most 256
extern "C" int run_mma(const char* name, const short* A, const short* Bt, float* C, int K) {
  if (K < 64 || K > 256 || K % 64) return -2;
  if (!std::strcmp(name, "mma_loop32")) hipLaunchKernelGGL(mma_loop32, dim3(1), dim3(64), 0, 0, A, Bt, C, K);
  else if (!std::strcmp(name, "mma_loop64")) hipLaunchKernelGGL(mma_loop64, dim3(1), dim3(64), 0, 0, A, Bt, C, K);
  else if (K != 64) return -2;
  else if (!std::strcmp(name, "mma_unrolled")) hipLaunchKernelGGL(mma_unrolled, dim3(1), dim3(64), 0, 0, A, Bt, C);
  else if (!std::strcmp(name, "mma_two_acc")) hipLaunchKernelGGL(mma_two_acc, dim3(1), dim3(64), 0, 0, A, Bt, C);
  else if (!std::strcmp(name, "mma_reversed")) hipLaunchKernelGGL(mma_reversed, dim3(1), dim3(64), 0, 0, A, Bt, C);
  else return -1;
  return hipDeviceSynchronize() == hipSuccess ? 0 : -3;
}
