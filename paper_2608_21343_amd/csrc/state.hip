// Stream start / restart kernels (per-stream model id and carried state).
#include "device.hpp"
#include "launch.hpp"

namespace tbias {

__global__ void init_states_kernel(ArenaView A, int32_t B, int32_t K, const int32_t* model_ids,
                                   int32_t* states, float* scores) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)B * K) return;
  int32_t b = (int32_t)(i / K), k = (int32_t)(i % K);
  int32_t m = model_ids[b];
  int32_t s = (m == -1) ? TB_STATE_NONE : ((m < -1 || m >= A.n_models) ? TB_STATE_INVALID : 0);
  states[i] = s;
  if (scores) scores[i] = (k == 0) ? 0.f : -__builtin_huge_valf();
}

// tb_init_states plus empty hypotheses and trees of the streaming beam.
__global__ void init_beam_stream_kernel(ArenaView A, int32_t B, int32_t K,
                                        const int32_t* model_ids, int32_t* states, float* scores,
                                        tb_hyp* hyps, int32_t* tree_len) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)B * K) return;
  int32_t b = (int32_t)(i / K), k = (int32_t)(i % K);
  int32_t m = model_ids[b];
  states[i] = (m == -1) ? TB_STATE_NONE : ((m < -1 || m >= A.n_models) ? TB_STATE_INVALID : 0);
  scores[i] = (k == 0) ? 0.f : -__builtin_huge_valf();
  tb_hyp h;
  h.hash = 0ull;
  h.prefix_hash = 0ull;
  h.last = -1;
  h.node = -1;
  hyps[i] = h;
  if (k == 0) tree_len[b] = 0;
}

__global__ void reset_stream_kernel(int32_t b, int32_t m, int32_t K, int32_t* model_ids,
                                    int32_t* states, float* scores) {
  int32_t k = threadIdx.x;
  if (k >= K) return;
  if (k == 0) model_ids[b] = m;
  states[(int64_t)b * K + k] = (m == -1) ? TB_STATE_NONE : 0;
  if (scores) scores[(int64_t)b * K + k] = (k == 0) ? 0.f : -__builtin_huge_valf();
}

// A kernel that does nothing, for measuring what a launch of a given shape
// costs by itself (tb_debug_launch_empty).
__global__ void empty_kernel(int32_t* sink) {
  extern __shared__ int32_t pad[];
  if (sink && threadIdx.x == 0 && blockIdx.x == 0xffffffffu) sink[0] = pad[0];
}

hipError_t launch_empty(int32_t grid, int32_t block, int32_t lds_bytes, hipStream_t st) {
  if (lds_bytes > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&empty_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, lds_bytes);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(empty_kernel, dim3(grid), dim3(block), (size_t)lds_bytes, st, nullptr);
  return hipGetLastError();
}

hipError_t launch_init_states(const ArenaView& A, int32_t B, int32_t K, const int32_t* model_ids,
                              int32_t* states, float* scores, hipStream_t st) {
  int64_t n = (int64_t)B * K;
  int threads = 256;
  int blocks = (int)((n + threads - 1) / threads);
  hipLaunchKernelGGL(init_states_kernel, dim3(blocks), dim3(threads), 0, st, A, B, K, model_ids,
                     states, scores);
  return hipGetLastError();
}

hipError_t launch_init_beam_stream(const ArenaView& A, int32_t B, int32_t K,
                                   const int32_t* model_ids, int32_t* states, float* scores,
                                   tb_hyp* hyps, int32_t* tree_len, hipStream_t st) {
  int64_t n = (int64_t)B * K;
  int threads = 256;
  int blocks = (int)((n + threads - 1) / threads);
  hipLaunchKernelGGL(init_beam_stream_kernel, dim3(blocks), dim3(threads), 0, st, A, B, K,
                     model_ids, states, scores, hyps, tree_len);
  return hipGetLastError();
}

hipError_t launch_reset_stream(int32_t b, int32_t m, int32_t K, int32_t* model_ids,
                               int32_t* states, float* scores, hipStream_t st) {
  hipLaunchKernelGGL(reset_stream_kernel, dim3(1), dim3(64), 0, st, b, m, K, model_ids, states,
                     scores);
  return hipGetLastError();
}

}  // namespace tbias
