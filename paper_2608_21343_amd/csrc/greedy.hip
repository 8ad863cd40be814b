// Boosted greedy step (reference kernel): one workgroup per stream.
//
// Per step the workgroup (Sec. II-B fused scoring operation):
//   1. reads the stream's logit row and forms the log-softmax normaliser;
//   2. runs the suffix-link traversal from the current state: the children of
//      every state on the suffix chain s, link(s), ... (excluding the root)
//      override the root move of their class, the deepest state winning;
//   3. forms key[v] = z[v] + psi[delta(s, class v)] (blank: z[V] + phi[s]),
//      takes the lowest-index maximum and advances the state.
// The override table lives in LDS, indexed by class: the overriding target
// state of every class, and one bit per class marking the entries written for
// the current state (cleared every step), 4 B + 1 bit per class, so any V up
// to the 32767 tokens the boundary accepts fits.
#include <climits>

#include "device.hpp"
#include "ref_table.hpp"
#include "launch.hpp"

namespace tbias {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline float block_max(float x, float* red) {
  x = wave_max(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r = fmaxf(r, red[i]);
  __syncthreads();
  return r;
}

__device__ inline float block_sum(float x, float* red) {
  x = wave_sum(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r += red[i];
  __syncthreads();
  return r;
}

__device__ inline void block_argmax(float& k, int32_t& i, float* redk, int32_t* redi) {
  wave_argmax(k, i);
  if ((threadIdx.x & 63) == 0) {
    redk[threadIdx.x >> 6] = k;
    redi[threadIdx.x >> 6] = i;
  }
  __syncthreads();
  k = redk[0];
  i = redi[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w)
    if (better(redk[w], redi[w], k, i)) { k = redk[w]; i = redi[w]; }
  __syncthreads();
}

template <class Ld>
__global__ __launch_bounds__(kThreads) void greedy_ref_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  extern __shared__ int32_t smem[];
  lds_poison(smem, ref_table_bytes(A.V1 - 1));  // the launch's dynamic LDS
  const int32_t V1 = A.V1, V = V1 - 1;
  int32_t* odst = smem;
  uint32_t* mark = reinterpret_cast<uint32_t*>(smem + V);
  const int32_t n_mark = (V + 31) >> 5;
  __shared__ float redf[kWaves];
  __shared__ int32_t redi[kWaves];
  __shared__ int32_t s_next;

  const int tid = threadIdx.x;
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  int32_t s = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s, off, n);  // 1 biased, 0 none, -1 invalid
  const int32_t fixed = unbiased_state(mode, s == TB_STATE_TIMEOUT);
  const float* rpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* rdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;

  for (int32_t t = 0; t < T; ++t) {
    const typename Ld::T* row = logits + ((int64_t)t * B + b) * stride;
    float mx = -__builtin_huge_valf();
    for (int32_t v = tid; v < V1; v += kThreads) mx = fmaxf(mx, Ld::get(row, v));
    mx = block_max(mx, redf);
    float se = 0.f;
    for (int32_t v = tid; v < V1; v += kThreads) se += expf(Ld::get(row, v) - mx);
    se = block_sum(se, redf);
    const float lse = mx + logf(se);

    float phi_s = 0.f;
    if (mode == 1) {
      phi_s = A.phi[off + s];
      for (int32_t i = tid; i < n_mark; i += kThreads) mark[i] = 0u;
      __syncthreads();
      for (int32_t x = s; x != 0; x = A.link[off + x]) {
        const int32_t fc = A.first_child[off + x], nc = A.n_child[off + x];
        for (int32_t j = tid; j < nc; j += kThreads) {
          const int32_t y = fc + j;
          const int32_t c = A.label[off + y];
          if (!ref_marked(mark, c)) {  // children of one state: distinct classes
            atomicOr(&mark[c >> 5], 1u << (c & 31));
            odst[c] = y;
          }
        }
        __syncthreads();
      }
    }

    float bk = -__builtin_huge_valf();
    int32_t bi = INT_MAX;
    for (int32_t v = tid; v < V1; v += kThreads) {
      const float z = Ld::get(row, v);
      float p = 0.f;
      if (mode == 1) {
        if (v == V) {
          p = phi_s;
        } else {
          const int32_t c = A.class_map[v];
          p = (c >= 0 && ref_marked(mark, c)) ? A.psi[off + odst[c]] : rpsi[v];
        }
      }
      const float key = z + p;
      if (better(key, v, bk, bi)) { bk = key; bi = v; }
    }
    block_argmax(bk, bi, redf, redi);

    if (tid == 0) {
      const int32_t v = bi;
      int32_t ns;
      float bst = 0.f;
      if (mode == 1) {
        if (v == V) {
          ns = s;
        } else {
          const int32_t c = A.class_map[v];
          ns = (c >= 0 && ref_marked(mark, c)) ? odst[c] : rdst[v];
          bst = A.psi[off + ns] - phi_s;
        }
      } else {
        ns = fixed;
      }
      const float z = Ld::get(row, v);
      const int64_t o = (int64_t)t * B + b;
      out_tok[o] = v;
      out_state[o] = ns;
      out_score[o] = (z - lse) + bst;
      s_next = ns;
    }
    __syncthreads();
    s = s_next;
  }
  if (tid == 0 && T > 0) states[b] = s;
}

}  // namespace

hipError_t launch_greedy(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                         int32_t B, int64_t row_stride, const int32_t* model_ids, int32_t* states,
                         int32_t* out_tok, int32_t* out_state, float* out_score, hipStream_t st) {
  // the segmented kernels (waves as segments for V+1 <= 2048, workgroups as
  // segments above); the reference kernel for anything larger, or when a
  // test selects it
  if (debug_greedy_kernel() != kGreedyRef) {
    hipError_t e = launch_greedy_seg(A, logits, dtype, T, B, row_stride, model_ids, states,
                                     out_tok, out_state, out_score, st);
    if (e != hipErrorNotSupported) return e;
    (void)hipGetLastError();  // clear the sticky "not supported" before the fallback
    e = launch_greedy_wide(A, logits, dtype, T, B, row_stride, model_ids, states, out_tok,
                           out_state, out_score, st);
    if (e != hipErrorNotSupported) return e;
    (void)hipGetLastError();
  }
  const size_t lds = ref_table_bytes(A.V1 - 1);
  if (dtype == TB_F32) {
    allow_dynamic_lds(&greedy_ref_kernel<LoadF32>, lds);
    hipLaunchKernelGGL(greedy_ref_kernel<LoadF32>, dim3(B), dim3(kThreads), lds, st, A,
                       static_cast<const float*>(logits), T, B, row_stride, model_ids, states,
                       out_tok, out_state, out_score);
  } else {
    allow_dynamic_lds(&greedy_ref_kernel<LoadBF16>, lds);
    hipLaunchKernelGGL(greedy_ref_kernel<LoadBF16>, dim3(B), dim3(kThreads), lds, st, A,
                       static_cast<const uint16_t*>(logits), T, B, row_stride, model_ids, states,
                       out_tok, out_state, out_score);
  }
  return hipGetLastError();
}

}  // namespace tbias
