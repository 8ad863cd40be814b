// Boosted greedy step for wide vocabularies (V+1 > 2048 logits per row).
//
// A row is spread over one workgroup of 256 threads: thread i holds tokens
// v = i + 256 j (j < TPV) and keeps, in registers, their logits (the next
// row's already in flight), their classes, and their root move (target state
// and its psi). A step from state s (Sec. II-B fused scoring operation):
//
//  1. the children of the states on s's suffix chain (s, link(s), ..., the
//     root excluded) override the root move of their class, the deepest state
//     first: a per-class tag table in LDS points the overridden classes at a
//     short list of (target state, psi) built level by level;
//  2. every thread forms key[v] = z[v] + psi[delta(s, class v)] for its tokens
//     (blank: z[V] + phi[s], which keeps the state), its best (key, index)
//     and its part of the log-sum-exp (its own max and sum of exponentials);
//  3. one workgroup reduction gives the lowest-index maximum, the state it
//     moves to, and lse.
//
// The T steps of a stream are cut into segments decoded by separate
// workgroups in parallel, as the segmented kernel does with waves: a segment
// after the first starts two rows early from the root state (a guess), and
// greedy_wide_fix_kernel then repairs the segment boundaries in order from the
// exact state, recomputing until the trajectory meets the stored one. The
// outputs equal sequential decoding for any input.
#include "launch.hpp"
#include "wide.hpp"

namespace tbias {
namespace wide {

constexpr int kWarm = 2;     // warm-up rows of a guessed segment start
constexpr int kMinSeg = 16;  // shortest segment worth a workgroup
struct Red {
  float k, z, psi, m, s;
  int32_t v, ns;
};

// (key, index) argmax carrying the target state, psi and logit of the winner,
// together with a log-sum-exp (max m, sum s of exp(z - m)) merge.
__device__ __forceinline__ void merge(Red& a, const Red& b) {
  if (better(b.k, b.v, a.k, a.v)) {
    a.k = b.k;
    a.v = b.v;
    a.ns = b.ns;
    a.psi = b.psi;
    a.z = b.z;
  }
  const float M = fmaxf(a.m, b.m);
  const float sa = (a.m == M) ? a.s : a.s * __expf(a.m - M);
  const float sb = (b.m == M) ? b.s : b.s * __expf(b.m - M);
  a.m = M;
  a.s = sa + sb;
}

// One step from state s on the row in o.z; returns the winner and lse in
// every thread. Contains workgroup barriers: all threads must call it.
template <int TPV>
__device__ __forceinline__ Red step(Ctx& C, const Own<TPV>& o, int32_t s, int32_t V1, Red* red) {
  const int32_t V = V1 - 1;
  const int tid = threadIdx.x;
  float phi_s;
  const bool chain = build_overrides(C, s, phi_s);

  float bk = kNegInf, bpsi = 0.f, bz = 0.f;
  int32_t bv = INT_MAX, bns = 0;
  float m = kNegInf;
#pragma unroll
  for (int j = 0; j < TPV; ++j) m = fmaxf(m, o.z[j]);
  float se = 0.f;  // the blank's logit is also in its slot of o.z: counted once there
#pragma unroll
  for (int j = 0; j < TPV; ++j) se += (o.z[j] == kNegInf) ? 0.f : __expf(o.z[j] - m);
  for_each_move<TPV>(C, o, chain, [&](int j, float p, int32_t ns) {
    const float key = o.z[j] + p;
    const bool gt = key > bk;  // tokens ascend: strict > keeps the lowest index on ties
    bk = gt ? key : bk;
    bv = gt ? tid + kThreads * j : bv;
    bns = gt ? ns : bns;
    bpsi = gt ? p : bpsi;
    bz = gt ? o.z[j] : bz;
  });
  if (tid == V % kThreads) {  // the blank keeps the state; phi[s] in its key, no boost
    const float key = o.zb + phi_s;
    if (better(key, V, bk, bv)) {
      bk = key;
      bv = V;
      bns = (C.mode == 1) ? s : C.fixed;
      bpsi = phi_s;
      bz = o.zb;
    }
  }
  // wave reductions (DPP): the winner's fields from its lane, and the
  // log-sum-exp as the wave max of the thread maxima and the rescaled sums
  Red r;
  const int32_t wl = wave_argmax_dpp(bk, bv, r.k, r.v);
  r.ns = __builtin_amdgcn_readlane(bns, wl);
  r.psi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bpsi), wl));
  r.z = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(bz), wl));
  r.m = wave_max_dpp(m);
  r.s = wave_sum_dpp((m == r.m) ? se : se * __expf(m - r.m));
  if ((tid & 63) == 0) red[tid >> 6] = r;
  __syncthreads();
  Red f = red[0];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) merge(f, red[w]);
  __syncthreads();  // red is rewritten by the next step
  f.psi -= phi_s;   // the boost: psi[next] - phi[s] (0 for the blank)
  return f;
}

struct Shared {
  Red red[kWaves];
  int32_t nlist;
};

template <class Ld, int TPV>
__global__ __launch_bounds__(kThreads) void greedy_wide_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ Shared sh;
  lds_poison(&sh, sizeof(sh));
  lds_poison(dyn, wide::lds_bytes(A));
  const int32_t V1 = A.V1;
  const int32_t b = blockIdx.x % B;
  const int32_t g = blockIdx.x / B;
  const typename Ld::T* col = logits + (int64_t)b * stride;
  const int64_t tstride = (int64_t)B * stride;
  const int32_t m = model_ids[b];
  const int32_t s0 = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s0, off, n);
  const int32_t t0 = g * L;
  const int32_t t1 = (t0 + L < T) ? t0 + L : T;
  const bool exact = (g == 0) || mode != 1;
  const int32_t tw = exact ? t0 : (t0 - kWarm > 0 ? t0 - kWarm : 0);

  Own<TPV> o;
  float zn[TPV], zbn = kNegInf;
  if (t0 < t1) load_row<Ld, TPV>(o.z, o.zb, col + (int64_t)tw * tstride, V1);
  const int32_t fixed = unbiased_state(mode, s0 == TB_STATE_TIMEOUT);
  own_tables<TPV>(o, A, m, mode, fixed);
  Ctx C = make_ctx(A, off, mode, fixed, &sh.nlist, dyn);
  __syncthreads();

  int32_t s = (mode == 1) ? (g == 0 ? s0 : 0) : C.fixed;
  for (int32_t t = tw; t < t1; ++t) {
    if (t + 1 < t1) load_row<Ld, TPV>(zn, zbn, col + (int64_t)(t + 1) * tstride, V1);
    const Red f = step<TPV>(C, o, s, V1, sh.red);
    if (t >= t0 && threadIdx.x == 0) {
      const int64_t oi = (int64_t)t * B + b;
      out_tok[oi] = f.v;
      out_state[oi] = f.ns;
      out_score[oi] = (f.z - (f.m + __logf(f.s))) + f.psi;
    }
    s = f.ns;
    if (t + 1 < t1) {
#pragma unroll
      for (int j = 0; j < TPV; ++j) o.z[j] = zn[j];
      o.zb = zbn;
    }
  }
  if (G == 1 && threadIdx.x == 0 && T > 0) states[b] = s;
}

// Repairs the segment boundaries of each stream in order and writes the carry.
template <class Ld, int TPV>
__global__ __launch_bounds__(kThreads) void greedy_wide_fix_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ Shared sh;
  lds_poison(&sh, sizeof(sh));
  lds_poison(dyn, wide::lds_bytes(A));
  const int32_t V1 = A.V1;
  const int32_t b = blockIdx.x;
  const typename Ld::T* col = logits + (int64_t)b * stride;
  const int64_t tstride = (int64_t)B * stride;
  const int32_t m = model_ids[b];
  // the main kernel consumed the carried state; only biased streams whose
  // carried state was valid have guessed segment starts
  const bool biased = m >= 0 && m < A.n_models;
  int32_t done = 0;      // rows before this are exact
  int32_t x_done = 0;    // exact state after row done-1, when done > 0 came from a repair
  if (biased) {
    const int32_t off = A.model_off[m];
    Own<TPV> o;
    float zn[TPV], zbn = kNegInf;
    own_tables<TPV>(o, A, m, 1, 0);
    Ctx C = make_ctx(A, off, 1, 0, &sh.nlist, dyn);
    __syncthreads();
    for (int32_t gg = 1; gg < G; ++gg) {
      const int32_t tb0 = gg * L;
      if (tb0 >= T) break;
      if (done > tb0) continue;  // an earlier repair already ran past this boundary
      int32_t x = (done == tb0) ? x_done : out_state[(int64_t)(tb0 - 1) * B + b];
      if (x < 0) break;  // an invalid carried state: the stream was decoded unbiased
      load_row<Ld, TPV>(o.z, o.zb, col + (int64_t)tb0 * tstride, V1);
      int32_t t = tb0;
      for (; t < T; ++t) {
        if (t + 1 < T) load_row<Ld, TPV>(zn, zbn, col + (int64_t)(t + 1) * tstride, V1);
        const int64_t oi = (int64_t)t * B + b;
        const int32_t old = out_state[oi];
        const Red f = step<TPV>(C, o, x, V1, sh.red);
        if (threadIdx.x == 0) {
          out_tok[oi] = f.v;
          out_state[oi] = f.ns;
          out_score[oi] = (f.z - (f.m + __logf(f.s))) + f.psi;
        }
        x = f.ns;
        if (x == old) {  // the stored trajectory from here on is exact
          ++t;
          break;
        }
        if (t + 1 < T) {
#pragma unroll
          for (int j = 0; j < TPV; ++j) o.z[j] = zn[j];
          o.zb = zbn;
        }
      }
      done = t;
      x_done = x;
    }
  }
  if (threadIdx.x == 0 && T > 0)
    states[b] = (done == T) ? x_done : out_state[(int64_t)(T - 1) * B + b];
}

// Segments per stream: enough workgroups for about two per CU, segments of
// at least kMinSeg rows, every workgroup owning rows.
inline void wide_geometry(int32_t T, int32_t B, int32_t& G, int32_t& L) {
  G = (512 + B - 1) / B;
  const int32_t gmax = T / kMinSeg;
  if (G > gmax) G = gmax;
  if (G < 1) G = 1;
  L = (T + G - 1) / G;
  while (G > 1 && (G - 1) * L >= T) --G;
}

template <class Ld, int TPV>
hipError_t launch_t(const ArenaView& A, const void* logits, int32_t T, int32_t B, int64_t stride,
                    const int32_t* model_ids, int32_t* states, int32_t* out_tok,
                    int32_t* out_state, float* out_score, hipStream_t st) {
  typedef typename Ld::T TT;
  const size_t lds = lds_bytes(A);
  int32_t G, L;
  wide_geometry(T, B, G, L);
  hipLaunchKernelGGL((greedy_wide_kernel<Ld, TPV>), dim3(B * G), dim3(kThreads), lds, st, A,
                     static_cast<const TT*>(logits), T, B, stride, G, L, model_ids, states,
                     out_tok, out_state, out_score);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || G == 1) return e;
  hipLaunchKernelGGL((greedy_wide_fix_kernel<Ld, TPV>), dim3(B), dim3(kThreads), lds, st, A,
                     static_cast<const TT*>(logits), T, B, stride, G, L, model_ids, states,
                     out_tok, out_state, out_score);
  return hipGetLastError();
}

}  // namespace wide

// Wide vocabularies: V+1 in (2048, 256 * 41]. hipErrorNotSupported otherwise,
// or when the LDS tables would not fit.
hipError_t launch_greedy_wide(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, int32_t* out_tok, int32_t* out_state,
                              float* out_score, hipStream_t st) {
  const int32_t V1 = A.V1;
  if (V1 <= 2048 || V1 > wide::kThreads * 41) return hipErrorNotSupported;
  if (wide::lds_bytes(A) > 60 * 1024) return hipErrorNotSupported;
  const int tpv = (V1 + wide::kThreads - 1) / wide::kThreads;
#define TB_WIDE(N)                                                                           \
  if (tpv <= N)                                                                              \
    return dtype == TB_F32                                                                   \
               ? wide::launch_t<LoadF32, N>(A, logits, T, B, row_stride, model_ids, states,  \
                                            out_tok, out_state, out_score, st)               \
               : wide::launch_t<LoadBF16, N>(A, logits, T, B, row_stride, model_ids, states, \
                                             out_tok, out_state, out_score, st);
  TB_WIDE(12)
  TB_WIDE(16)
  TB_WIDE(24)
  TB_WIDE(33)
  TB_WIDE(41)
#undef TB_WIDE
  return hipErrorNotSupported;
}

}  // namespace tbias
