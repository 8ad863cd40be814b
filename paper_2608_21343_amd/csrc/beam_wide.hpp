// Boosted beam step for wide vocabularies (V+1 > 2048, K <= 8): one
// workgroup of 256 threads per stream (templates; instantiated in
// beam_wide_f32.hip and beam_wide_bf16.hip).
//
// Per step the workgroup takes the K hypotheses in turn, each with its own
// logit row [t, b, k] (the next row is loaded while one is scored):
//
//  * the row's normaliser: max in float32, sum of exponentials and log in
//    float64 (exp_nonpos), rounded once to float32, as every beam kernel;
//  * the classes overridden in the hypothesis' state (wide.hpp), then the
//    candidates c_k + key over the row with c_k = (S_k - lse_k) - phi(s_k);
//    each thread keeps its MAXK best (value, flat index k*(V+1)+v) with the
//    state the candidate moves to, its psi and its logit;
//  * after the K rows, K rounds of a workgroup argmax over the threads' list
//    heads give the K best in order (larger value, then lower flat index);
//    slot j takes parent k_j, token v_j, the target state, step score
//    (z - lse_k) + (psi - phi(s_k)) (0 boost for the blank) and S_j.
//
// States and scores are carried across calls (Sec. II-C).
#pragma once

#include "launch.hpp"
#include "wide.hpp"

namespace tbias {
namespace wide {

// A candidate: value, flat index, target state, psi of the move, logit.
struct Cand {
  float c, psi, z;
  int32_t f, ns;
};

template <int MAXK>
struct alignas(16) BeamShared {
  Cand red[kWaves];
  float redm[kWaves];
  double reds[kWaves];
  int32_t nlist;
  int32_t bad;
  int32_t tmo;  // a slot carried TB_STATE_TIMEOUT
  int32_t hyp_s[MAXK];
  float hyp_S[MAXK];
  float hyp_lse[MAXK];
  float hyp_phi[MAXK];
  Cand sel[MAXK];
};

template <int MAXK>
__device__ __forceinline__ void list_insert(Cand (&l)[MAXK], const Cand& x) {
  if (!better(x.c, x.f, l[MAXK - 1].c, l[MAXK - 1].f)) return;
  l[MAXK - 1] = x;
#pragma unroll
  for (int j = MAXK - 1; j > 0; --j) {
    if (better(l[j].c, l[j].f, l[j - 1].c, l[j - 1].f)) {
      const Cand tmp = l[j];
      l[j] = l[j - 1];
      l[j - 1] = tmp;
    }
  }
}

template <class Ld, int TPV, int MAXK>
__global__ __launch_bounds__(kThreads) void beam_wide_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int32_t K,
    int64_t stride, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    float* __restrict__ scores, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_parent,
    int32_t* __restrict__ out_state, float* __restrict__ out_step, float* __restrict__ out_cum) {
  extern __shared__ __align__(16) unsigned char dyn[];
  __shared__ BeamShared<MAXK> sh;
  lds_poison(&sh, sizeof(sh));
  lds_poison(dyn, lds_bytes(A));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int tid = threadIdx.x;
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  int mode = (m == -1) ? 0 : 1;
  if (m < -1 || m >= A.n_models) mode = -1;
  int32_t off = 0, n = 0;
  if (mode == 1) {
    off = A.model_off[m];
    n = A.model_n[m];
  }
  if (tid == 0) { sh.bad = 0; sh.tmo = 0; }
  __syncthreads();
  if (tid < K) {
    const int32_t s = states[(int64_t)b * K + tid];
    sh.hyp_s[tid] = s;
    sh.hyp_S[tid] = scores[(int64_t)b * K + tid];
    if (mode == 1 && (s < 0 || s >= n)) sh.bad = 1;
    if (s == TB_STATE_TIMEOUT) sh.tmo = 1;
  }
  __syncthreads();
  if (mode == 1 && sh.bad) mode = -1;  // uniform: an invalid carried state decodes unbiased
  const int32_t fixed = unbiased_state(mode, sh.tmo != 0);
  Own<TPV> o;
  float zn[TPV], zbn = kNegInf;
  own_tables<TPV>(o, A, m, mode, fixed);
  Ctx C = make_ctx(A, off, mode, fixed, &sh.nlist, dyn);
  auto row_of = [&](int32_t t, int32_t k) {
    return logits + (((int64_t)t * B + b) * K + k) * stride;
  };
  if (T > 0) load_row<Ld, TPV>(o.z, o.zb, row_of(0, 0), V1);
  __syncthreads();

  for (int32_t t = 0; t < T; ++t) {
    Cand l[MAXK];
#pragma unroll
    for (int j = 0; j < MAXK; ++j) l[j] = Cand{kNegInf, 0.f, 0.f, INT_MAX, 0};
    for (int32_t k = 0; k < K; ++k) {
      const bool more = (k + 1 < K) || (t + 1 < T);
      if (more) {
        const int32_t tn = (k + 1 < K) ? t : t + 1, kn = (k + 1 < K) ? k + 1 : 0;
        load_row<Ld, TPV>(zn, zbn, row_of(tn, kn), V1);
      }
      const int32_t s = __builtin_amdgcn_readfirstlane(sh.hyp_s[k]);
      const float S_k = sh.hyp_S[k];
      // normaliser: float32 max, float64 sum and log, one rounding
      float mx = kNegInf;
#pragma unroll
      for (int j = 0; j < TPV; ++j) mx = fmaxf(mx, o.z[j]);
      mx = wave_max_dpp(mx);
      if ((tid & 63) == 0) sh.redm[tid >> 6] = mx;
      __syncthreads();
      float M = sh.redm[0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) M = fmaxf(M, sh.redm[w]);
      const double Md = (double)M;
      double se = 0.0;
#pragma unroll
      for (int j = 0; j < TPV; ++j)
        se += (o.z[j] == kNegInf) ? 0.0 : exp_nonpos((double)o.z[j] - Md);
      se = wave_sum_d(se);
      if ((tid & 63) == 0) sh.reds[tid >> 6] = se;
      __syncthreads();
      double St = sh.reds[0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) St += sh.reds[w];
      const float lse = (float)(Md + log(St));
      float phi_s;
      const bool chain = build_overrides(C, s, phi_s);
      const float ck = (S_k - lse) - phi_s;
      const int32_t fk = k * V1;
      for_each_move<TPV>(C, o, chain, [&](int j, float p, int32_t ns) {
        const float key = o.z[j] + p;
        list_insert<MAXK>(l, Cand{ck + key, p, o.z[j], fk + tid + kThreads * j, ns});
      });
      if (tid == V % kThreads)  // the blank keeps the state; phi[s] in its key, no boost
        list_insert<MAXK>(l, Cand{ck + (o.zb + phi_s), phi_s, o.zb, fk + V,
                                  (mode == 1) ? s : fixed});
      if (tid == 0) {
        sh.hyp_lse[k] = lse;
        sh.hyp_phi[k] = phi_s;
      }
      __syncthreads();  // the next row rewrites the override table and reductions
      if (more) {
#pragma unroll
        for (int j = 0; j < TPV; ++j) o.z[j] = zn[j];
        o.zb = zbn;
      }
    }

    // K rounds of a workgroup argmax over the threads' list heads
    for (int32_t j = 0; j < K; ++j) {
      float bc;
      int32_t bf;
      const int32_t wl = wave_argmax_dpp(l[0].c, l[0].f, bc, bf);
      if ((tid & 63) == 0) {
        Cand w;
        w.c = bc;
        w.f = bf;
        w.ns = __builtin_amdgcn_readlane(l[0].ns, wl);
        w.psi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l[0].psi), wl));
        w.z = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l[0].z), wl));
        sh.red[tid >> 6] = w;
      }
      // lane wl of its wave held the head; it pops it if it wins overall
      __syncthreads();
      Cand best = sh.red[0];
#pragma unroll
      for (int w = 1; w < kWaves; ++w)
        if (better(sh.red[w].c, sh.red[w].f, best.c, best.f)) best = sh.red[w];
      if (l[0].f == best.f) {
#pragma unroll
        for (int q = 0; q < MAXK - 1; ++q) l[q] = l[q + 1];
        l[MAXK - 1] = Cand{kNegInf, 0.f, 0.f, INT_MAX, 0};
      }
      if (tid == 0) sh.sel[j] = best;
      __syncthreads();
    }
    if (tid < K) {
      const Cand c = sh.sel[tid];
      const int32_t f = (c.f >= 0 && c.f < K * V1) ? c.f : 0;  // only with NaN logits
      const int32_t k = f / V1, v = f - k * V1;
      const int64_t oi = ((int64_t)t * B + b) * K + tid;
      out_tok[oi] = v;
      out_parent[oi] = k;
      out_state[oi] = c.ns;
      out_step[oi] = (c.z - sh.hyp_lse[k]) + (c.psi - sh.hyp_phi[k]);
      out_cum[oi] = c.c;
    }
    __syncthreads();  // every slot has read its parent's entries
    if (tid < K) {
      sh.hyp_s[tid] = sh.sel[tid].ns;
      sh.hyp_S[tid] = sh.sel[tid].c;
    }
    __syncthreads();
  }
  if (tid < K && T > 0) {
    states[(int64_t)b * K + tid] = sh.hyp_s[tid];
    scores[(int64_t)b * K + tid] = sh.hyp_S[tid];
  }
}

template <class Ld, int TPV, int MAXK>
hipError_t launch_beam_wide_t(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                              int32_t K, int64_t stride, const int32_t* model_ids, int32_t* states,
                              float* scores, int32_t* out_tok, int32_t* out_parent,
                              int32_t* out_state, float* out_step, float* out_cum,
                              hipStream_t st) {
  hipLaunchKernelGGL((beam_wide_kernel<Ld, TPV, MAXK>), dim3(B), dim3(kThreads), lds_bytes(A),
                     st, A, static_cast<const typename Ld::T*>(logits), T, B, K, stride,
                     model_ids, states, scores, out_tok, out_parent, out_state, out_step,
                     out_cum);
  return hipGetLastError();
}

typedef hipError_t (*BeamWideLaunch)(const ArenaView&, const void*, int32_t, int32_t, int32_t,
                                     int64_t, const int32_t*, int32_t*, float*, int32_t*,
                                     int32_t*, int32_t*, float*, float*, hipStream_t);

// Launcher for tokens per thread tpv and list size maxk (nullptr if none).
template <class Ld>
BeamWideLaunch beam_wide_launcher(int tpv, int maxk) {
#define TB_BW(N)                                                                  \
  if (tpv <= N) return maxk <= 4 ? &launch_beam_wide_t<Ld, N, 4> : &launch_beam_wide_t<Ld, N, 8>;
  TB_BW(16)
  TB_BW(33)
  TB_BW(41)
#undef TB_BW
  return nullptr;
}

BeamWideLaunch beam_wide_launcher_f32(int tpv, int maxk);
BeamWideLaunch beam_wide_launcher_bf16(int tpv, int maxk);

}  // namespace wide
}  // namespace tbias
