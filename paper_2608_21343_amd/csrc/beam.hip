// Boosted beam step (reference kernel): one workgroup per stream.
//
// For each of the K hypotheses of a stream the workgroup forms the row's
// log-sum-exp (float64 sum and log, rounded once to float32), the boosted keys
// key[v] = z[v] + psi[delta(s_k, class v)] (blank: z[V] + phi[s_k]) and the
// candidates cand = ((S_k - lse_k) - phi[s_k]) + key[v]. Every thread keeps
// its own best MAXK candidates; K rounds of a workgroup argmax then pick the
// K best over all K*(V+1) candidates (ties to the lowest flat index
// k*(V+1)+v), and the surviving hypotheses are reordered with their advanced
// graph states (Sec. II-C: scores and states carried across calls).
#include <climits>

#include "beam_fast.hpp"
#include "beam_pipe.hpp"
#include "beam_wide.hpp"
#include "device.hpp"
#include "ref_table.hpp"
#include "launch.hpp"

namespace tbias {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ inline float bmax(float x, float* red) {
  x = wave_max(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  float r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r = fmaxf(r, red[i]);
  __syncthreads();
  return r;
}

__device__ inline double bsum_d(double x, double* red) {
  x = wave_sum_d(x);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  double r = red[0];
#pragma unroll
  for (int i = 1; i < kWaves; ++i) r += red[i];
  __syncthreads();
  return r;
}

__device__ inline void bargmax(float& k, int32_t& i, float* redk, int32_t* redi) {
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

// Aho-Corasick move from local state x on class c (global memory walk).
__device__ inline int32_t ac_move(const ArenaView& A, int32_t off, int32_t x, int32_t c) {
  for (;;) {
    int32_t lo = A.first_child[off + x], hi = lo + A.n_child[off + x];
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      const int32_t l = A.label[off + mid];
      if (l == c) return mid;
      if (l < c) lo = mid + 1; else hi = mid;
    }
    if (x == 0) return 0;
    x = A.link[off + x];
  }
}

// With STREAM, the streaming beam (tb_boost_step_beam_stream) for rows and
// beams the one-wave-per-hypothesis kernel does not take: every hypothesis'
// normaliser first, then the recombination of equal label sequences (x's
// blank extension and the extension of x's prefix slot y by x's last label:
// the better in (value, flat index) order gets log(e^a + e^b), the other
// -inf), applied to the candidates as they are formed; hashes and tree
// records as in the fast kernel.
template <class Ld, int MAXK, bool STREAM>
__global__ __launch_bounds__(kThreads) void beam_ref_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int32_t K,
    int64_t stride, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    float* __restrict__ scores, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_parent,
    int32_t* __restrict__ out_state, float* __restrict__ out_step, float* __restrict__ out_cum,
    beamk::StreamArgs sa) {
  extern __shared__ int32_t smem[];
  lds_poison(smem, ref_table_bytes(A.V1 - 1));  // the launch's dynamic LDS
  const int32_t V1 = A.V1, V = V1 - 1;
  int32_t* odst = smem;
  uint32_t* mark = reinterpret_cast<uint32_t*>(smem + V);
  const int32_t n_mark = (V + 31) >> 5;
  __shared__ float redf[kWaves];
  __shared__ int32_t redi[kWaves];
  __shared__ double redd[kWaves];
  __shared__ int32_t sh_state[MAXK];
  __shared__ float sh_S[MAXK];
  __shared__ float sh_lse[MAXK];
  __shared__ float sh_phi[MAXK];
  __shared__ int32_t sel_idx[MAXK];
  __shared__ float sel_val[MAXK];
  __shared__ int32_t sh_bad, sh_tmo;
  // streaming beam: hypothesis carry and this step's merges (slot y's
  // patched tokens and values; slot x's blank)
  constexpr int SK = STREAM ? MAXK : 1;
  __shared__ uint64_t sh_h[SK], sh_hp[SK];
  __shared__ int32_t sh_lv[SK], sh_node[SK];
  __shared__ int32_t mod_n[SK], mod_tok[SK][SK];
  __shared__ float mod_val[SK][SK], blank_val[SK];
  __shared__ int32_t blank_set[SK];

  const int tid = threadIdx.x;
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  if (tid == 0) { sh_bad = 0; sh_tmo = 0; }
  __syncthreads();
  int32_t off = 0, n = 0;
  int mode = (m == -1) ? 0 : 1;
  if (m < -1 || m >= A.n_models) mode = -1;
  if (mode == 1) { off = A.model_off[m]; n = A.model_n[m]; }
  if (tid < K) {
    const int32_t s = states[(int64_t)b * K + tid];
    sh_state[tid] = s;
    sh_S[tid] = scores[(int64_t)b * K + tid];
    if (mode == 1 && (s < 0 || s >= n)) sh_bad = 1;
    if (s == TB_STATE_TIMEOUT) sh_tmo = 1;
    if constexpr (STREAM) {
      const tb_hyp hy = sa.hyps[(int64_t)b * K + tid];
      sh_h[tid] = hy.hash;
      sh_hp[tid] = hy.prefix_hash;
      sh_lv[tid] = hy.last;
      sh_node[tid] = hy.node;
    }
  }
  int32_t tlen = 0;
  if constexpr (STREAM) {
    const int32_t l = sa.tree_len[b];
    tlen = l < 0 ? 0 : (l > sa.cap ? sa.cap : l);
  }
  __syncthreads();  // sh_bad and sh_tmo are complete
  if (mode == 1 && sh_bad) mode = -1;
  const float* rpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* rdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;

  for (int32_t t = 0; t < T; ++t) {
    float lk[MAXK];
    int32_t li[MAXK];
#pragma unroll
    for (int j = 0; j < MAXK; ++j) { lk[j] = -__builtin_huge_valf(); li[j] = INT_MAX; }

    auto row_of = [&](int32_t k) {
      return logits + (((int64_t)t * B + b) * K + k) * stride;
    };
    auto row_lse = [&](const typename Ld::T* row) -> float {
      float mx = -__builtin_huge_valf();
      for (int32_t v = tid; v < V1; v += kThreads) mx = fmaxf(mx, Ld::get(row, v));
      mx = bmax(mx, redf);
      double se = 0.0;
      const double mxd = (double)mx;
      for (int32_t v = tid; v < V1; v += kThreads) se += exp((double)Ld::get(row, v) - mxd);
      se = bsum_d(se, redd);
      return (float)(mxd + log(se));
    };
    if constexpr (STREAM) {
      // every hypothesis' normaliser and phi, then the merges of the step
      for (int32_t k = 0; k < K; ++k) {
        const float l = row_lse(row_of(k));
        if (tid == 0) {
          sh_lse[k] = l;
          sh_phi[k] = (mode == 1) ? A.phi[off + sh_state[k]] : 0.f;
        }
      }
      if (tid < K) {
        mod_n[tid] = 0;
        blank_set[tid] = 0;
      }
      __syncthreads();
      if (tid == 0 && sa.recombine) {
        for (int32_t x = 0; x < K; ++x) {
          const int32_t v = sh_lv[x];
          if (!(sh_S[x] > -__builtin_huge_valf()) || v < 0 || v >= V) continue;
          for (int32_t y = 0; y < K; ++y) {
            if (y == x || !(sh_S[y] > -__builtin_huge_valf()) || sh_h[y] != sh_hp[x]) continue;
            const float cx = (sh_S[x] - sh_lse[x]) - sh_phi[x];
            const float cy = (sh_S[y] - sh_lse[y]) - sh_phi[y];
            const float psi_x = (mode == 1) ? A.psi[off + sh_state[x]] : 0.f;
            const float a = cx + (Ld::get(row_of(x), V) + sh_phi[x]);
            const float bv = cy + (Ld::get(row_of(y), v) + psi_x);
            if (a > -__builtin_huge_valf() && bv > -__builtin_huge_valf()) {
              const float merged = beamk::logaddexp32(a, bv);
              const bool keep_a = a > bv || (a == bv && x * V1 + V < y * V1 + v);
              blank_set[x] = 1;
              blank_val[x] = keep_a ? merged : -__builtin_huge_valf();
              const int32_t q = mod_n[y]++;
              mod_tok[y][q] = v;
              mod_val[y][q] = keep_a ? -__builtin_huge_valf() : merged;
            }
            break;  // the first prefix slot in index order
          }
        }
      }
      __syncthreads();
    }

    for (int32_t k = 0; k < K; ++k) {
      const typename Ld::T* row = row_of(k);
      float lse;
      if constexpr (STREAM) {
        lse = sh_lse[k];
      } else {
        lse = row_lse(row);
      }
      const int32_t s = sh_state[k];

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
      const float ck = (sh_S[k] - lse) - phi_s;
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
        float cand = ck + key;
        if constexpr (STREAM) {
          if (v == V) {
            if (blank_set[k]) cand = blank_val[k];
          } else {
            for (int32_t q = 0; q < mod_n[k]; ++q)
              if (mod_tok[k][q] == v) cand = mod_val[k][q];
          }
        }
        const int32_t f = k * V1 + v;
        if (better(cand, f, lk[MAXK - 1], li[MAXK - 1])) {
          lk[MAXK - 1] = cand;
          li[MAXK - 1] = f;
#pragma unroll
          for (int j = MAXK - 1; j > 0; --j) {
            if (better(lk[j], li[j], lk[j - 1], li[j - 1])) {
              const float tk = lk[j]; lk[j] = lk[j - 1]; lk[j - 1] = tk;
              const int32_t ti = li[j]; li[j] = li[j - 1]; li[j - 1] = ti;
            }
          }
        }
      }
      if (tid == 0) { sh_lse[k] = lse; sh_phi[k] = phi_s; }
      __syncthreads();  // the next hypothesis rewrites the override table
    }

    // K rounds of a workgroup argmax over the per-thread heads
    for (int32_t j = 0; j < K; ++j) {
      float hk = lk[0];
      int32_t hi = li[0];
      bargmax(hk, hi, redf, redi);
      if (li[0] == hi) {
#pragma unroll
        for (int q = 0; q < MAXK - 1; ++q) { lk[q] = lk[q + 1]; li[q] = li[q + 1]; }
        lk[MAXK - 1] = -__builtin_huge_valf();
        li[MAXK - 1] = INT_MAX;
      }
      if (tid == 0) { sel_val[j] = hk; sel_idx[j] = hi; }
    }
    __syncthreads();

    int32_t ns = 0;
    float nS = 0.f;
    uint64_t nh = 0ull, nhp = 0ull;
    int32_t nlv = -1, nnode = -1;
    int32_t nb_total = 0;  // kept non-blank extensions (streaming beam)
    if constexpr (STREAM) {
      for (int32_t q = 0; q < K; ++q) {
        int32_t fq = sel_idx[q];
        if (fq < 0 || fq >= K * V1) fq = 0;
        nb_total += (fq % V1 != V) ? 1 : 0;
      }
    }
    if (tid < K) {
      const int32_t j = tid;
      int32_t f = sel_idx[j];
      if (f < 0 || f >= K * V1) f = 0;  // only reachable with NaN logits
      const int32_t k = f / V1, v = f - k * V1;
      if constexpr (STREAM) {
        int32_t before = 0;
        for (int32_t q = 0; q < j; ++q) {
          int32_t fq = sel_idx[q];
          if (fq < 0 || fq >= K * V1) fq = 0;
          before += (fq % V1 != V) ? 1 : 0;
        }
        nh = sh_h[k];
        nhp = sh_hp[k];
        nlv = sh_lv[k];
        nnode = sh_node[k];
        if (v != V) {
          const int32_t r = tlen + before;
          nhp = sh_h[k];
          nh = sh_h[k] * (uint64_t)TB_HASH_MUL + (uint64_t)(v + 1);
          nlv = v;
          nnode = (r < sa.cap) ? r : -2;
          if (r < sa.cap) {
            sa.tree[((int64_t)b * sa.cap + r) * 2] = v;
            sa.tree[((int64_t)b * sa.cap + r) * 2 + 1] = sh_node[k];
          }
        }
      }
      const int32_t s = sh_state[k];
      float bst = 0.f;
      if (mode == 1) {
        if (v == V) {
          ns = s;
        } else {
          const int32_t c = A.class_map[v];
          ns = (c >= 0) ? ac_move(A, off, s, c) : rdst[v];
          bst = A.psi[off + ns] - sh_phi[k];
        }
      } else {
        ns = unbiased_state(mode, sh_tmo != 0);
      }
      const typename Ld::T* row = logits + (((int64_t)t * B + b) * K + k) * stride;
      const float z = Ld::get(row, v);
      const int64_t o = ((int64_t)t * B + b) * K + j;
      nS = sel_val[j];
      out_tok[o] = v;
      out_parent[o] = k;
      out_state[o] = ns;
      out_step[o] = (z - sh_lse[k]) + bst;
      out_cum[o] = nS;
    }
    __syncthreads();
    if (tid < K) {
      sh_state[tid] = ns;
      sh_S[tid] = nS;
      if constexpr (STREAM) {
        sh_h[tid] = nh;
        sh_hp[tid] = nhp;
        sh_lv[tid] = nlv;
        sh_node[tid] = nnode;
      }
    }
    if constexpr (STREAM) tlen += nb_total;
    __syncthreads();
  }
  if (tid < K && T > 0) {
    states[(int64_t)b * K + tid] = sh_state[tid];
    scores[(int64_t)b * K + tid] = sh_S[tid];
    if constexpr (STREAM) {
      tb_hyp hy;
      hy.hash = sh_h[tid];
      hy.prefix_hash = sh_hp[tid];
      hy.last = sh_lv[tid];
      hy.node = sh_node[tid];
      sa.hyps[(int64_t)b * K + tid] = hy;
      if (tid == 0) sa.tree_len[b] = tlen < sa.cap ? tlen : sa.cap;
    }
  }
}

template <class Ld, int MAXK, bool STREAM>
void launch_t(const ArenaView& A, const void* logits, int32_t T, int32_t B, int32_t K,
              int64_t stride, const int32_t* model_ids, int32_t* states, float* scores,
              int32_t* out_tok, int32_t* out_parent, int32_t* out_state, float* out_step,
              float* out_cum, hipStream_t st, beamk::StreamArgs sa) {
  const size_t lds = ref_table_bytes(A.V1 - 1);
  allow_dynamic_lds(&beam_ref_kernel<Ld, MAXK, STREAM>, lds);
  hipLaunchKernelGGL((beam_ref_kernel<Ld, MAXK, STREAM>), dim3(B), dim3(kThreads), lds, st, A,
                     static_cast<const typename Ld::T*>(logits), T, B, K, stride, model_ids,
                     states, scores, out_tok, out_parent, out_state, out_step, out_cum, sa);
}

template <class Ld, bool STREAM = false>
void launch_k(const ArenaView& A, const void* logits, int32_t T, int32_t B, int32_t K,
              int64_t stride, const int32_t* model_ids, int32_t* states, float* scores,
              int32_t* out_tok, int32_t* out_parent, int32_t* out_state, float* out_step,
              float* out_cum, hipStream_t st, beamk::StreamArgs sa = beamk::StreamArgs{}) {
  if (K <= 2)
    launch_t<Ld, 2, STREAM>(A, logits, T, B, K, stride, model_ids, states, scores, out_tok,
                            out_parent, out_state, out_step, out_cum, st, sa);
  else if (K <= 4)
    launch_t<Ld, 4, STREAM>(A, logits, T, B, K, stride, model_ids, states, scores, out_tok,
                            out_parent, out_state, out_step, out_cum, st, sa);
  else if (K <= 8)
    launch_t<Ld, 8, STREAM>(A, logits, T, B, K, stride, model_ids, states, scores, out_tok,
                            out_parent, out_state, out_step, out_cum, st, sa);
  else if (K <= 16)
    launch_t<Ld, 16, STREAM>(A, logits, T, B, K, stride, model_ids, states, scores, out_tok,
                             out_parent, out_state, out_step, out_cum, st, sa);
  else
    launch_t<Ld, 32, STREAM>(A, logits, T, B, K, stride, model_ids, states, scores, out_tok,
                             out_parent, out_state, out_step, out_cum, st, sa);
}

}  // namespace

// Kernel choice: the helper-wave kernel serves V+1 > 2048 with K <= 4 (rows
// up to 4224 float32 or 8320 bfloat16 tokens, where its two-slot LDS ring
// fits); the one-wave-per-hypothesis kernel serves V+1 <= 2048 with K <= 8
// (override sets that fit its lists); the wide-row kernel serves K <= 8 and
// V+1 in (2048, 256 * 41]; the reference kernel serves the rest. Tests can
// force the reference kernel, or skip the helper-wave kernel, through
// tb_debug_select_kernels.
hipError_t launch_beam(const ArenaView& A, const void* logits, int32_t dtype, int32_t T, int32_t B,
                       int32_t K, int64_t row_stride, const int32_t* model_ids, int32_t* states,
                       float* scores, int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                       float* out_step, float* out_cum, hipStream_t st) {
  const int32_t choice = debug_beam_kernel();
  const bool ref = choice == kBeamRef;
  const bool nopipe = choice == kBeamNoPipe;
  if (!ref && !nopipe && K <= 8) {
    bpipe::PipeLaunch f = dtype == TB_F32 ? bpipe::pipe_launcher_f32(A.V1, K)
                                          : bpipe::pipe_launcher_bf16(A.V1, K);
    if (f)
      return f(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok, out_parent,
               out_state, out_step, out_cum, st);
  }
  if (!ref && K <= 8 && A.V1 >= 2 && A.V1 <= 64 * 32 && A.max_override <= beamk::kOverCap) {
    const int per = (A.V1 + 63) / 64;
    const int maxk = K <= 2 ? 2 : (K <= 4 ? 4 : 8);
    beamk::BeamLaunch f = per <= 8    ? beamk::beam_launcher_1_8(per, maxk, dtype)
                          : per <= 16 ? beamk::beam_launcher_9_16(per, maxk, dtype)
                          : per <= 24 ? beamk::beam_launcher_17_24(per, maxk, dtype)
                                      : beamk::beam_launcher_25_32(per, maxk, dtype);
    if (f)
      return f(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok, out_parent,
               out_state, out_step, out_cum, st);
  }
  if (!ref && K <= 8 && A.V1 > 64 * 32 && A.V1 <= wide::kThreads * 41 &&
      wide::lds_bytes(A) <= 60 * 1024) {
    const int tpv = (A.V1 + wide::kThreads - 1) / wide::kThreads;
    const int maxk = K <= 4 ? 4 : 8;
    wide::BeamWideLaunch f = dtype == TB_F32 ? wide::beam_wide_launcher_f32(tpv, maxk)
                                             : wide::beam_wide_launcher_bf16(tpv, maxk);
    if (f)
      return f(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok, out_parent,
               out_state, out_step, out_cum, st);
  }
  if (dtype == TB_F32)
    launch_k<LoadF32>(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok,
                      out_parent, out_state, out_step, out_cum, st);
  else
    launch_k<LoadBF16>(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok,
                       out_parent, out_state, out_step, out_cum, st);
  return hipGetLastError();
}

// The streaming beam runs the one-wave-per-hypothesis kernel with the
// recombination and tree stages where that kernel applies (K <= 8, V+1 <=
// 2048, override sets within its lists), else the reference kernel's.
bool beam_stream_supported(int32_t v_plus_blank, int32_t max_override, int32_t K) {
  if (K < 1 || K > 8 || v_plus_blank < 2 || v_plus_blank > 64 * 32 || K > v_plus_blank)
    return false;
  return max_override <= beamk::kOverCap;
}

hipError_t launch_beam_stream(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int32_t K, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, float* scores, tb_hyp* hyps, int32_t* tree,
                              int32_t tree_cap, int32_t* tree_len, int32_t recombine,
                              int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                              float* out_step, float* out_cum, hipStream_t st) {
  beamk::StreamArgs sa;
  sa.hyps = hyps;
  sa.tree = tree;
  sa.cap = tree_cap;
  sa.tree_len = tree_len;
  sa.recombine = recombine;
  if (debug_beam_kernel() != kBeamRef && beam_stream_supported(A.V1, A.max_override, K)) {
    const int per = (A.V1 + 63) / 64;
    beamk::BeamStreamLaunch f = per <= 8    ? beamk::beam_stream_launcher_1_8(per, dtype)
                                : per <= 16 ? beamk::beam_stream_launcher_9_16(per, dtype)
                                : per <= 24 ? beamk::beam_stream_launcher_17_24(per, dtype)
                                            : beamk::beam_stream_launcher_25_32(per, dtype);
    if (f)
      return f(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok, out_parent,
               out_state, out_step, out_cum, st, sa);
  }
  // any other row width, beam or override set: the reference kernel's stage
  if (dtype == TB_F32)
    launch_k<LoadF32, true>(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok,
                            out_parent, out_state, out_step, out_cum, st, sa);
  else
    launch_k<LoadBF16, true>(A, logits, T, B, K, row_stride, model_ids, states, scores, out_tok,
                             out_parent, out_state, out_step, out_cum, st, sa);
  return hipGetLastError();
}

}  // namespace tbias
