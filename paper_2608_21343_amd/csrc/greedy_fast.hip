// Boosted greedy step, pipelined kernel for V+1 <= 64*PER (one workgroup per stream).
//
// The greedy decode of one stream is a chain: the state after step t depends
// on the token chosen at step t, which depends on the state. Everything that
// does not depend on the state is taken off that chain, and the state-
// dependent part is precomputed for the states the stream is likely in:
//
//  * 5 loader waves stream the logit rows (row t belongs to loader t % 5,
//    three rows in flight per loader) and compute per row the log-softmax
//    normaliser and the best root move r1 = argmax_v z[v] + psi[root move of
//    v] (ties to the lowest v, blank excluded) into a ring of row summaries in
//    LDS. The rows themselves stay in global memory (and L2), where the
//    evaluations below read the few logits they need.
//  * 10 compute waves evaluate the complete step from up to three predicted
//    states: x1 = the root-move target of r1 of the previous row (the carried
//    state itself at the first row of a call), x2 = the answer from x1 of the
//    previous row, x3 = the answer from x2 of the previous row. The outputs of
//    the x1 answer are written speculatively.
//  * One consumer wave (raised issue priority) walks the chain: in state x1
//    the step is a compare (its outputs are already written); in x2 or x3 it
//    writes that answer; otherwise it evaluates the step itself.
//
// Evaluating a step from state x (the suffix-link traversal of the boosting
// graph): the children of x, link(x), ... (excluding the root) override the
// root move of their class, deeper states first; a wave-local LDS table of
// 8-bit tags marks the classes already claimed. The candidates are every
// override class (its best case variant in the row), the best root move whose
// class is not overridden, and the blank (z[V] + phi[x]); the largest key
// wins, ties to the lowest token id. The records of the first states
// (breadth-first ids, so the shallow ones) are cached in LDS for long calls.
//
// LDS is a static struct sized by the template (all addressing constant
// offset). Waves hand rows over through per-slot flags holding the row index,
// written after the data they guard and read before it. Every wait is
// bounded; on exhaustion the stream's outputs are marked with state -3.
#include <climits>

#include "device.hpp"
#include "launch.hpp"

namespace tbias {

namespace {

constexpr int kWaves = 16;                // wave 0 consumer, 1..5 loaders, 6..15 computers
constexpr int kConsumerAhead = 4;         // summaries the consumer keeps in flight
constexpr int kLoaders = 5;
constexpr int kLoadDepth = 3;             // rows in flight per loader (vmcnt budget)
constexpr int kComputers = kWaves - 1 - kLoaders;
constexpr int kThreads = 64 * kWaves;
constexpr uint32_t kSpinLimit = 1u << 24;
constexpr int32_t kStateTimeout = -3;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
// states cached in LDS (ids < HOT): smaller for the largest rows to fit 160 KB
constexpr int hot_states(int per) { return per <= 17 ? 4096 : 2048; }
constexpr int32_t kHotMinT = 64;          // shorter calls read the graph from global memory

typedef int32_t v4i __attribute__((ext_vector_type(4)));

// One row's summary. `ready` (row index) is written after everything else
// and read before it.
struct alignas(16) RowSum {
  v4i c0;  // ready, x1, ns1, x2
  v4i c1;  // ns2, tok2, b2, zv2
  v4i c2;  // x3, ns3, tok3, b3
  v4i c3;  // zv3, lse, zb, r1_tok
  v4i c4;  // r1_y, r1_dst, r1_cls, -
};

template <class TT, int PER, int NSLOT>
struct alignas(16) Lds {
  RowSum sum[NSLOT];
  int32_t ready[NSLOT];           // row whose summary is complete
  int32_t a_flag[NSLOT];          // row whose normaliser and r1 are published
  int32_t p1_flag[NSLOT];         // row whose x1 answer is published
  int32_t p2_flag[NSLOT];         // row whose x2 answer is published
  int32_t freed;                  // rows < freed may be overwritten
  int32_t abort_flag;
  float rpsi[64 * PER];           // psi of the root move; -inf for blank and padding
  int32_t rdst[64 * PER];         // target of the root move
  uint16_t cls[64 * PER];         // class of every token (0xffff: none)
  uint16_t cls_ptr[64 * PER + 4]; // members of class c: cls_tok[cls_ptr[c] .. cls_ptr[c+1])
  uint16_t cls_tok[64 * PER];
  uint8_t stamps[kWaves][64 * PER];
  // records of the first kHot states (breadth-first ids: the shallow ones)
  static constexpr int32_t kHot = hot_states(PER);
  int32_t hs_fc[kHot];            // first child
  uint32_t hs_lknc[kHot];         // link | n_child << 16
  float hs_phi[kHot];
  float hs_psi[kHot];
  uint16_t hs_label[kHot];
};

struct Answer {
  int32_t tok, ns;
  float b, zv;
};

// LDS hand-over primitives. Flags are relaxed workgroup-scope atomics and
// data are plain accesses, so that they compile to ds_read/ds_write: through
// a generic volatile pointer they would become flat accesses that wait for
// every outstanding global load of the wave. Ordering comes from the LDS
// executing one wave's accesses in order plus the waits below.
__device__ __forceinline__ void cbar() { asm volatile("" ::: "memory"); }
__device__ __forceinline__ void lds_fence() {
  // this wave's LDS writes are complete before anything after it is issued
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}
__device__ __forceinline__ int32_t vload(int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void vstore(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ v4i vload4(const v4i* p) {
  cbar();
  const v4i r = *p;
  cbar();
  return r;
}

// Spin until *p == want (or >= want when at_least), backing off so that
// waiting waves do not crowd the LDS queue. Returns false on abort/timeout.
__device__ bool wait_flag(int32_t* p, int32_t want, bool at_least, int32_t* abort_flag) {
  uint32_t n = 0;
  for (;;) {
    const int32_t v = vload(p);
    if (at_least ? (v >= want) : (v == want)) break;
    if (vload(abort_flag)) return false;
    if (++n > kSpinLimit) {
      vstore(abort_flag, 1);
      return false;
    }
    if (n < 4) {
      __builtin_amdgcn_s_sleep(1);
    } else if (n < 16) {
      __builtin_amdgcn_s_sleep(4);
    } else {
      __builtin_amdgcn_s_sleep(16);
    }
  }
  cbar();
  return true;
}

__device__ __forceinline__ int32_t rl(int32_t v, int32_t lane) {
  return __builtin_amdgcn_readlane(v, lane);
}
__device__ __forceinline__ float rlf(float v, int32_t lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// The boosted step from state x on logit row zrow (global memory), given that
// row's best root move. All lanes take part; the result is uniform.
template <class Ld, class L>
__device__ Answer eval_state(const ArenaView& A, int32_t off, L& S,
                             const typename Ld::T* __restrict__ zrow, int32_t x,
                             float zb, float r1_y, int32_t r1_tok, int32_t r1_dst, int32_t r1_cls,
                             int wave, uint32_t& tag, int32_t V, int32_t nhot) {
  const int lane = __lane_id();
  uint8_t* stamps = S.stamps[wave];
  if (++tag == 256u) {  // 8-bit tags: clear this wave's table on wrap
    uint32_t* w = reinterpret_cast<uint32_t*>(stamps);
    for (int32_t i = lane; i < (int32_t)sizeof(S.stamps[0]) / 4; i += 64) w[i] = 0u;
    tag = 1;
  }
  const uint8_t tg = (uint8_t)tag;
  const float phi_x = (x < nhot) ? S.hs_phi[x] : A.phi[off + x];

  float lk = kNegInf;
  int32_t lt = INT_MAX, lns = 0;
  float lpsi = 0.f;
  for (int32_t c = x; c != 0;) {
    int32_t fc, nc, lnk;
    if (c < nhot) {
      fc = S.hs_fc[c];
      const uint32_t ln = S.hs_lknc[c];
      lnk = (int32_t)(ln & 0xffffu);
      nc = (int32_t)(ln >> 16);
    } else {
      fc = A.first_child[off + c];
      nc = A.n_child[off + c];
      lnk = A.link[off + c];
    }
    const bool hot_kids = fc + nc <= nhot;
    for (int32_t j0 = 0; j0 < nc; j0 += 64) {
      const int32_t j = j0 + lane;
      if (j < nc) {
        const int32_t y = fc + j;
        const int32_t lab = hot_kids ? (int32_t)S.hs_label[y] : A.label[off + y];
        if (stamps[lab] != tg) {
          stamps[lab] = tg;
          const float py = hot_kids ? S.hs_psi[y] : A.psi[off + y];
          const int32_t m0 = S.cls_ptr[lab], m1 = S.cls_ptr[lab + 1];
          for (int32_t q = m0; q < m1; ++q) {
            const int32_t tok = S.cls_tok[q];
            const float k = Ld::get(zrow, tok) + py;
            if (better(k, tok, lk, lt)) { lk = k; lt = tok; lns = y; lpsi = py; }
          }
        }
      }
    }
    c = lnk;
  }
  float ok;
  int32_t ot;
  const int32_t wl = wave_argmax_dpp(lk, lt, ok, ot);
  const int32_t o_ns = rl(lns, wl);
  const float o_psi = rlf(lpsi, wl);

  // best root move whose class is not overridden
  float rk = r1_y;
  int32_t rt = r1_tok, r_ns = r1_dst;
  if (r1_cls >= 0 && stamps[r1_cls] == tg) {
    float k2 = kNegInf;
    int32_t t2 = INT_MAX, d2 = 0;
    for (int32_t v = lane; v < V; v += 64) {
      const int32_t c = S.cls[v];
      if (c != 0xffff && stamps[c] == tg) continue;
      const float k = Ld::get(zrow, v) + S.rpsi[v];
      if (better(k, v, k2, t2)) { k2 = k; t2 = v; d2 = S.rdst[v]; }
    }
    const int32_t l2 = wave_argmax_dpp(k2, t2, rk, rt);
    r_ns = rl(d2, l2);
  }
  Answer a;
  a.tok = V;
  a.ns = x;
  a.b = 0.f;
  a.zv = zb;
  float bk = zb + phi_x;  // blank keeps the state
  int32_t bt = V;
  if (better(ok, ot, bk, bt)) {
    bk = ok;
    bt = ot;
    a.tok = ot;
    a.ns = o_ns;
    a.b = o_psi - phi_x;
  }
  if (better(rk, rt, bk, bt)) {
    bk = rk;
    bt = rt;
    a.tok = rt;
    a.ns = r_ns;
    a.b = ((r_ns < nhot) ? S.hs_psi[r_ns] : A.psi[off + r_ns]) - phi_x;
  }
  if (a.tok != V) a.zv = Ld::get(zrow, a.tok);
  return a;
}

template <class Ld, int PER, int NSLOT>
__global__ __launch_bounds__(kThreads) void greedy_fast_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  typedef typename Ld::T TT;
  typedef Lds<TT, PER, NSLOT> L;
  __shared__ L S;
  const int32_t V1 = A.V1, V = V1 - 1;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int32_t b = blockIdx.x;

  const int32_t m = model_ids[b];
  const int32_t s0 = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s0, off, n);
  {
    const float* gpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
    const int32_t* gdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;
    for (int32_t i = threadIdx.x; i < 64 * PER; i += kThreads) {
      S.rpsi[i] = (i < V) ? (mode == 1 ? gpsi[i] : 0.f) : kNegInf;
      S.rdst[i] = (i < V && mode == 1) ? gdst[i] : 0;
      const int32_t c = (i < V1) ? A.class_map[i] : -1;
      S.cls[i] = c < 0 ? (uint16_t)0xffff : (uint16_t)c;
      S.cls_ptr[i] = (i < V1) ? (uint16_t)A.cls_ptr[i] : (uint16_t)0;
      S.cls_tok[i] = (i < V) ? (uint16_t)A.cls_tok[i] : (uint16_t)0;
    }
  }
  // hot graph records (long calls only: a short call would read more graph
  // than logits)
  const int32_t nhot = (mode == 1 && T >= kHotMinT) ? (n < L::kHot ? n : L::kHot) : 0;
  for (int32_t i = threadIdx.x; i < nhot; i += kThreads) {
    S.hs_fc[i] = A.first_child[off + i];
    S.hs_lknc[i] = (uint32_t)A.link[off + i] | ((uint32_t)A.n_child[off + i] << 16);
    S.hs_phi[i] = A.phi[off + i];
    S.hs_psi[i] = A.psi[off + i];
    S.hs_label[i] = (uint16_t)(A.label[off + i] < 0 ? 0 : A.label[off + i]);
  }
  for (int32_t i = threadIdx.x; i < NSLOT; i += kThreads) {
    S.sum[i].c0.x = -1;
    S.ready[i] = -1;
    S.a_flag[i] = -1;
    S.p1_flag[i] = -1;
    S.p2_flag[i] = -1;
  }
  if (threadIdx.x == 0) {
    S.freed = 0;
    S.abort_flag = 0;
  }
  for (int32_t i = threadIdx.x; i < (int32_t)sizeof(S.stamps) / 4; i += kThreads)
    reinterpret_cast<uint32_t*>(&S.stamps[0][0])[i] = 0u;
  __syncthreads();

  uint32_t tag = 0;

  if (wave == 0) {
    // ------------------------------------------------------------ consumer
    __builtin_amdgcn_s_setprio(3);
    // unbiased streams never leave their constant state
    int32_t s = (mode == 1) ? s0 : ((mode == 0) ? TB_STATE_NONE : TB_STATE_INVALID);
    bool ok = true;
    // summaries of the next kConsumerAhead rows: the ready flag is read
    // before the data, so a flag equal to the row index vouches for the data
    int32_t pf[kConsumerAhead];
    v4i pd[kConsumerAhead];
#pragma unroll
    for (int k = 0; k < kConsumerAhead; ++k) {
      pf[k] = vload(&S.ready[k % NSLOT]);
      cbar();
      pd[k] = S.sum[k % NSLOT].c0;
      cbar();
    }
    for (int32_t t0 = 0; t0 < T && ok; t0 += kConsumerAhead) {
#pragma unroll
      for (int k = 0; k < kConsumerAhead; ++k) {
        const int32_t t = t0 + k;
        if (t < T && ok) {
          const int32_t slot = t % NSLOT;
          uint32_t spins = 0;
          while (__builtin_amdgcn_readfirstlane(pf[k]) != t) {
            if (vload(&S.abort_flag) || ++spins > 64u * kSpinLimit) { ok = false; break; }
            pf[k] = vload(&S.ready[slot]);
            cbar();
            pd[k] = S.sum[slot].c0;
            cbar();
          }
          if (ok) {
            const int32_t x1 = __builtin_amdgcn_readfirstlane(pd[k].y);
            const int32_t ns1 = __builtin_amdgcn_readfirstlane(pd[k].z);
            const int32_t x2 = __builtin_amdgcn_readfirstlane(pd[k].w);
            // refill this prefetch slot with row t + kConsumerAhead
            const int32_t nslot = (t + kConsumerAhead) % NSLOT;
            pf[k] = vload(&S.ready[nslot]);
            cbar();
            pd[k] = S.sum[nslot].c0;
            cbar();
            if (s == x1 || mode != 1) {
              s = ns1;  // the x1 answer's outputs are already written
            } else {
              const RowSum& rs = S.sum[slot];
              const TT* zrow = logits + ((int64_t)t * B + b) * stride;
              const v4i c1 = rs.c1, c2 = rs.c2, c3 = rs.c3, c4 = rs.c4;
              const float lse = __int_as_float(__builtin_amdgcn_readfirstlane(c3.y));
              Answer a;
              if (s == x2) {
                a.ns = __builtin_amdgcn_readfirstlane(c1.x);
                a.tok = __builtin_amdgcn_readfirstlane(c1.y);
                a.b = __int_as_float(__builtin_amdgcn_readfirstlane(c1.z));
                a.zv = __int_as_float(__builtin_amdgcn_readfirstlane(c1.w));
              } else if (s == __builtin_amdgcn_readfirstlane(c2.x)) {
                a.ns = __builtin_amdgcn_readfirstlane(c2.y);
                a.tok = __builtin_amdgcn_readfirstlane(c2.z);
                a.b = __int_as_float(__builtin_amdgcn_readfirstlane(c2.w));
                a.zv = __int_as_float(__builtin_amdgcn_readfirstlane(c3.x));
              } else {
                a = eval_state<Ld>(A, off, S, zrow, s,
                                   __int_as_float(__builtin_amdgcn_readfirstlane(c3.z)),
                                   __int_as_float(__builtin_amdgcn_readfirstlane(c4.x)),
                                   __builtin_amdgcn_readfirstlane(c3.w),
                                   __builtin_amdgcn_readfirstlane(c4.y),
                                   __builtin_amdgcn_readfirstlane(c4.z), 0, tag, V, nhot);
              }
              if (lane == 0) {
                const int64_t oi = (int64_t)t * B + b;
                out_tok[oi] = a.tok;
                out_state[oi] = a.ns;
                out_score[oi] = (a.zv - lse) + a.b;
              }
              s = __builtin_amdgcn_readfirstlane(a.ns);
            }
            if (lane == 0) vstore(&S.freed, t);  // rows < t may be overwritten
          }
        }
      }
    }
    if (ok) {
      if (lane == 0 && T > 0) states[b] = s;
    } else {
      vstore(&S.abort_flag, 1);
      for (int32_t t = lane; t < T; t += 64) out_state[(int64_t)t * B + b] = kStateTimeout;
      if (lane == 0) states[b] = kStateTimeout;
    }
    return;
  }

  // ---------------------------------------------------------------- loaders
  if (wave <= kLoaders) {
    // rows t = li, li + kLoaders, ...; kLoadDepth rows in flight in registers
    const int li = wave - 1;
    float buf[kLoadDepth][PER];
    float rp[PER];  // root-move psi of this lane's tokens (-inf past V - 1)
#pragma unroll
    for (int j = 0; j < PER; ++j) rp[j] = S.rpsi[64 * j + lane];
    auto issue = [&](float* dst, int32_t tr) {
      const TT* row = logits + ((int64_t)tr * B + b) * stride;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int32_t v = 64 * j + lane;
        if (64 * (j + 1) <= V1) {  // uniform: the whole wave is inside the row
          dst[j] = Ld::get(row, v);
        } else {
          dst[j] = (v < V1) ? Ld::get(row, v) : kNegInf;
        }
      }
    };
#pragma unroll
    for (int k = 0; k < kLoadDepth; ++k) {
      const int32_t tr = li + k * kLoaders;
      if (tr < T) issue(buf[k], tr);
    }
    for (int32_t t0 = li; t0 < T; t0 += kLoadDepth * kLoaders) {
#pragma unroll
      for (int k = 0; k < kLoadDepth; ++k) {
        const int32_t t = t0 + k * kLoaders;
        if (t < T) {
          const int32_t slot = t % NSLOT;
          // the slot held row t - NSLOT: wait until the consumer is past row t - NSLOT + 1
          if (!wait_flag(&S.freed, t - NSLOT + 1, true, &S.abort_flag)) return;
          const float* cur = buf[k];
          // ---- normaliser and best root move (padding past V+1 is -inf)
          float ymax = kNegInf;
          float zb = 0.f;
#pragma unroll
          for (int j = 0; j < PER; ++j) {
            const float yj = cur[j] + rp[j];
            ymax = ymax > yj ? ymax : yj;
            if (j == (V >> 6)) zb = rlf(cur[j], V & 63);
          }
          ymax = wave_max_dpp(ymax);
          const float mref = ymax > zb ? ymax : zb;
          const float mL = mref * kLog2e;
          float se = 0.f;
#pragma unroll
          for (int j = 0; j < PER; ++j)
            se += __builtin_amdgcn_exp2f(__builtin_fmaf(cur[j], kLog2e, -mL));
          se = wave_sum_dpp(se);
          const float lse = mref + __logf(se);
          int32_t hit = INT_MAX;
#pragma unroll
          for (int j = PER - 1; j >= 0; --j) {
            const float yj = cur[j] + rp[j];
            hit = (yj == ymax) ? 64 * j + lane : hit;
          }
          int32_t r1_tok = wave_min_i32_dpp(hit);
          if (r1_tok >= V) r1_tok = 0;  // only with -inf / nan logits: keep indices in range
          const int32_t r1_dst = S.rdst[r1_tok];
          const int32_t c16 = S.cls[r1_tok];
          const int32_t r1_cls = (c16 == 0xffff) ? -1 : c16;
          RowSum& rs = S.sum[slot];
          if (lane == 0) {
            rs.c3.y = __float_as_int(lse);
            rs.c3.z = __float_as_int(zb);
            rs.c3.w = r1_tok;
            rs.c4 = v4i{__float_as_int(ymax), r1_dst, r1_cls, 0};
          }
          lds_fence();
          if (lane == 0) vstore(&S.a_flag[slot], t);
          const int32_t tn = t + kLoadDepth * kLoaders;
          if (tn < T) issue(buf[k], tn);
        }
      }
    }
    return;
  }

  // -------------------------------------------------------------- computers
  for (int32_t t = wave - 1 - kLoaders; t < T; t += kComputers) {
    const int32_t slot = t % NSLOT;
    if (!wait_flag(&S.a_flag[slot], t, false, &S.abort_flag)) return;
    RowSum& rs = S.sum[slot];
    const TT* zrow = logits + ((int64_t)t * B + b) * stride;
    const v4i c3 = rs.c3, c4 = rs.c4;
    const float lse = __int_as_float(__builtin_amdgcn_readfirstlane(c3.y));
    const float zb = __int_as_float(__builtin_amdgcn_readfirstlane(c3.z));
    const int32_t r1_tok = __builtin_amdgcn_readfirstlane(c3.w);
    const float ymax = __int_as_float(__builtin_amdgcn_readfirstlane(c4.x));
    const int32_t r1_dst = __builtin_amdgcn_readfirstlane(c4.y);
    const int32_t r1_cls = __builtin_amdgcn_readfirstlane(c4.z);

    int32_t x1, x2 = -4, x3 = -4;
    Answer a1;
    if (mode != 1) {
      // no biasing: the answer does not depend on the (constant) state
      const bool blank = !better(ymax, r1_tok, zb, V);
      x1 = (mode == 0) ? TB_STATE_NONE : TB_STATE_INVALID;
      a1.tok = blank ? V : r1_tok;
      a1.ns = x1;
      a1.b = 0.f;
      a1.zv = blank ? zb : ymax;
    } else {
      // ---- answer from x1 (the carried state at t = 0)
      if (t == 0) {
        x1 = s0;
      } else {
        const int32_t ps = (t - 1) % NSLOT;
        if (!wait_flag(&S.a_flag[ps], t - 1, false, &S.abort_flag)) return;
        x1 = __builtin_amdgcn_readfirstlane(S.sum[ps].c4.y);
      }
      a1 = eval_state<Ld>(A, off, S, zrow, x1, zb, ymax, r1_tok, r1_dst, r1_cls, wave, tag, V,
                          nhot);
    }
    if (lane == 0) {
      // speculative outputs: right whenever the stream is in x1 at step t
      const int64_t oi = (int64_t)t * B + b;
      out_tok[oi] = a1.tok;
      out_state[oi] = a1.ns;
      out_score[oi] = (a1.zv - lse) + a1.b;
      rs.c0.y = x1;
      rs.c0.z = a1.ns;
    }
    lds_fence();
    if (lane == 0) vstore(&S.p1_flag[slot], t);
    if (mode == 1) {
      // ---- answer from the previous row's x1 answer
      if (t > 0) {
        const int32_t ps = (t - 1) % NSLOT;
        if (!wait_flag(&S.p1_flag[ps], t - 1, false, &S.abort_flag)) return;
        x2 = __builtin_amdgcn_readfirstlane(S.sum[ps].c0.z);
      }
      int32_t ns2 = -4;
      if (x2 >= 0 && x2 != x1) {
        const Answer a2 =
            eval_state<Ld>(A, off, S, zrow, x2, zb, ymax, r1_tok, r1_dst, r1_cls, wave, tag, V,
                           nhot);
        ns2 = a2.ns;
        if (lane == 0) rs.c1 = v4i{a2.ns, a2.tok, __float_as_int(a2.b), __float_as_int(a2.zv)};
      } else {
        x2 = -4;
      }
      if (lane == 0) rs.c0.w = x2;
      if (lane == 0) rs.c4.w = ns2;
      lds_fence();
      if (lane == 0) vstore(&S.p2_flag[slot], t);
      // ---- answer from the previous row's x2 answer
      if (t > 0) {
        const int32_t ps = (t - 1) % NSLOT;
        if (!wait_flag(&S.p2_flag[ps], t - 1, false, &S.abort_flag)) return;
        x3 = __builtin_amdgcn_readfirstlane(S.sum[ps].c4.w);
      }
      if (x3 >= 0 && x3 != x1 && x3 != x2) {
        const Answer a3 =
            eval_state<Ld>(A, off, S, zrow, x3, zb, ymax, r1_tok, r1_dst, r1_cls, wave, tag, V,
                           nhot);
        if (lane == 0) {
          rs.c2 = v4i{x3, a3.ns, a3.tok, __float_as_int(a3.b)};
          rs.c3.x = __float_as_int(a3.zv);
        }
      } else if (lane == 0) {
        rs.c2.x = -4;
      }
    } else if (lane == 0) {
      rs.c0.w = -4;
      rs.c2.x = -4;
    }
    // the speculative outputs land before the row is published, so that a
    // correction by the consumer is ordered after them
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_fence();
    if (lane == 0) vstore(&S.ready[slot], t);  // publishes row t
    cbar();
  }
}

template <class Ld, int PER, int NSLOT>
hipError_t launch_fast(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                       int64_t stride, const int32_t* model_ids, int32_t* states,
                       int32_t* out_tok, int32_t* out_state, float* out_score, hipStream_t st) {
  typedef typename Ld::T TT;
  static_assert(sizeof(Lds<TT, PER, NSLOT>) <= 160 * 1024, "LDS budget");
  hipLaunchKernelGGL((greedy_fast_kernel<Ld, PER, NSLOT>), dim3(B), dim3(kThreads), 0, st, A,
                     static_cast<const TT*>(logits), T, B, stride, model_ids, states, out_tok,
                     out_state, out_score);
  return hipGetLastError();
}

}  // namespace

// Returns hipErrorNotSupported when the vocabulary is too large for this kernel.
hipError_t launch_greedy_fast(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, int32_t* out_tok, int32_t* out_state,
                              float* out_score, hipStream_t st) {
  const int32_t V1 = A.V1;
  if (V1 > 64 * 32 || V1 < 2) return hipErrorNotSupported;
#define TB_FAST(LD, P, NS)                                                                     \
  return launch_fast<LD, P, NS>(A, logits, T, B, row_stride, model_ids, states, out_tok,       \
                                out_state, out_score, st)
  if (dtype == TB_F32) {
    if (V1 <= 64 * 5) TB_FAST(LoadF32, 5, 64);
    if (V1 <= 64 * 17) TB_FAST(LoadF32, 17, 64);
    TB_FAST(LoadF32, 32, 64);
  } else {
    if (V1 <= 64 * 5) TB_FAST(LoadBF16, 5, 64);
    if (V1 <= 64 * 17) TB_FAST(LoadBF16, 17, 64);
    TB_FAST(LoadBF16, 32, 64);
  }
#undef TB_FAST
}

}  // namespace tbias
