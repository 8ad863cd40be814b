// Boosted greedy step, pipelined kernel for V+1 <= 64*PER (one workgroup per stream).
//
// The greedy decode of one stream is a chain: the state after step t depends
// on the token chosen at step t, which depends on the state. Everything that
// does not depend on the state is taken off that chain:
//
//  * 4 loader waves stream the logit rows into a ring of LDS slots (row t
//    belongs to loader t % 4, three rows in flight per loader, non-temporal
//    loads); loaders issue no other memory traffic, so nothing waits behind
//    their loads.
//  * 11 compute waves take the rows from LDS and compute per row the
//    log-softmax normaliser and the best root move
//    r1 = argmax_v z[v] + psi[root move of v] (ties to the lowest v, blank
//    excluded).
//  * They also evaluate the complete step from two predicted states and store
//    both answers: x1 = the root-move target of r1 of the previous row, and
//    x2 = the answer of the previous row's x1 evaluation (at the first row of
//    a call x1 is the carried state itself). A stream that follows the best
//    root move, or did so one step earlier, is in one of these states.
//  * One consumer wave (raised issue priority) walks the chain: when the
//    stream's state is x1 or x2 the step is a compare and a select;
//    otherwise it evaluates the step itself with the same routine.
//
// Evaluating a step from state x (the suffix-link traversal of the boosting
// graph): the children of x, link(x), ... (excluding the root) override the
// root move of their class, deeper states first; a wave-local LDS table of
// 8-bit tags marks the classes already claimed. The candidates are every
// override class (its best case variant in the row), the best root move whose
// class is not overridden, and the blank (z[V] + phi[x]); the largest key
// wins, ties to the lowest token id.
//
// LDS is a static struct sized by the template (all addressing constant
// offset). Producers and consumer hand rows over through per-slot flags
// holding the row index. Every wait is bounded; on exhaustion the stream's
// outputs are marked with state -3.
#include <climits>

#include "device.hpp"
#include "launch.hpp"

namespace tbias {

namespace {

constexpr int kWaves = 16;                // wave 0 consumer, 1..4 loaders, 5..15 computers
constexpr int kLoaders = 4;
constexpr int kLoadDepth = 3;             // rows in flight per loader (vmcnt budget)
constexpr int kComputers = kWaves - 1 - kLoaders;
constexpr int kThreads = 64 * kWaves;
constexpr uint32_t kSpinLimit = 1u << 24;
constexpr int32_t kStateTimeout = -3;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
// states cached in LDS (ids < HOT): smaller for the largest rows to fit 160 KB
constexpr int hot_states(int per) { return per <= 17 ? 2048 : 1024; }
constexpr int32_t kHotMinT = 64;          // shorter calls read the graph from global memory

typedef int32_t v4i __attribute__((ext_vector_type(4)));

// One row's summary. c0.x is the "fully ready" flag (row index); it is read
// first, so the chunks read after it are complete.
struct alignas(16) RowSum {
  v4i c0;  // ready, lse, zb, x1
  v4i c1;  // tok1, ns1, b1, zv1
  v4i c2;  // x2, tok2, ns2, b2
  v4i c3;  // zv2, r1_y, r1_tok, r1_dst
  v4i c4;  // r1_cls, -, -, -
};

template <class TT, int PER, int NSLOT>
struct alignas(16) Lds {
  TT z[NSLOT][64 * PER];          // logit rows (ring)
  RowSum sum[NSLOT];
  int32_t loaded[NSLOT];          // row whose logits are in the slot
  int32_t a_flag[NSLOT];          // row whose r1 is published
  int32_t p1_flag[NSLOT];         // row whose x1 answer is published
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

// The boosted step from state x on the row in `slot`, given that row's best
// root move. All lanes take part; the result is uniform.
template <class Ld, class L>
__device__ Answer eval_state(const ArenaView& A, int32_t off, L& S, int32_t slot, int32_t x,
                             float zb, float r1_y, int32_t r1_tok, int32_t r1_dst, int32_t r1_cls,
                             int wave, uint32_t& tag, int32_t V, int32_t nhot) {
  const int lane = __lane_id();
  const auto* zrow = S.z[slot];
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
    S.loaded[i] = -1;
    S.a_flag[i] = -1;
    S.p1_flag[i] = -1;
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
    int32_t s = s0;
    bool ok = true;
    int32_t o_tok = 0, o_st = 0;
    float o_sc = 0.f;
    v4i c0 = vload4(&S.sum[0].c0);
    v4i c1 = S.sum[0].c1, c2 = S.sum[0].c2;
    for (int32_t t = 0; t < T; ++t) {
      const int32_t slot = t % NSLOT;
      uint32_t spins = 0;
      while (__builtin_amdgcn_readfirstlane(c0.x) != t) {
        if (vload(&S.abort_flag) || ++spins > 64u * kSpinLimit) { ok = false; break; }
        c0 = vload4(&S.sum[slot].c0);
        c1 = S.sum[slot].c1;
        c2 = S.sum[slot].c2;
      }
      if (!ok) break;
      // the summary is uniform: move it to scalar registers
      const float lse = __int_as_float(__builtin_amdgcn_readfirstlane(c0.y));
      const float zb = __int_as_float(__builtin_amdgcn_readfirstlane(c0.z));
      const int32_t x1 = __builtin_amdgcn_readfirstlane(c0.w);
      const int32_t x2 = __builtin_amdgcn_readfirstlane(c2.x);
      const v4i h1 = c1, h2 = c2;
      // prefetch the next row's summary (checked at the top of the next step)
      const int32_t nslot = (t + 1) % NSLOT;
      c0 = vload4(&S.sum[nslot].c0);
      c1 = S.sum[nslot].c1;
      c2 = S.sum[nslot].c2;
      Answer a;
      if (s == x1) {
        a.tok = __builtin_amdgcn_readfirstlane(h1.x);
        a.ns = __builtin_amdgcn_readfirstlane(h1.y);
        a.b = __int_as_float(__builtin_amdgcn_readfirstlane(h1.z));
        a.zv = __int_as_float(__builtin_amdgcn_readfirstlane(h1.w));
      } else if (s == x2) {
        a.tok = __builtin_amdgcn_readfirstlane(h2.y);
        a.ns = __builtin_amdgcn_readfirstlane(h2.z);
        a.b = __int_as_float(__builtin_amdgcn_readfirstlane(h2.w));
        a.zv = __int_as_float(__builtin_amdgcn_readfirstlane(S.sum[slot].c3.x));
      } else {
        const v4i c3 = S.sum[slot].c3;
        const int32_t r1_cls = __builtin_amdgcn_readfirstlane(S.sum[slot].c4.x);
        a = eval_state<Ld>(A, off, S, slot, s, zb, __int_as_float(__builtin_amdgcn_readfirstlane(c3.y)),
                           __builtin_amdgcn_readfirstlane(c3.z), __builtin_amdgcn_readfirstlane(c3.w),
                           r1_cls, 0, tag, V, nhot);
      }
      // lane (t % 64) keeps step t; one store per 64 steps
      const int32_t ln = t & 63;
      const float sc = (a.zv - lse) + a.b;
      const bool mine = lane == ln;
      o_tok = mine ? a.tok : o_tok;
      o_st = mine ? a.ns : o_st;
      o_sc = mine ? sc : o_sc;
      if (ln == 63 || t == T - 1) {
        if (lane <= ln) {
          const int64_t oi = (int64_t)(t - ln + lane) * B + b;
          out_tok[oi] = o_tok;
          out_state[oi] = o_st;
          out_score[oi] = o_sc;
        }
      }
      s = __builtin_amdgcn_readfirstlane(a.ns);
      if (lane == 0) vstore(&S.freed, t);  // rows < t may be overwritten
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
    auto issue = [&](float* dst, int32_t tr) {
      const TT* row = logits + ((int64_t)tr * B + b) * stride;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const int32_t v = 64 * j + lane;
        if (64 * (j + 1) <= V1) {  // uniform: the whole wave is inside the row
          dst[j] = Ld::get_nt(row, v);
        } else {
          dst[j] = (v < V1) ? Ld::get_nt(row, v) : kNegInf;
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
#pragma unroll
          for (int j = 0; j < PER; ++j) {
            const int32_t v = 64 * j + lane;
            if (sizeof(TT) == 4) {
              reinterpret_cast<float*>(S.z[slot])[v] = buf[k][j];
            } else {
              reinterpret_cast<uint16_t*>(S.z[slot])[v] =
                  (uint16_t)(__float_as_uint(buf[k][j]) >> 16);
            }
          }
          lds_fence();
          if (lane == 0) vstore(&S.loaded[slot], t);
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
    if (!wait_flag(&S.loaded[slot], t, false, &S.abort_flag)) return;

    // ---- normaliser and best root move of row t
    constexpr bool kKeepY = PER <= 17;  // larger rows recompute y to stay within 128 VGPRs
    // the loaders pad every slot past V+1 with -inf, and rpsi is -inf past
    // V - 1, so the whole 64*PER range is read without guards
    float cur[PER];
    float y[kKeepY ? PER : 1];
    float ymax = kNegInf;
    const float zb = Ld::get(S.z[slot], V);
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int32_t v = 64 * j + lane;
      cur[j] = Ld::get(S.z[slot], v);
      const float yj = cur[j] + S.rpsi[v];
      if (kKeepY) y[kKeepY ? j : 0] = yj;
      ymax = ymax > yj ? ymax : yj;
    }
    ymax = wave_max_dpp(ymax);
    const float mref = ymax > zb ? ymax : zb;
    const float mL = mref * kLog2e;
    float se = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j) se += __builtin_amdgcn_exp2f(__builtin_fmaf(cur[j], kLog2e, -mL));
    se = wave_sum_dpp(se);
    const float lse = mref + __logf(se);
    // lowest token whose root key equals ymax: per-lane first hit, then a wave min
    int32_t hit = INT_MAX;
#pragma unroll
    for (int j = PER - 1; j >= 0; --j) {
      const float yj = kKeepY ? y[kKeepY ? j : 0] : cur[j] + S.rpsi[64 * j + lane];
      hit = (yj == ymax) ? 64 * j + lane : hit;
    }
    int32_t r1_tok = wave_min_i32_dpp(hit);
    if (r1_tok >= V) r1_tok = 0;  // only with -inf / nan logits: keep indices in range
    const int32_t r1_dst = S.rdst[r1_tok];
    const int32_t c16 = S.cls[r1_tok];
    const int32_t r1_cls = (c16 == 0xffff) ? -1 : c16;
    RowSum& rs = S.sum[slot];
    if (lane == 0) {
      rs.c3.y = __float_as_int(ymax);
      rs.c3.z = r1_tok;
      rs.c3.w = r1_dst;
      rs.c4.x = r1_cls;
    }
    lds_fence();
    if (lane == 0) vstore(&S.a_flag[slot], t);

    v4i c0 = v4i{t, __float_as_int(lse), __float_as_int(zb), -4};
    if (mode != 1) {
      // no biasing: the answer does not depend on the (constant) state
      const bool blank = !better(ymax, r1_tok, zb, V);
      const int32_t st = (mode == 0) ? TB_STATE_NONE : TB_STATE_INVALID;
      if (lane == 0)
        rs.c1 = v4i{blank ? V : r1_tok, st, 0, __float_as_int(blank ? zb : ymax)};
      c0.w = st;
    } else {
      // ---- answer from x1 (the carried state at t = 0)
      int32_t x1;
      if (t == 0) {
        x1 = s0;
      } else {
        const int32_t ps = (t - 1) % NSLOT;
        if (!wait_flag(&S.a_flag[ps], t - 1, false, &S.abort_flag)) return;
        x1 = S.sum[ps].c3.w;
      }
      x1 = __builtin_amdgcn_readfirstlane(x1);
      const Answer a1 =
          eval_state<Ld>(A, off, S, slot, x1, zb, ymax, r1_tok, r1_dst, r1_cls, wave, tag, V, nhot);
      if (lane == 0) rs.c1 = v4i{a1.tok, a1.ns, __float_as_int(a1.b), __float_as_int(a1.zv)};
      lds_fence();
      if (lane == 0) vstore(&S.p1_flag[slot], t);
      // ---- answer from the previous row's x1 answer
      int32_t x2 = -4;
      if (t > 0) {
        const int32_t ps = (t - 1) % NSLOT;
        if (!wait_flag(&S.p1_flag[ps], t - 1, false, &S.abort_flag)) return;
        x2 = S.sum[ps].c1.y;
      }
      x2 = __builtin_amdgcn_readfirstlane(x2);
      Answer a2 = a1;
      if (x2 >= 0 && x2 != x1) {
        a2 = eval_state<Ld>(A, off, S, slot, x2, zb, ymax, r1_tok, r1_dst, r1_cls, wave, tag, V, nhot);
      } else {
        x2 = -4;
      }
      if (lane == 0) {
        rs.c2 = v4i{x2, a2.tok, a2.ns, __float_as_int(a2.b)};
        rs.c3.x = __float_as_int(a2.zv);
      }
      c0.w = x1;
    }
    lds_fence();
    if (lane == 0) rs.c0 = c0;  // publishes row t
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
    if (V1 <= 64 * 5) TB_FAST(LoadF32, 5, 16);
    if (V1 <= 64 * 17) TB_FAST(LoadF32, 17, 16);
    TB_FAST(LoadF32, 32, 8);
  } else {
    if (V1 <= 64 * 5) TB_FAST(LoadBF16, 5, 16);
    if (V1 <= 64 * 17) TB_FAST(LoadBF16, 17, 16);
    TB_FAST(LoadBF16, 32, 16);
  }
#undef TB_FAST
}

}  // namespace tbias
