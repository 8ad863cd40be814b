// Boosted beam step for wide rows (V+1 > 2048, K <= 4): a producer/consumer
// split inside one workgroup per stream (templates; instantiated in
// beam_pipe_f32.hip and beam_pipe_bf16.hip).
//
// Much of a step does not depend on the hypotheses' states: the logit row
// [t, b, k] a slot reads is fixed, and so are its normaliser and its root
// moves. Helper waves do that part one step ahead while the hypothesis waves
// score the current step, so only the state-dependent part stays on the
// sequential path. The workgroup has 4 hypothesis waves and 8 helper waves,
// two per slot, each owning half of the row:
//
//  * helper (k, h) stores its half of row [t+1, b, k] in an LDS ring of two
//    slots (its loads were issued a step earlier into registers) and
//    summarises it: the half's largest logit m_h, the float64 sum of
//    exp(z - m_h) over the half, and a list of its best root moves: every
//    lane keeps its four best keys z + psi(root move), the 32 best of those
//    256 are listed with logit, class, target and psi, and beta_h bounds
//    every root move of the half that is not listed (the best key a lane kept
//    but did not list, or a lane's fifth best);
//  * hypothesis wave k takes hypothesis k of step t. The normaliser is
//    lse_k = M + log(sum_h s_h exp(m_h - M)) with M = max(m_0, m_1), in
//    float64 and rounded once (the sum of exp(z - M) over the row, in another
//    order). c_k = (S_k - lse_k) - phi(s_k) plus the keys of the override
//    members along s_k's suffix chain (children of the chain states, deepest
//    first; an LDS class bitmap keeps the deepest), of the 64 listed root
//    moves whose class is not overridden and of the blank go into per-lane
//    lists; K rounds of a wave argmax give the hypothesis' K best. Every
//    unlisted root move has a candidate of at most c_k + max(beta_0, beta_1),
//    so the K best are exact when the K-th is larger; otherwise the wave
//    rescans the whole row (rare: most of the list overridden). A hypothesis
//    with score -inf has only -inf candidates: its K best are its K lowest
//    flat indices;
//  * after one workgroup barrier every hypothesis wave merges the K lists of
//    K (K rounds of a wave argmax over K*K records) and takes slot k: parent,
//    token, state (blank keeps it), step score (z - lse_k) + (psi - phi(s_k))
//    and cumulative score.
//
// One barrier per step orders both roles: a ring slot is rewritten only
// after the step that read it has passed the barrier, and the merge records
// are double buffered. States and scores are carried across calls
// (Sec. II-C).
#pragma once

#include <climits>

#include "device.hpp"
#include "launch.hpp"

namespace tbias {
namespace bpipe {

constexpr int kList = 32;    // root moves listed per half row
constexpr int kSlots = 4;    // hypotheses per stream (K <= kSlots)
constexpr int kHelpers = 8;  // two per slot
constexpr int kThreads = 64 * (kSlots + kHelpers);
constexpr float kNegInf = -__builtin_huge_valf();

struct alignas(16) HalfList {
  double se;  // sum of exp(z - m) over the half
  float m;    // largest logit of the half
  float beta;
  int32_t n, pad;
  float z[kList];
  uint32_t tc[kList];  // token | class << 16 (class 0xffff: unbiased stream)
  int32_t dst[kList];
  float psi[kList];
};

struct alignas(16) Rec {
  float c;
  int32_t f;  // flat index k * (V+1) + v
  int32_t dst;
  float step;
};

// A candidate in a lane's list.
struct Cand {
  float c;
  int32_t f, dst;
  float step;
};

template <class RT, int TPH>
struct alignas(16) PipeLds {
  RT rows[2][kSlots][128 * TPH];    // the ring: raw logit rows, -inf padded
  uint32_t marks[kSlots][4 * TPH];  // class bitmap of every hypothesis wave
  HalfList list[2][kSlots][2];
  Rec rec[2][kSlots * kSlots];
  int32_t hyp_s[kSlots];
  float hyp_S[kSlots];
  int32_t bad;
  int32_t tmo;  // a slot carried TB_STATE_TIMEOUT
};

template <class RT>
__device__ __forceinline__ RT neg_inf();
template <>
__device__ __forceinline__ float neg_inf<float>() { return kNegInf; }
template <>
__device__ __forceinline__ uint16_t neg_inf<uint16_t>() { return (uint16_t)0xff80u; }

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(uint16_t x) { return __uint_as_float(((uint32_t)x) << 16); }

template <class T>
__device__ __forceinline__ T sld(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}

// The row length and the lane id pass through empty asm statements where
// they bound or index the unrolled per-slot loops, so that the compiler
// keeps each bounds test and address at its use instead of hoisting one
// lane mask and one offset per slot out of the step loop.
__device__ __forceinline__ int32_t opaque(int32_t x) {
  asm volatile("" : "+s"(x));
  return x;
}
__device__ __forceinline__ int32_t opaque_v(int32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Barrier that waits for this wave's LDS operations only (global loads in
// flight stay in flight).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Monotone map of a float key to an unsigned integer.
__device__ __forceinline__ uint32_t ordered(float x) {
  const uint32_t b = __float_as_uint(x);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ __forceinline__ void list_clear(Cand (&l)[kSlots]) {
#pragma unroll
  for (int j = 0; j < kSlots; ++j) l[j] = Cand{kNegInf, INT_MAX, 0, 0.f};
}

__device__ __forceinline__ void list_insert(Cand (&l)[kSlots], const Cand& x) {
  if (!better(x.c, x.f, l[kSlots - 1].c, l[kSlots - 1].f)) return;
  l[kSlots - 1] = x;
#pragma unroll
  for (int j = kSlots - 1; j > 0; --j) {
    if (better(l[j].c, l[j].f, l[j - 1].c, l[j - 1].f)) {
      const Cand tmp = l[j];
      l[j] = l[j - 1];
      l[j - 1] = tmp;
    }
  }
}

__device__ __forceinline__ bool is_marked(const uint32_t* mk, int32_t c) {
  return (mk[c >> 5] >> (c & 31)) & 1u;
}

// What a hypothesis wave needs to score one hypothesis row.
template <class RT>
struct Hyp {
  const RT* zr;  // the row in the ring
  float lse, phi, ck;
  int32_t s, fbase;  // state, k * (V+1)
};

// Candidate of token t moved to state y with psi py.
template <class RT>
__device__ __forceinline__ void offer(Cand (&l)[kSlots], const Hyp<RT>& h, int32_t t, int32_t y,
                                      float py) {
  const float z = widen(h.zr[t]);
  const float key = z + py;
  list_insert(l, Cand{h.ck + key, h.fbase + t, y, (z - h.lse) + (py - h.phi)});
}

// The children of the states on s's suffix chain (root excluded), deepest
// first: a class already taken by a deeper state keeps that move. Marks the
// classes in mk (nw words, cleared first) and offers every member of every
// class.
template <class RT>
__device__ __forceinline__ void overrides(Cand (&l)[kSlots], const ArenaView& A, int32_t off,
                                          uint32_t* mk, int32_t nw, const Hyp<RT>& h) {
  const int lane = __lane_id();
  for (int i = lane; i < nw; i += 64) mk[i] = 0u;
  asm volatile("" ::: "memory");
  for (int32_t x = h.s; x != 0;) {
    const int32_t fc = sld(A.first_child + off + x);
    const int32_t nc = sld(A.n_child + off + x);
    const int32_t lk = sld(A.link + off + x);
    for (int32_t j = lane; j < nc; j += 64) {
      const int32_t y = fc + j;
      const int64_t q = 2 * ((int64_t)off + y);
      const uint32_t w0 = A.arc_mem[q], w1 = A.arc_mem[q + 1];
      const float py = A.psi[off + y];
      const int32_t c = (int32_t)((w1 >> 16) & 0x7fffu);
      if (!is_marked(mk, c)) {  // siblings have distinct classes
        atomicOr(mk + (c >> 5), 1u << (c & 31));
        if (!(w1 >> 31)) {  // up to three members, ascending (repeated when fewer)
          const int32_t t0 = (int32_t)(w0 & 0xffffu), t1 = (int32_t)(w0 >> 16);
          const int32_t t2 = (int32_t)(w1 & 0xffffu);
          offer<RT>(l, h, t0, y, py);
          if (t1 != t0) offer<RT>(l, h, t1, y, py);
          if (t2 != t1) offer<RT>(l, h, t2, y, py);
        } else {
          const int32_t q1 = A.cls_ptr[c + 1];
          for (int32_t p = A.cls_ptr[c]; p < q1; ++p) offer<RT>(l, h, A.cls_tok[p], y, py);
        }
      }
    }
    asm volatile("" ::: "memory");  // this level's marks before the next level's reads
    x = lk;
  }
}

// K rounds of a wave argmax over the lane lists; round j's winner goes to
// out[j] (lane 0 writes). Returns the K-th best.
__device__ __forceinline__ void take_best(Cand (&l)[kSlots], int32_t K, Rec* out, float& kc,
                                          int32_t& kf) {
  const int lane = __lane_id();
  kc = kNegInf;
  kf = INT_MAX;
  for (int32_t j = 0; j < K; ++j) {
    float bc;
    int32_t bf;
    const int32_t wl = wave_argmax_dpp(l[0].c, l[0].f, bc, bf);
    const int32_t dst = __builtin_amdgcn_readlane(l[0].dst, wl);
    const float step = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(l[0].step), wl));
    if (lane == wl) {
#pragma unroll
      for (int q = 0; q < kSlots - 1; ++q) l[q] = l[q + 1];
      l[kSlots - 1] = Cand{kNegInf, INT_MAX, 0, 0.f};
    }
    if (lane == 0) out[j] = Rec{bc, bf, dst, step};
    kc = bc;
    kf = bf;
  }
}

template <class Ld, int TPH>
__global__ __launch_bounds__(kThreads) void beam_pipe_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int32_t K,
    int64_t stride, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    float* __restrict__ scores, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_parent,
    int32_t* __restrict__ out_state, float* __restrict__ out_step, float* __restrict__ out_cum) {
  typedef typename Ld::T RT;
  constexpr int32_t HL = 64 * TPH;  // tokens per half row
  __shared__ PipeLds<RT, TPH> sh;
  lds_poison(&sh, sizeof(sh));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int lane = __lane_id();
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const bool helper = wave >= kSlots;
  const int hw = helper ? wave - kSlots : 0;
  const int k = helper ? hw >> 1 : wave;  // slot
  const int half = hw & 1;                // the helper's half of the row
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  int mode = (m == -1) ? 0 : 1;
  if (m < -1 || m >= A.n_models) mode = -1;
  int32_t off = 0, n = 0;
  if (mode == 1) {
    off = A.model_off[m];
    n = A.model_n[m];
  }
  if (threadIdx.x == 0) { sh.bad = 0; sh.tmo = 0; }
  __syncthreads();
  if ((int32_t)threadIdx.x < K) {
    const int32_t s = states[(int64_t)b * K + threadIdx.x];
    sh.hyp_s[threadIdx.x] = s;
    sh.hyp_S[threadIdx.x] = scores[(int64_t)b * K + threadIdx.x];
    if (mode == 1 && (s < 0 || s >= n)) sh.bad = 1;
    if (s == TB_STATE_TIMEOUT) sh.tmo = 1;
  }
  __syncthreads();
  if (mode == 1 && sh.bad) mode = -1;  // uniform: an invalid carried state decodes unbiased
  const int32_t fixed = unbiased_state(mode, sh.tmo != 0);
  const float* rpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* rdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;
  auto row_of = [&](int32_t t, int32_t kk) {
    return logits + (((int64_t)t * B + b) * K + kk) * stride;
  };

  // ---------------- helper: half a row, one step ahead ----------------
  RT raw[TPH];
  const int32_t hbase = half * HL;
  auto load_raw = [&](int32_t t) {
    const int32_t V1o = opaque(__builtin_amdgcn_readfirstlane(V1)), lo = opaque_v(lane);
    const RT* row = row_of(t, k);
#pragma unroll
    for (int j = 0; j < TPH; ++j) {
      const int32_t v = hbase + lo + 64 * j;
      raw[j] = (v < V1o) ? __builtin_nontemporal_load(row + v) : (RT)0;
    }
  };
  // The half's sum of exponentials about its largest logit mx, its root-move
  // list and bound (the half is in the ring, padded with -inf).
  auto summarise = [&](int32_t t, float mx) {
    const RT* zr = sh.rows[t & 1][k];
    const double Md = (double)mx;
    // One branch-free pass (exp_nonpos maps -inf to 0; the blank and the
    // padding have root psi -inf); root psi values are read in groups of kG
    // tokens, one group ahead.
    constexpr int kG = 4;
    auto load_rp = [&](int32_t g, float (&dst)[kG]) {
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        const int32_t v = hbase + lane + 64 * (g * kG + i);
        dst[i] = (g * kG + i < TPH && v < V) ? (mode == 1 ? rpsi[v] : 0.f) : kNegInf;
      }
    };
    float rpn[kG];
    load_rp(0, rpn);
    double se = 0.0;
    float k0 = kNegInf, k1 = kNegInf, k2 = kNegInf, k3 = kNegInf;
    int32_t v0 = INT_MAX, v1 = INT_MAX, v2 = INT_MAX, v3 = INT_MAX;
    float rest = kNegInf;
#pragma unroll 1
    for (int32_t g = 0; g * kG < TPH; ++g) {
      float rpc[kG], z[kG];
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        rpc[i] = rpn[i];
        const int32_t j = g * kG + i;
        z[i] = widen(zr[hbase + lane + 64 * (j < TPH ? j : TPH - 1)]);
      }
      if ((g + 1) * kG < TPH) load_rp(g + 1, rpn);
      double e[kG];
#pragma unroll
      for (int i = 0; i < kG; ++i) e[i] = exp_nonpos((double)z[i] - Md);
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        const bool in = g * kG + i < TPH;
        se += in ? e[i] : 0.0;
        const float key = in ? z[i] + rpc[i] : kNegInf;
        const int32_t v = hbase + lane + 64 * (g * kG + i);
        // insertion into the sorted four (tokens ascend: an equal key keeps
        // the earlier token)
        const bool g0 = key > k0, g1 = key > k1, g2 = key > k2, g3 = key > k3;
        rest = fmaxf(rest, g3 ? k3 : key);
        k3 = g2 ? k2 : (g3 ? key : k3);
        v3 = g2 ? v2 : (g3 ? v : v3);
        k2 = g1 ? k1 : (g2 ? key : k2);
        v2 = g1 ? v1 : (g2 ? v : v2);
        k1 = g0 ? k0 : (g1 ? key : k1);
        v1 = g0 ? v0 : (g1 ? v : v1);
        k0 = g0 ? key : k0;
        v0 = g0 ? v : v0;
      }
    }
    se = wave_sum_d(se);
    const float ek[4] = {k0, k1, k2, k3};
    const int32_t ev[4] = {v0, v1, v2, v3};
    // the kList-th largest of the 256 kept keys, bit by bit
    uint32_t u[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) u[q] = (ev[q] != INT_MAX) ? ordered(ek[q]) : 0u;
    uint32_t thr = 0u;
    for (int bit = 31; bit >= 0; --bit) {
      const uint32_t t2 = thr | (1u << bit);
      int32_t cnt = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) cnt += __builtin_popcountll(__ballot(u[q] >= t2));
      if (cnt >= kList) thr = t2;
    }
    HalfList& L = sh.list[t & 1][k][half];
    int32_t base = 0;
    int32_t pos[4];
    bool put[4];
    float unl = rest;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool valid = ev[q] != INT_MAX;
      const bool sel = valid && u[q] >= thr && u[q] != 0u;
      const uint64_t msk = __ballot(sel);
      pos[q] = base + (int32_t)__builtin_amdgcn_mbcnt_hi(
                          (uint32_t)(msk >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)msk, 0u));
      base += __builtin_popcountll(msk);
      put[q] = sel && pos[q] < kList;
      if (valid && !put[q]) unl = fmaxf(unl, ek[q]);
    }
    // the listed moves' logit, class, target and psi, read together
    int32_t cq[4], dq[4];
    float pq[4], zq[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int32_t v = put[q] ? ev[q] : 0;
      zq[q] = widen(zr[v]);
      cq[q] = (mode == 1) ? A.class_map[v] : -1;
      dq[q] = (mode == 1) ? rdst[v] : fixed;
      pq[q] = (mode == 1) ? rpsi[v] : 0.f;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (put[q]) {
        L.z[pos[q]] = zq[q];
        L.tc[pos[q]] = (uint32_t)ev[q] | ((uint32_t)(cq[q] < 0 ? 0xffff : cq[q]) << 16);
        L.dst[pos[q]] = dq[q];
        L.psi[pos[q]] = pq[q];
      }
    }
    unl = wave_max_dpp(unl);
    if (lane == 0) {
      L.se = se;
      L.m = mx;
      L.beta = unl;
      L.n = base < kList ? base : kList;
    }
  };
  // Stores the staged half of step t in the ring (padded with -inf),
  // summarises it, then issues the loads of step next (if next >= 0): loads
  // complete in issue order, so issuing them earlier would make the
  // summary's root psi reads wait for them.
  auto produce = [&](int32_t t, int32_t next) {
    const int32_t V1o = opaque(__builtin_amdgcn_readfirstlane(V1)), lo = opaque_v(lane);
    RT* zr = sh.rows[t & 1][k];
    float mx = kNegInf;
#pragma unroll
    for (int j = 0; j < TPH; ++j) {
      const int32_t v = hbase + lo + 64 * j;
      const RT x = (v < V1o) ? raw[j] : neg_inf<RT>();
      zr[v] = x;
      mx = fmaxf(mx, widen(x));
    }
    summarise(t, wave_max_dpp(mx));
    if (next >= 0) load_raw(next);
  };

  // ---------------- hypothesis wave ----------------
  int32_t s = 0;
  float S = 0.f;
  if (!helper && k < K) {
    s = __builtin_amdgcn_readfirstlane(sh.hyp_s[k]);
    S = sh.hyp_S[k];
  }
  uint32_t* mk = sh.marks[k];
  constexpr int32_t kMarkWords = 4 * TPH;
  auto consume = [&](int32_t t) {
    const HalfList& L0 = sh.list[t & 1][k][0];
    const HalfList& L1 = sh.list[t & 1][k][1];
    Hyp<RT> h;
    h.zr = sh.rows[t & 1][k];
    {
      const float M = fmaxf(L0.m, L1.m);
      const double Md = (double)M;
      const double St =
          L0.se * exp_nonpos((double)L0.m - Md) + L1.se * exp_nonpos((double)L1.m - Md);
      h.lse = (float)(Md + log(St));
    }
    h.phi = (mode == 1) ? sld(A.phi + off + s) : 0.f;
    h.ck = (S - h.lse) - h.phi;
    h.s = s;
    h.fbase = k * V1;
    const bool chain = mode == 1 && s != 0;
    const int32_t bdst = (mode == 1) ? s : fixed;
    Rec* out = sh.rec[t & 1] + k * K;
    float kc;
    int32_t kf;
    Cand l[kSlots];
    list_clear(l);
    if (chain) overrides<RT>(l, A, off, mk, kMarkWords, h);
    if (h.ck == kNegInf) {
      // Every candidate of this hypothesis is -inf (finite keys), so its K
      // best are the K lowest flat indices: tokens 0..K-1 (override members
      // among them are already offered), then the blank.
      if (lane < K) {
        const int32_t c = A.class_map[lane];
        if (!(chain && c >= 0 && is_marked(mk, c)))
          offer<RT>(l, h, lane, mode == 1 ? rdst[lane] : fixed, mode == 1 ? rpsi[lane] : 0.f);
      }
      if (lane == 0) offer<RT>(l, h, V, bdst, h.phi);
      take_best(l, K, out, kc, kf);
      return;
    }
    {
      const HalfList& L = lane < 32 ? L0 : L1;
      const int32_t e = lane & 31;
      if (e < L.n) {
        const uint32_t tc = L.tc[e];
        const int32_t c = (int32_t)(tc >> 16);
        if (!(chain && c != 0xffff && is_marked(mk, c))) {
          const float z = L.z[e], py = L.psi[e];
          const float key = z + py;
          list_insert(l, Cand{h.ck + key, h.fbase + (int32_t)(tc & 0xffffu), L.dst[e],
                              (z - h.lse) + (py - h.phi)});
        }
      }
    }
    if (lane == 0) offer<RT>(l, h, V, bdst, h.phi);  // the blank: key z + phi, no boost
    take_best(l, K, out, kc, kf);
    const float bound = h.ck + fmaxf(L0.beta, L1.beta);
    if (!(kc > bound)) {
      // rescan: every root move of the row, four tokens per lane at a time
      list_clear(l);
      if (chain) overrides<RT>(l, A, off, mk, kMarkWords, h);
      if (lane == 0) offer<RT>(l, h, V, bdst, h.phi);
      for (int32_t v0 = 0; v0 < V; v0 += 64 * 4) {
        int32_t cv[4], dv[4];
        float pv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int32_t v = v0 + lane + 64 * i;
          const int32_t vc = v < V ? v : 0;
          cv[i] = A.class_map[vc];
          dv[i] = mode == 1 ? rdst[vc] : fixed;
          pv[i] = mode == 1 ? rpsi[vc] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int32_t v = v0 + lane + 64 * i;
          if (v < V && !(chain && cv[i] >= 0 && is_marked(mk, cv[i])))
            offer<RT>(l, h, v, dv[i], pv[i]);
        }
      }
      take_best(l, K, out, kc, kf);
    }
  };

  if (T <= 0) return;
  if (helper && k < K) {
    load_raw(0);
    produce(0, T > 1 ? 1 : -1);
  }
  lds_barrier();
  for (int32_t t = 0; t < T; ++t) {
    if (!helper) {
      if (k < K) consume(t);
    } else if (k < K && t + 1 < T) {
      produce(t + 1, t + 2 < T ? t + 2 : -1);
    }
    lds_barrier();
    if (!helper && k < K) {
      const int32_t nr = K * K;
      Rec r = (lane < nr) ? sh.rec[t & 1][lane] : Rec{kNegInf, INT_MAX, 0, 0.f};
      float mc = 0.f, mstep = 0.f;
      int32_t mf = 0, mdst = 0;
      for (int32_t j = 0; j <= k; ++j) {
        float bc;
        int32_t bf;
        const int32_t wl = wave_argmax_dpp(r.c, r.f, bc, bf);
        if (j == k) {
          mc = bc;
          mf = bf;
          mdst = __builtin_amdgcn_readlane(r.dst, wl);
          mstep = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(r.step), wl));
        }
        if (lane == wl) {
          r.c = kNegInf;
          r.f = INT_MAX;
        }
      }
      if (lane == 0) {
        const int32_t f = (mf >= 0 && mf < K * V1) ? mf : 0;  // only with NaN logits
        const int32_t kp = f / V1, v = f - kp * V1;
        const int64_t oi = ((int64_t)t * B + b) * K + k;
        out_tok[oi] = v;
        out_parent[oi] = kp;
        out_state[oi] = mdst;
        out_step[oi] = mstep;
        out_cum[oi] = mc;
      }
      s = mdst;
      S = mc;
    }
  }
  if (!helper && k < K && lane == 0) {
    states[(int64_t)b * K + k] = s;
    scores[(int64_t)b * K + k] = S;
  }
}

template <class Ld, int TPH>
hipError_t launch_pipe_t(const ArenaView& A, const void* logits, int32_t T, int32_t B, int32_t K,
                         int64_t stride, const int32_t* model_ids, int32_t* states, float* scores,
                         int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                         float* out_step, float* out_cum, hipStream_t st) {
  hipLaunchKernelGGL((beam_pipe_kernel<Ld, TPH>), dim3(B), dim3(kThreads), 0, st, A,
                     static_cast<const typename Ld::T*>(logits), T, B, K, stride, model_ids,
                     states, scores, out_tok, out_parent, out_state, out_step, out_cum);
  return hipGetLastError();
}

typedef hipError_t (*PipeLaunch)(const ArenaView&, const void*, int32_t, int32_t, int32_t, int64_t,
                                 const int32_t*, int32_t*, float*, int32_t*, int32_t*, int32_t*,
                                 float*, float*, hipStream_t);

// Launcher for V+1 tokens and K hypotheses (nullptr when no instance fits:
// K > 4, V+1 <= 2048, or rows too long for the ring).
PipeLaunch pipe_launcher_f32(int32_t V1, int32_t K);
PipeLaunch pipe_launcher_bf16(int32_t V1, int32_t K);

}  // namespace bpipe
}  // namespace tbias
