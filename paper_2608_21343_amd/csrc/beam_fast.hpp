// Boosted beam step for V+1 <= 64*PER: a row-preparation kernel over every
// row of the call, then one workgroup per stream with one wave per
// hypothesis (templates; instantiated per chunk count in beam_fast_*.hip).
//
// Part of a beam step does not depend on the hypotheses: a slot reads its own
// row [t, b, k] whatever the selection was, so the row's normaliser and its
// best root moves can be taken for every row of the call at once, on every
// CU, before the sequential part starts. beam_prep_kernel does that, one wave
// per row:
//
//  * the normaliser: max in float32, sum of exponentials and log in float64,
//    rounded once to float32 (beam scores are carried and compared, so they
//    follow the exact reading);
//  * the kList best root moves y = z + psi(root move) of the row in (y
//    descending, token ascending) order, over every token of the row (the
//    root-move psi of the stream's model; zero for unbiased streams).
//
// It stores them in the call's own output rows of that (t, b, k): out_step
// holds the normaliser and out_tok, out_parent, out_state and out_cum two
// 16-bit token ids each. The step kernel reads a row's entries one step ahead
// (wave k reads only row k, and writes row k's outputs afterwards), so the
// call needs no workspace.
//
// Per step, wave k takes hypothesis k:
//
//  * c_k = (S_k - lse_k) - phi(s_k), and the candidates c_k + key over the row:
//    root moves z + psi(root move) from registers (tokens whose class is
//    overridden in s_k excluded through a class-mark table), the override
//    members of the classes of the children along s_k's suffix chain (deepest
//    state first) listed in LDS, and the blank c_k + z[V] + phi(s_k);
//  * the K best of all K*(V+1) candidates (larger first, ties to the lower
//    flat index k*(V+1)+v): the listed root moves of every slot whose class
//    is not overridden are real candidates, so the K-th largest of them,
//    theta, bounds the K-th best from below; every candidate >= theta is
//    compacted into LDS and ranked exactly. When fewer than K listed moves
//    remain, or too many candidates reach theta, K rounds of a workgroup
//    argmax select the K best instead;
//  * slot j takes the j-th best: its parent, token, advanced state (blank
//    keeps it), step score (z - lse) + boost and cumulative score.
//
// Graph records: every state of the model (up to the LDS budget) as a packed
// 12-byte record with the model's psi and phi value tables in LDS, so the
// sequential part of a step reads no arena memory.
#pragma once

#include <climits>

#include "device.hpp"
#include "greedy_seg.hpp"

namespace tbias {
namespace beamk {

using seg::kNegInf;
using seg::RowShape;
using seg::StateHot;
using seg::Tables;

constexpr int kOverCap = 256;  // override members listed per hypothesis
constexpr int kCandCap = 64;   // candidates compacted for the final selection (one per lane)
constexpr int kList = 8;       // best root moves listed per row by beam_prep_kernel
constexpr int kPrepThreads = 256;
constexpr uint32_t kNoTok = 0xffffu;

// SK: MAXK for the streaming beam, 1 (fields unused) otherwise.
template <int PER, int MAXK, int SK>
struct alignas(16) BeamFixed {
  Tables<PER> tab;
  float zbuf[MAXK][64 * PER];  // row of every hypothesis
  uint8_t stamps[MAXK][64 * PER];
  // override candidates of hypothesis k (the streaming beam appends its
  // merged candidates: up to SK - 1 more)
  float ov_val[MAXK][kOverCap + SK - 1];
  int32_t ov_tok[MAXK][kOverCap + SK - 1];
  int32_t ov_dst[MAXK][kOverCap + SK - 1];
  float cand_val[kCandCap];
  int32_t cand_f[kCandCap];
  int32_t cand_dst[kCandCap];
  int32_t hyp_s[2][MAXK];  // states and scores of the hypotheses, double buffered
  float hyp_S[2][MAXK];
  float hyp_lse[MAXK];
  float hyp_phi[MAXK];
  float listed[MAXK * kList];  // candidates of every slot's listed root moves
  int32_t cnt_w[MAXK];
  float sel_val[MAXK];
  int32_t sel_f[MAXK];
  int32_t sel_dst[MAXK];
  float red_val[MAXK];
  int32_t red_f[MAXK];
  int32_t red_dst[MAXK];
  // streaming beam (tb_boost_step_beam_stream): hypothesis carry, double
  // buffered, and the listed tokens
  uint64_t hyp_h[2][SK], hyp_hp[2][SK];
  int32_t hyp_lv[2][SK], hyp_node[2][SK];
  int32_t listed_tok[SK * kList];
};

// Carry of the streaming beam (tb_boost_step_beam_stream); unused otherwise.
struct StreamArgs {
  tb_hyp* hyps;        // [B*K]
  int32_t* tree;       // [B*cap*2] (label, parent record)
  int32_t cap;
  int32_t* tree_len;   // [B]
  int32_t recombine;
};

// log(exp(a) + exp(b)) of two finite float32 values, in float64, rounded once.
__device__ __forceinline__ float logaddexp32(float a, float b) {
  const double hi = (double)(a > b ? a : b), lo = (double)(a > b ? b : a);
  return (float)(hi + log1p(exp(lo - hi)));
}

template <int PER, int MAXK, int SK>
constexpr int beam_hot() {
  const int budget = 160 * 1024 - 1024;
  const int room = (budget - (int)sizeof(BeamFixed<PER, MAXK, SK>) - 2048) / seg::kStateHotBytes;
  const int h = (room / 64) * 64;
  return h > 8192 ? 8192 : (h < 0 ? 0 : h);
}

template <int PER, int MAXK, int SK = 1>
struct alignas(16) BeamLds : BeamFixed<PER, MAXK, SK> {
  static constexpr int HOT = beam_hot<PER, MAXK, SK>() > 64 ? beam_hot<PER, MAXK, SK>() : 64;
  StateHot<HOT> hot;
};

// Exclusive prefix sum over the lanes of a wave (lane i gets the sum of lanes
// < i) and the wave total: row shifts within rows of 16 lanes, then the gfx9
// row broadcasts; every lane of the wave must be active.
__device__ __forceinline__ int32_t wave_excl_scan(int32_t v, int32_t& total) {
  int32_t x = v;
  x += dpp_i<0x111, 0xf>(0, x);  // row_shr:1
  x += dpp_i<0x112, 0xf>(0, x);  // row_shr:2
  x += dpp_i<0x114, 0xf>(0, x);  // row_shr:4
  x += dpp_i<0x118, 0xf>(0, x);  // row_shr:8
  x += dpp_i<0x142, 0xa>(0, x);  // row_bcast:15 into rows 1 and 3
  x += dpp_i<0x143, 0xc>(0, x);  // row_bcast:31 into rows 2 and 3
  total = __builtin_amdgcn_readlane(x, 63);
  return x - v;
}

// (value, flat index) order of the selection: larger value, then lower index.
__device__ __forceinline__ bool cbetter(float a, int32_t fa, float b, int32_t fb) {
  return a > b || (a == b && fa < fb);
}

// Float order as unsigned integers (larger float, larger key; -0 below +0).
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float from_order_key(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

// The n-th largest lane value of the wave, counting equal values separately
// (n >= 1): bitwise search for the largest key t with at least n lanes >= t.
__device__ __forceinline__ float wave_nth_largest(float x, int32_t n) {
  const uint32_t k = order_key(x);
  uint32_t t = 0u;
#pragma unroll
  for (int bit = 31; bit >= 0; --bit) {
    const uint32_t c = t | (1u << bit);
    if ((int32_t)__builtin_popcountll(__ballot(k >= c)) >= n) t = c;
  }
  return from_order_key(t);
}

// The state-independent part of every beam row of a call (see above): one
// wave per row (t, b, k), rows in (t*B + b)*K + k order.
template <class Ld, int PER>
__global__ __launch_bounds__(kPrepThreads) void beam_prep_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int64_t r0, int64_t n_rows, int32_t B,
    int32_t K, int64_t stride, const int32_t* __restrict__ model_ids,
    const int32_t* __restrict__ states, int32_t* __restrict__ out_tok,
    int32_t* __restrict__ out_parent, int32_t* __restrict__ out_state,
    float* __restrict__ out_step, float* __restrict__ out_cum) {
  __shared__ float g_key[kPrepThreads / 64][64];
  __shared__ int32_t g_tok[kPrepThreads / 64][64];
  lds_poison(g_key, sizeof(g_key));
  lds_poison(g_tok, sizeof(g_tok));
  const int lane = __lane_id();
  const int64_t r = r0 + (int64_t)blockIdx.x * (kPrepThreads / 64) + (threadIdx.x >> 6);
  if (r >= n_rows) return;  // uniform per wave; no barrier follows
  const int32_t V1 = A.V1, V = V1 - 1;
  const int32_t b = (int32_t)((r / K) % B);
  // the step kernel's decision: biased when the model id and every carried
  // state of the stream are in range
  const int32_t m = model_ids[b];
  bool biased = m >= 0 && m < A.n_models;
  if (biased) {
    const int32_t n = A.model_n[m];
    const int32_t s = (lane < K) ? states[(int64_t)b * K + lane] : 0;
    biased = __ballot(s < 0 || s >= n) == 0ull;
  }
  const RowShape<PER> rs(V1);
  float z[PER];
  seg::load_row<Ld, PER>(z, logits + r * stride, rs);
  const float* gpsi = A.root_psi + (int64_t)(biased ? m : 0) * V1;

  // normaliser (as the one-wave-per-row kernels always took it)
  float zmax = kNegInf;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const float zj = (j < PER - 1 || rs.last_ok) ? z[j] : kNegInf;
    zmax = __builtin_fmaxf(zmax, zj);
  }
  zmax = wave_max_dpp(zmax);
  double se = 0.0;
  const double zmd = (double)zmax;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const bool ok = (j < PER - 1) || rs.last_ok;
    se += ok ? exp_nonpos((double)z[j] - zmd) : 0.0;
  }
  se = wave_sum_d(se);
  const float lse = (float)(zmd + log(se));

  // root-move keys, then the kList best in (key, token) order
  float y[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int32_t v = (j < PER - 1) ? 64 * j + lane : rs.last_idx;
    const bool ok = ((j < PER - 1) || rs.last_ok) && v < V;
    y[j] = ok ? z[j] + (biased ? gpsi[v] : 0.f) : kNegInf;
  }
  // theta: the kList-th largest lane maximum; kList lanes hold a move >= theta,
  // so every listed move is >= theta. The moves >= theta (few) are gathered
  // in LDS and ranked in (key, token) order.
  const int wv = threadIdx.x >> 6;
  float lm = kNegInf;
#pragma unroll
  for (int j = 0; j < PER; ++j) lm = __builtin_fmaxf(lm, y[j]);
  const float theta = wave_nth_largest(lm, kList);
  int32_t cnt = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) cnt += (theta > kNegInf && y[j] >= theta) ? 1 : 0;
  int32_t total;
  int32_t pos = wave_excl_scan(cnt, total);
  uint32_t words[kList / 2] = {0u, 0u, 0u, 0u};
  if (theta > kNegInf && total <= 64) {
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      if (y[j] >= theta) {
        g_key[wv][pos] = y[j];
        g_tok[wv][pos] = (j == PER - 1) ? rs.last_idx : 64 * j + lane;
        ++pos;
      }
    }
    __builtin_amdgcn_wave_barrier();
    const float ki = (lane < total) ? g_key[wv][lane] : kNegInf;
    const int32_t ti = (lane < total) ? g_tok[wv][lane] : INT_MAX;
    int32_t rank = 0;
    for (int32_t q = 0; q < total; ++q) {
      const float kq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ki), q));
      const int32_t tq = __builtin_amdgcn_readlane(ti, q);
      rank += (kq > ki || (kq == ki && tq < ti)) ? 1 : 0;
    }
#pragma unroll
    for (int i = 0; i < kList; ++i) {
      const uint64_t who = __ballot(lane < total && rank == i);
      const uint32_t tok =
          who ? (uint32_t)__builtin_amdgcn_readlane(ti, (int32_t)__builtin_ctzll(who)) : kNoTok;
      words[i >> 1] |= tok << (16 * (i & 1));
    }
  } else {
    // fewer than kList finite moves, or very many equal keys: kList rounds
    // of a wave argmax
    uint32_t taken = 0u;
#pragma unroll
    for (int i = 0; i < kList; ++i) {
      float bk = kNegInf;
      int32_t bj = -1;
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const bool gt = !((taken >> j) & 1u) && y[j] > bk;
        bk = gt ? y[j] : bk;
        bj = gt ? j : bj;
      }
      const int32_t idx = (bj < 0) ? INT_MAX : ((bj == PER - 1) ? rs.last_idx : 64 * bj + lane);
      float wk;
      int32_t wt;
      wave_argmax_dpp(bj < 0 ? kNegInf : bk, idx, wk, wt);
      const bool none = !(wk > kNegInf);
      if (!none && idx == wt) taken |= 1u << bj;
      const uint32_t tok = none ? kNoTok : (uint32_t)wt;
      words[i >> 1] |= tok << (16 * (i & 1));
    }
  }
  if (lane == 0) {
    out_step[r] = lse;
    out_tok[r] = (int32_t)words[0];
    out_parent[r] = (int32_t)words[1];
    out_state[r] = (int32_t)words[2];
    out_cum[r] = __uint_as_float(words[3]);
  }
}

template <class Ld, int PER, int MAXK, bool STREAM>
__global__ __launch_bounds__(64 * MAXK) void beam_fast_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int32_t K,
    int64_t stride, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    float* __restrict__ scores, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_parent,
    int32_t* __restrict__ out_state, float* __restrict__ out_step, float* __restrict__ out_cum,
    StreamArgs sa) {
  typedef BeamLds<PER, MAXK, STREAM ? MAXK : 1> Lds;
  constexpr int HOT = Lds::HOT;
  __shared__ Lds S;
  lds_poison(&S, sizeof(S));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int nt = (int)blockDim.x;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // hypothesis / slot
  const int lane = __lane_id();
  const int32_t b = blockIdx.x;
  const int64_t tstride = (int64_t)B * K * stride;  // row (t, b, w) = base + t * tstride
  const typename Ld::T* base = logits + ((int64_t)b * K + w) * stride;
  const int64_t ostride = (int64_t)B * K;  // output / row-summary entry (t, b, w) = o0 + t * ostride
  const int64_t o0 = (int64_t)b * K + w;

  const int32_t m = model_ids[b];
  int mode = (m == -1) ? 0 : ((m < -1 || m >= A.n_models) ? -1 : 1);
  int32_t off = 0, n = 0;
  if (mode == 1) {
    off = A.model_off[m];
    n = A.model_n[m];
  }
  // every wave reads the carried states and takes the same decision: a slot
  // out of range decodes the stream unbiased, before any table is filled
  const int32_t s_lane = (lane < K) ? states[(int64_t)b * K + lane] : 0;
  if (mode == 1 && __ballot(lane < K && (s_lane < 0 || s_lane >= n)) != 0ull) mode = -1;
  const bool tmo = __ballot(lane < K && s_lane == TB_STATE_TIMEOUT) != 0ull;
  if (threadIdx.x < K) {
    const int32_t s = s_lane;
    S.hyp_s[0][threadIdx.x] = s;
    S.hyp_S[0][threadIdx.x] = scores[(int64_t)b * K + threadIdx.x];
    if constexpr (STREAM) {
      const tb_hyp hy = sa.hyps[(int64_t)b * K + threadIdx.x];
      S.hyp_h[0][threadIdx.x] = hy.hash;
      S.hyp_hp[0][threadIdx.x] = hy.prefix_hash;
      S.hyp_lv[0][threadIdx.x] = hy.last;
      S.hyp_node[0][threadIdx.x] = hy.node;
    }
  }
  int32_t tlen = 0;  // tree records of this stream (streaming beam)
  if constexpr (STREAM) {
    const int32_t l = sa.tree_len[b];  // clamped: records are only written at [0, cap)
    tlen = l < 0 ? 0 : (l > sa.cap ? sa.cap : l);
  }
  const RowShape<PER> rs(V1);
  float cur[PER], nxt[PER];
  // row summary of this slot's row: normaliser and four words of listed tokens
  float lse_cur = 0.f, lse_nxt = 0.f;
  uint32_t lw_cur[kList / 2], lw_nxt[kList / 2];
  auto load_summary = [&](int32_t t, float& l, uint32_t* lw) {
    const int64_t o = o0 + (int64_t)t * ostride;
    l = out_step[o];
    lw[0] = (uint32_t)out_tok[o];
    lw[1] = (uint32_t)out_parent[o];
    lw[2] = (uint32_t)out_state[o];
    lw[3] = __float_as_uint(out_cum[o]);
  };
  if (T > 0) {
    seg::load_row<Ld, PER>(cur, base, rs);
    load_summary(0, lse_cur, lw_cur);
  }

  // tables: root row, class map and members; packed state records; marks
  {
    const int32_t mm = (mode == 1) ? m : 0;
    const float* gpsi = A.root_psi + (int64_t)mm * V1;
    const int32_t* gdst = A.root_dst + (int64_t)mm * V1;
    for (int32_t i = threadIdx.x; i < 64 * PER; i += nt) {
      S.tab.rpsi[i] = (i < V) ? (mode == 1 ? gpsi[i] : 0.f) : kNegInf;
      S.tab.rdst[i] = (i < V && mode == 1) ? gdst[i] : 0;
      const int32_t c = (i < V1) ? A.class_map[i] : -1;
      S.tab.cls[i] = c < 0 ? (uint16_t)0xffff : (uint16_t)c;
      S.tab.cls_ptr[i] = (i < V1) ? (uint16_t)A.cls_ptr[i] : (uint16_t)0;
      S.tab.cls_tok[i] = (i < V) ? (uint16_t)A.cls_tok[i] : (uint16_t)0;
    }
    const int32_t nhot0 = (mode == 1) ? (n < HOT ? n : HOT) : 0;
    const uint32_t* src = A.state_rec + 3 * (int64_t)off;
    for (int32_t i = threadIdx.x; i < nhot0; i += nt) {
      S.hot.w0[i] = src[3 * i];
      S.hot.w1[i] = src[3 * i + 1];
      S.hot.w2[i] = src[3 * i + 2];
    }
    if (nhot0 > 0) {
      const float* vt = A.value_tab + 512 * (int64_t)m;
      for (int32_t i = threadIdx.x; i < 512; i += nt) {
        if (i < 256) S.hot.vpsi[i] = vt[i];
        else S.hot.vphi[i - 256] = vt[i];
      }
    }
    for (int32_t i = threadIdx.x; i < MAXK * 16 * PER; i += nt)
      reinterpret_cast<uint32_t*>(&S.stamps[0][0])[i] = 0u;
  }
  __syncthreads();
  const int32_t nhot = (mode == 1) ? (n < HOT ? n : HOT) : 0;
  const seg::SGraph G(A, off, nhot, S.hot, S.tab);
  float* zrow = S.zbuf[w];
  uint8_t* stamps = S.stamps[w];
  uint32_t tag = 0;
  float rp[PER];
  uint32_t clsr[PER];  // class of every element of this lane (0xffff: none)
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) {
    rp[j] = S.tab.rpsi[64 * j + lane];
    clsr[j] = S.tab.cls[64 * j + lane];
  }
  rp[PER - 1] = rs.last_ok ? S.tab.rpsi[rs.last_idx] : kNegInf;
  clsr[PER - 1] = S.tab.cls[rs.last_idx];

  for (int32_t t = 0; t < T; ++t) {
    const int par = t & 1;
    {  // prefetch this slot's next row and its summary (the last ones are read again)
      const int32_t tn = (t + 1 < T) ? t + 1 : t;
      seg::load_row<Ld, PER>(nxt, base + (int64_t)tn * tstride, rs);
      load_summary(tn, lse_nxt, lw_nxt);
    }
    const int32_t s_k = __builtin_amdgcn_readfirstlane(S.hyp_s[par][w]);
    const float S_k = S.hyp_S[par][w];
    // streaming beam: bit 8x+y of pairs says that live slot y holds live slot
    // x's sequence without its last label (lane 8x+y tests it; every wave
    // forms the same mask); pair_lv on lane 8x is x's last label
    uint64_t pairs = 0ull;
    int32_t pair_lv = -1;
    if constexpr (STREAM) {
      static_assert(MAXK <= 8 && kList == 8, "pair mask layout: 8 slots, 8 listed moves");
      const int32_t x = lane >> 3, y = lane & 7;
      bool is_pair = false;
      if (sa.recombine && x < K && y < K) {
        pair_lv = S.hyp_lv[par][x];
        is_pair = x != y && pair_lv >= 0 && pair_lv < V && S.hyp_S[par][x] > kNegInf &&
                  S.hyp_S[par][y] > kNegInf && S.hyp_hp[par][x] == S.hyp_h[par][y];
      }
      pairs = __ballot(is_pair);
    }

    // ---- row to LDS; the normaliser comes from the row summary
#pragma unroll
    for (int j = 0; j < PER - 1; ++j) zrow[64 * j + lane] = cur[j];
    zrow[rs.last_idx] = cur[PER - 1];
    const float zb = seg::rlf(cur[PER - 1], PER > 1 ? 63 : V);
    const float lse = lse_cur;  // every lane loaded the same entry
    float phi_s = 0.f;
    int32_t fc_s = 0, nc_s = 0, lk_s = 0;  // s_k's record, for the listing below
    if (mode == 1) G.rec(s_k, fc_s, nc_s, lk_s, phi_s);
    const float c = (S_k - lse) - phi_s;
    if (lane == 0) {
      S.hyp_lse[w] = lse;
      S.hyp_phi[w] = phi_s;
    }

    // ---- override members of s_k (classes of the children along its suffix
    // chain, deepest state first), listed in LDS, their classes marked
    int32_t n_ov = 0;
    uint8_t tg = 0;
    if (mode == 1 && s_k != 0) {
      tg = seg::next_tag<PER>(stamps, tag);
      int32_t fc = fc_s, nc = nc_s, lnk = lk_s;
      float phi_unused;
      for (int32_t lvl = 0;; ++lvl) {
        for (int32_t j0 = 0; j0 < nc; j0 += 64) {
          const int32_t j = j0 + lane;
          int32_t y = fc, lab = 0, nm = 0, q0 = 0;
          uint2 mem = make_uint2(0u, 0u);
          float py = 0.f;
          bool take = false;
          if (j < nc) {
            y = fc + j;
            seg::child_rec(G, y, mem, py);
            lab = seg::arc_class(mem);
            take = lvl == 0 || stamps[lab] != tg;
            if (take) {
              stamps[lab] = tg;
              if (!seg::arc_more(mem)) {
                const uint32_t t0 = mem.x & 0xffffu, t1 = mem.x >> 16, t2 = mem.y & 0xffffu;
                nm = (t1 == t0) ? 1 : ((t2 == t1) ? 2 : 3);
              } else {
                q0 = S.tab.cls_ptr[lab];
                nm = S.tab.cls_ptr[lab + 1] - q0;
              }
            }
          }
          int32_t tot;
          const int32_t pos = n_ov + wave_excl_scan(nm, tot);
          for (int32_t i = 0; i < nm; ++i) {
            int32_t tok;
            if (!seg::arc_more(mem)) {
              tok = (int32_t)(i == 0 ? (mem.x & 0xffffu) : i == 1 ? (mem.x >> 16) : (mem.y & 0xffffu));
            } else {
              tok = S.tab.cls_tok[q0 + i];
            }
            if (pos + i < kOverCap) {
              S.ov_val[w][pos + i] = c + (zrow[tok] + py);
              S.ov_tok[w][pos + i] = tok;
              S.ov_dst[w][pos + i] = y;
            }
          }
          n_ov += tot;
        }
        if (lnk == 0) break;
        G.rec(lnk, fc, nc, lnk, phi_unused);
      }
    }
    // the launcher checks that the arena's largest override set fits the list
    n_ov = n_ov < kOverCap ? n_ov : kOverCap;
    uint32_t xm = 0u;  // bit j: this lane's element of chunk j is overridden
    if (n_ov > 0) {
#pragma unroll
      for (int j = 0; j < PER; ++j)
        xm |= (clsr[j] != 0xffffu && stamps[clsr[j]] == tg) ? (1u << j) : 0u;
    }

    // ---- the listed root moves of this row that are not overridden: real
    // candidates, hence lower bounds of the K-th best
    {
      float lv = kNegInf;
      if (lane < kList) {
        const uint32_t tok = (lw_cur[lane >> 1] >> (16 * (lane & 1))) & 0xffffu;
        if (tok != kNoTok && (int32_t)tok < V) {
          const uint32_t cl = S.tab.cls[tok];
          const bool over = n_ov > 0 && cl != 0xffffu && stamps[cl] == tg;
          if (!over) lv = c + (zrow[tok] + S.tab.rpsi[tok]);
        }
        S.listed[w * kList + lane] = lv;
        if constexpr (STREAM) S.listed_tok[w * kList + lane] = (int32_t)tok;
      }
    }

    // ---- candidates of this lane: dense root moves (unless overridden), the
    // lane's override entries and (lane 0) the blank
    float cb = c + (zb + phi_s);
    const int32_t fbase = w * V1;
    auto dense_val = [&](int j) -> float {
      const bool okl = (j < PER - 1) || rs.last_ok;
      const float v = c + (cur[j] + rp[j]);  // -inf for the blank and masked lanes
      return (okl && !((xm >> j) & 1u)) ? v : kNegInf;
    };
    auto dense_f = [&](int j) -> int32_t {
      return fbase + ((j < PER - 1) ? 64 * j + lane : rs.last_idx);
    };
    __syncthreads();
    // streaming beam: recombination. Two live slots x and y with
    // seq(y) = seq(x) without its last label v make one hypothesis of x's
    // blank extension and y's extension by v (state s_x). Both slots form the
    // pair from the rows in LDS and decide alike: the better in (value, flat
    // index) order keeps its place with the merged value, the other becomes
    // -inf. x updates its blank; y patches its candidate for v (an override
    // entry, or a new entry that masks the dense root move). A slot pairs
    // with its lowest-numbered prefix slot only.
    if constexpr (STREAM) {
      if (pairs != 0ull) {
        // the class marks of this step exist only when the walk listed
        // overrides (otherwise tg is stale)
        const int32_t n_walk = n_ov;
        struct Merge {
          float a, bv, merged;
          bool ok;
        };
        auto merge = [&](int32_t x, int32_t y) -> Merge {
          const int32_t s_x = __builtin_amdgcn_readfirstlane(S.hyp_s[par][x]);
          const int32_t v = __builtin_amdgcn_readlane(pair_lv, 8 * x);
          const float phi_x = S.hyp_phi[x], phi_y = S.hyp_phi[y];
          const float c_x = (S.hyp_S[par][x] - S.hyp_lse[x]) - phi_x;
          const float c_y = (S.hyp_S[par][y] - S.hyp_lse[y]) - phi_y;
          const float psi_x = (mode == 1) ? G.psi_of(s_x) : 0.f;
          Merge r;
          r.a = c_x + (S.zbuf[x][V] + phi_x);
          r.bv = c_y + (S.zbuf[y][v] + psi_x);
          r.ok = r.a > kNegInf && r.bv > kNegInf;
          r.merged = r.ok ? logaddexp32(r.a, r.bv) : kNegInf;
          return r;
        };
        const uint32_t row_w = (uint32_t)(pairs >> (8 * w)) & 0xffu;
        if (row_w != 0u) {  // this slot is x; its prefix slot is y
          const int32_t y = __builtin_ctz(row_w);
          const Merge r = merge(w, y);
          if (r.ok) {
            const int32_t v = __builtin_amdgcn_readlane(pair_lv, 8 * w);
            const bool keep_a = r.a > r.bv || (r.a == r.bv && w * V1 + V < y * V1 + v);
            cb = keep_a ? r.merged : kNegInf;
          }
        }
        for (int32_t x = 0; x < K; ++x) {  // this slot is y for every such x
          const uint32_t row_x = (uint32_t)(pairs >> (8 * x)) & 0xffu;
          if (row_x == 0u || __builtin_ctz(row_x) != w) continue;
          const Merge r = merge(x, w);
          if (!r.ok) continue;
          const int32_t v = __builtin_amdgcn_readlane(pair_lv, 8 * x);
          const bool keep_a = r.a > r.bv || (r.a == r.bv && x * V1 + V < w * V1 + v);
          const float nv = keep_a ? kNegInf : r.merged;
          const uint32_t cl = S.tab.cls[v];
          const bool over = n_walk > 0 && cl != 0xffffu && stamps[cl] == tg;
          if (over) {
            for (int32_t q = lane; q < n_walk; q += 64)
              if (S.ov_tok[w][q] == v) S.ov_val[w][q] = nv;
          } else {
            if (lane == 0) {
              S.ov_val[w][n_ov] = nv;
              S.ov_tok[w][n_ov] = v;
              S.ov_dst[w][n_ov] = (mode == 1) ? __builtin_amdgcn_readfirstlane(S.hyp_s[par][x]) : -1;
            }
            ++n_ov;
            const bool last = PER > 1 && v >= 64 * (PER - 1);
            const int32_t ol = last ? v - (V1 - 64) : (v & 63);
            const int32_t oj = last ? PER - 1 : (v >> 6);
            if (lane == ol) xm |= 1u << oj;
          }
        }
      }
    }
    // theta: the K-th largest listed candidate over all slots (for the
    // streaming beam without the listed moves that a merge may change)
    float lval = (lane < K * kList) ? S.listed[lane] : kNegInf;
    if constexpr (STREAM) {
      if (pairs != 0ull && lane < K * kList) {
        const int32_t lk = lane / kList, ltok = S.listed_tok[lane];
        for (int32_t x = 0; x < K; ++x)
          if (((pairs >> (8 * x + lk)) & 1ull) && __builtin_amdgcn_readlane(pair_lv, 8 * x) == ltok)
            lval = kNegInf;
      }
    }
    const float theta = wave_nth_largest(lval, K);

    // count every candidate >= theta, keeping a lane's first two in registers
    int32_t mine = 0;
    float kv0 = kNegInf, kv1 = kNegInf;
    int32_t kf0 = 0, kf1 = 0, kd0 = -1, kd1 = -1;
#define TB_KEEP(pass, v, f, d)                                       \
  {                                                                  \
    const bool p0_ = (pass) && mine == 0, p1_ = (pass) && mine == 1; \
    kv0 = p0_ ? (v) : kv0;                                           \
    kf0 = p0_ ? (f) : kf0;                                           \
    kd0 = p0_ ? (d) : kd0;                                           \
    kv1 = p1_ ? (v) : kv1;                                           \
    kf1 = p1_ ? (f) : kf1;                                           \
    kd1 = p1_ ? (d) : kd1;                                           \
    mine += (pass) ? 1 : 0;                                          \
  }
    if (theta > kNegInf) {
      TB_KEEP(lane == 0 && cb >= theta, cb, fbase + V, -1);
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const float v = dense_val(j);
        TB_KEEP(v >= theta, v, dense_f(j), -1);
      }
      for (int32_t i = lane; i < n_ov; i += 64) {
        const float v = S.ov_val[w][i];
        const int32_t tk = S.ov_tok[w][i], dd = S.ov_dst[w][i];
        TB_KEEP(v >= theta, v, fbase + tk, dd);
      }
    }
#undef TB_KEEP
    int32_t wtot;
    const int32_t wpre = wave_excl_scan(mine, wtot);
    if (lane == 0) S.cnt_w[w] = wtot;
    __syncthreads();
    int32_t total = 0, woff = 0;
    for (int k = 0; k < K; ++k) {
      const int32_t ck = S.cnt_w[k];
      woff += (k < w) ? ck : 0;
      total += ck;
    }
    // one candidate per lane below: at most 64 take the fast path
    const bool fast = theta > kNegInf && total <= 64;
    int32_t sel_f_w = 0, sel_dst_w = -1;  // slot w's selection (uniform)
    float sel_val_w = kNegInf;
    int32_t nb_before = 0, nb_total = 0;  // kept non-blank extensions (streaming beam)
    if (fast && __ballot(mine > 2) == 0ull) {
      // every lane's candidates are in its registers
      const int32_t p = woff + wpre;
      if (mine > 0) {
        S.cand_val[p] = kv0;
        S.cand_f[p] = kf0;
        S.cand_dst[p] = kd0;
      }
      if (mine > 1) {
        S.cand_val[p + 1] = kv1;
        S.cand_f[p + 1] = kf1;
        S.cand_dst[p + 1] = kd1;
      }
    } else if (fast) {
      int32_t p = woff + wpre;
      if (lane == 0 && cb >= theta) {
        S.cand_val[p] = cb;
        S.cand_f[p] = fbase + V;
        S.cand_dst[p] = -1;
        ++p;
      }
#pragma unroll
      for (int j = 0; j < PER; ++j) {
        const float v = dense_val(j);
        if (v >= theta) {
          S.cand_val[p] = v;
          S.cand_f[p] = dense_f(j);
          S.cand_dst[p] = -1;
          ++p;
        }
      }
      for (int32_t i = lane; i < n_ov; i += 64) {
        const float v = S.ov_val[w][i];
        if (v >= theta) {
          S.cand_val[p] = v;
          S.cand_f[p] = fbase + S.ov_tok[w][i];
          S.cand_dst[p] = S.ov_dst[w][i];
          ++p;
        }
      }
    }
    if (fast) {
      __syncthreads();
      // exact K best of the compacted candidates, ranked by every wave (one
      // candidate per lane): the rank of a candidate is the number of
      // candidates before it in (value, flat index) order, and flat indices
      // are distinct, so ranks are distinct; slot w takes rank w
      const bool in = lane < total;
      const float vi = in ? S.cand_val[lane] : kNegInf;
      const int32_t fi = in ? S.cand_f[lane] : INT_MAX;
      const int32_t di = in ? S.cand_dst[lane] : -1;
      int32_t rank = 0;
      for (int32_t q = 0; q < total; ++q) {
        const float vq = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vi), q));
        const int32_t fq = __builtin_amdgcn_readlane(fi, q);
        rank += cbetter(vq, fq, vi, fi) ? 1 : 0;
      }
      const uint64_t mine_lane = __ballot(in && rank == w);
      const int32_t wl = mine_lane ? (int32_t)__builtin_ctzll(mine_lane) : 0;
      sel_f_w = __builtin_amdgcn_readlane(fi, wl);
      sel_val_w = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(vi), wl));
      sel_dst_w = __builtin_amdgcn_readlane(di, wl);
      if constexpr (STREAM) {
        const bool nb = in && rank < K && fi - (fi / V1) * V1 != V;
        nb_before = (int32_t)__builtin_popcountll(__ballot(nb && rank < w));
        nb_total = (int32_t)__builtin_popcountll(__ballot(nb));
      }
    } else {
      // K rounds of a workgroup argmax over every candidate not yet taken
      for (int32_t j = 0; j < K; ++j) {
        float bv = kNegInf;
        int32_t bf = INT_MAX, bd = -1;
        auto offer = [&](float v, int32_t f, int32_t d) {
          for (int32_t q = 0; q < j; ++q)
            if (S.sel_f[q] == f) return;
          if (cbetter(v, f, bv, bf)) { bv = v; bf = f; bd = d; }
        };
        if (lane == 0) offer(cb, fbase + V, -1);
#pragma unroll
        for (int jj = 0; jj < PER; ++jj) offer(dense_val(jj), dense_f(jj), -1);
        for (int32_t i = lane; i < n_ov; i += 64)
          offer(S.ov_val[w][i], fbase + S.ov_tok[w][i], S.ov_dst[w][i]);
        float wv;
        int32_t wf;
        const int32_t wl = wave_argmax_dpp(bv, bf, wv, wf);
        const int32_t wd = __builtin_amdgcn_readlane(bd, wl);
        if (lane == 0) {
          S.red_val[w] = wv;
          S.red_f[w] = wf;
          S.red_dst[w] = wd;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
          float gv = S.red_val[0];
          int32_t gf = S.red_f[0], gd = S.red_dst[0];
          for (int k = 1; k < K; ++k)
            if (cbetter(S.red_val[k], S.red_f[k], gv, gf)) {
              gv = S.red_val[k];
              gf = S.red_f[k];
              gd = S.red_dst[k];
            }
          S.sel_val[j] = gv;
          S.sel_f[j] = gf;
          S.sel_dst[j] = gd;
        }
        __syncthreads();
      }
      sel_f_w = __builtin_amdgcn_readfirstlane(S.sel_f[w]);
      sel_val_w = S.sel_val[w];
      sel_dst_w = __builtin_amdgcn_readfirstlane(S.sel_dst[w]);
      if constexpr (STREAM) {
        for (int32_t q = 0; q < K; ++q) {
          int32_t fq = S.sel_f[q];
          if (fq < 0 || fq >= K * V1) fq = 0;
          const int32_t nb = (fq % V1 != V) ? 1 : 0;
          nb_before += (q < w) ? nb : 0;
          nb_total += nb;
        }
      }
    }

    // ---- slot w takes the w-th best
    {
      int32_t f = sel_f_w;
      if (f < 0 || f >= K * V1) f = 0;  // only reachable with nan logits
      const int32_t k = f / V1, v = f - k * V1;
      const int32_t sp = S.hyp_s[par][k];
      const float phi_k = S.hyp_phi[k];
      int32_t ns;
      float bst = 0.f;
      if (mode == 1) {
        if (v == V) {
          ns = sp;
        } else {
          const int32_t d = sel_dst_w;
          ns = (d >= 0) ? d : S.tab.rdst[v];
          bst = ((d >= 0) ? G.psi_of(ns) : S.tab.rpsi[v]) - phi_k;
        }
      } else {
        ns = unbiased_state(mode, tmo);
      }
      const float z = S.zbuf[k][v];
      const float val = sel_val_w;
      if constexpr (STREAM) {
        // the slot's hypothesis: the parent's, extended by v unless v is the
        // blank; kept non-blank extensions get tree records in slot order
        const int32_t before = nb_before;
        const uint64_t hk = S.hyp_h[par][k];
        uint64_t nh = hk, nhp = S.hyp_hp[par][k];
        int32_t nlv = S.hyp_lv[par][k], nnode = S.hyp_node[par][k];
        if (v != V) {
          const int32_t r = tlen + before;
          nhp = hk;
          nh = hk * (uint64_t)TB_HASH_MUL + (uint64_t)(v + 1);
          nlv = v;
          nnode = (r < sa.cap) ? r : -2;
          if (lane == 0 && r < sa.cap) {
            sa.tree[((int64_t)b * sa.cap + r) * 2] = v;
            sa.tree[((int64_t)b * sa.cap + r) * 2 + 1] = S.hyp_node[par][k];
          }
        }
        if (lane == 0) {
          S.hyp_h[par ^ 1][w] = nh;
          S.hyp_hp[par ^ 1][w] = nhp;
          S.hyp_lv[par ^ 1][w] = nlv;
          S.hyp_node[par ^ 1][w] = nnode;
        }
        tlen += nb_total;
      }
      if (lane == 0) {
        const int64_t o = o0 + (int64_t)t * ostride;
        out_tok[o] = v;
        out_parent[o] = k;
        out_state[o] = ns;
        out_step[o] = (z - S.hyp_lse[k]) + bst;
        out_cum[o] = val;
        S.hyp_s[par ^ 1][w] = ns;
        S.hyp_S[par ^ 1][w] = val;
      }
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) cur[j] = nxt[j];
    lse_cur = lse_nxt;
#pragma unroll
    for (int i = 0; i < kList / 2; ++i) lw_cur[i] = lw_nxt[i];
  }
  if (lane == 0 && T > 0) {
    states[(int64_t)b * K + w] = S.hyp_s[T & 1][w];
    scores[(int64_t)b * K + w] = S.hyp_S[T & 1][w];
    if constexpr (STREAM) {
      tb_hyp hy;
      hy.hash = S.hyp_h[T & 1][w];
      hy.prefix_hash = S.hyp_hp[T & 1][w];
      hy.last = S.hyp_lv[T & 1][w];
      hy.node = S.hyp_node[T & 1][w];
      sa.hyps[(int64_t)b * K + w] = hy;
      if (w == 0) sa.tree_len[b] = tlen < sa.cap ? tlen : sa.cap;
    }
  }
}

template <class Ld, int PER, int MAXK, bool STREAM>
hipError_t launch_beam_any(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                           int32_t K, int64_t stride, const int32_t* model_ids, int32_t* states,
                           float* scores, int32_t* out_tok, int32_t* out_parent,
                           int32_t* out_state, float* out_step, float* out_cum, hipStream_t st,
                           StreamArgs sa) {
  static_assert(sizeof(BeamLds<PER, MAXK, STREAM ? MAXK : 1>) <= 160 * 1024, "LDS budget");
  typedef typename Ld::T TT;
  // rows [r0, n_rows) in launches of at most 2^30 workgroups
  const int64_t n_rows = (int64_t)T * B * K;
  constexpr int64_t kRowsPerLaunch = (int64_t)(kPrepThreads / 64) << 30;
  for (int64_t r0 = 0; r0 < n_rows; r0 += kRowsPerLaunch) {
    const int64_t nr = (n_rows - r0 < kRowsPerLaunch) ? n_rows - r0 : kRowsPerLaunch;
    const int64_t blocks = (nr + kPrepThreads / 64 - 1) / (kPrepThreads / 64);
    hipLaunchKernelGGL((beam_prep_kernel<Ld, PER>), dim3((uint32_t)blocks), dim3(kPrepThreads),
                       0, st, A, static_cast<const TT*>(logits), r0, n_rows, B, K, stride,
                       model_ids, states, out_tok, out_parent, out_state, out_step, out_cum);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((beam_fast_kernel<Ld, PER, MAXK, STREAM>), dim3(B), dim3(64 * K), 0, st, A,
                     static_cast<const TT*>(logits), T, B, K, stride, model_ids, states, scores,
                     out_tok, out_parent, out_state, out_step, out_cum, sa);
  return hipGetLastError();
}

template <class Ld, int PER, int MAXK>
hipError_t launch_beam_fast_t(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                              int32_t K, int64_t stride, const int32_t* model_ids,
                              int32_t* states, float* scores, int32_t* out_tok,
                              int32_t* out_parent, int32_t* out_state, float* out_step,
                              float* out_cum, hipStream_t st) {
  return launch_beam_any<Ld, PER, MAXK, false>(A, logits, T, B, K, stride, model_ids, states,
                                               scores, out_tok, out_parent, out_state, out_step,
                                               out_cum, st, StreamArgs{});
}

template <class Ld, int PER>
hipError_t launch_beam_stream_t(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                                int32_t K, int64_t stride, const int32_t* model_ids,
                                int32_t* states, float* scores, int32_t* out_tok,
                                int32_t* out_parent, int32_t* out_state, float* out_step,
                                float* out_cum, hipStream_t st, StreamArgs sa) {
  return launch_beam_any<Ld, PER, 8, true>(A, logits, T, B, K, stride, model_ids, states,
                                           scores, out_tok, out_parent, out_state, out_step,
                                           out_cum, st, sa);
}

typedef hipError_t (*BeamLaunch)(const ArenaView&, const void*, int32_t, int32_t, int32_t,
                                 int64_t, const int32_t*, int32_t*, float*, int32_t*, int32_t*,
                                 int32_t*, float*, float*, hipStream_t);
typedef hipError_t (*BeamStreamLaunch)(const ArenaView&, const void*, int32_t, int32_t, int32_t,
                                       int64_t, const int32_t*, int32_t*, float*, int32_t*,
                                       int32_t*, int32_t*, float*, float*, hipStream_t,
                                       StreamArgs);
BeamStreamLaunch beam_stream_launcher_1_8(int per, int32_t dtype);
BeamStreamLaunch beam_stream_launcher_9_16(int per, int32_t dtype);
BeamStreamLaunch beam_stream_launcher_17_24(int per, int32_t dtype);
BeamStreamLaunch beam_stream_launcher_25_32(int per, int32_t dtype);
BeamLaunch beam_launcher_1_8(int per, int maxk, int32_t dtype);
BeamLaunch beam_launcher_9_16(int per, int maxk, int32_t dtype);
BeamLaunch beam_launcher_17_24(int per, int maxk, int32_t dtype);
BeamLaunch beam_launcher_25_32(int per, int maxk, int32_t dtype);

}  // namespace beamk
}  // namespace tbias
