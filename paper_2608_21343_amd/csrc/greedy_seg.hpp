// Boosted greedy step, segmented kernel (templates; instantiated per chunk
// count PER = ceil((V+1)/64) in greedy_seg_*.hip).
//
// The greedy decode of a stream is a chain (the state after step t depends on
// the token chosen at step t, which depends on the state), but the boosting
// automaton forgets where it started within a few steps: from most states the
// best move is a root move, after which every trajectory is in the same
// state. The T steps of a stream are therefore cut into segments that are
// decoded in parallel, one wave per segment:
//
//  * a segment that does not start the call begins kWarm rows early from the
//    root state (its guess); the segment at t = 0 starts from the carried
//    state, which is exact;
//  * each wave runs complete steps over its rows: the row (prefetched one
//    row ahead) is held in registers, z[64j + lane] in chunk j, and copied to
//    a wave-private LDS buffer; the log-softmax normaliser and the best root
//    move r1 = argmax_v z[v] + psi[root move of v] come from registers; then
//    the step from the current state is evaluated (the children of the
//    state's suffix chain override the root move of their class, deeper
//    states first; the blank keeps the state);
//  * after its rows, wave w compares its start state with the exact final
//    state of wave w-1 (handed over in LDS, in order along the segments). On a
//    mismatch it recomputes from the exact state until its trajectory meets
//    the stored one, after which all later outputs are already right;
//  * when a stream spans several workgroups, greedy_fix_kernel repairs the
//    workgroup boundaries the same way, in order, after the main kernel.
//
// Row layout in registers: chunks 0 .. PER-2 are full; the last chunk is read
// from element V+1-64 on (so every load is in bounds and unconditional) and
// its lanes that repeat elements of chunk PER-2 are masked to -inf. The blank
// logit z[V] is lane 63 of the last chunk.
//
// Per-wave LDS: the row and an 8-bit tag table marking the classes that are
// overridden in the state being evaluated. Shared LDS: the model's root row,
// the class tables and the records of the first (shallowest) states.
#pragma once

#include <climits>

#include "device.hpp"

namespace tbias {
namespace seg {

constexpr int kWarm = 2;    // warm-up rows of a guessed segment start
constexpr int kTraj = 64;   // trajectory states kept per segment
constexpr int kMinSeg = 8;  // shortest segment worth a wave
constexpr uint32_t kSpinLimit = 1u << 26;
constexpr int32_t kStateTimeout = -3;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;

// Tables shared by the waves of one workgroup (one stream).
template <int PER>
struct alignas(16) Tables {
  float rpsi[64 * PER];            // psi of the root move; -inf for blank and padding
  int32_t rdst[64 * PER];          // target of the root move
  uint16_t cls[64 * PER];          // class of every token (0xffff: none)
  uint16_t cls_ptr[64 * PER + 8];  // members of class c: cls_tok[cls_ptr[c] .. cls_ptr[c+1])
  uint16_t cls_tok[64 * PER];
};

template <int PER>
struct Shape {
  static constexpr int W = PER <= 20 ? 16 : 8;  // waves (segments) per workgroup
  static constexpr int NT = 64 * W;
  // small rows leave room for two workgroups per CU
  static constexpr int kBudget = (PER <= 8 ? 80 : 160) * 1024 - 1024;
};

template <int PER>
struct alignas(16) FixedLds {
  static constexpr int W = Shape<PER>::W;
  float zbuf[W][64 * PER];  // row of the step each wave evaluates
  uint8_t stamps[W][64 * PER];
  Tables<PER> tab;
  int32_t traj[W][kTraj];  // state after each of the first kTraj steps
  int32_t fin_state[W];    // exact state after each segment
  int32_t fin_ready[W];
  int32_t abort_flag;
};

constexpr int kHotRecordBytes = 4 + 4 + 4 + 4 + 2;
template <int PER>
constexpr int hot_states() {
  const int room = (Shape<PER>::kBudget - (int)sizeof(FixedLds<PER>)) / kHotRecordBytes;
  const int h = (room / 64) * 64;
  return h > 4096 ? 4096 : h;
}

template <int PER>
struct alignas(16) SegLds : FixedLds<PER> {
  static constexpr int HOT = hot_states<PER>();
  int32_t hs_fc[HOT];      // records of states < nhot
  uint32_t hs_lknc[HOT];   // link | n_child << 16
  float hs_phi[HOT];
  float hs_psi[HOT];
  uint16_t hs_label[HOT];
};

struct Answer {
  int32_t tok, ns;
  float b, zv;
};

__device__ __forceinline__ int32_t lds_ld(int32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_st(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ int32_t rl(int32_t v, int32_t lane) {
  return __builtin_amdgcn_readlane(v, lane);
}
__device__ __forceinline__ float rlf(float v, int32_t lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// Graph records: from LDS for states < nhot, else from the arena.
struct Graph {
  const ArenaView* A;
  int32_t off, nhot;
  const int32_t* hs_fc;
  const uint32_t* hs_lknc;
  const float* hs_phi;
  const float* hs_psi;
  const uint16_t* hs_label;
  __device__ __forceinline__ float phi(int32_t x) const {
    return x < nhot ? hs_phi[x] : A->phi[off + x];
  }
  __device__ __forceinline__ float psi(int32_t x) const {
    return x < nhot ? hs_psi[x] : A->psi[off + x];
  }
  __device__ __forceinline__ void rec(int32_t x, int32_t& fc, int32_t& nc, int32_t& lnk) const {
    if (x < nhot) {
      fc = hs_fc[x];
      const uint32_t v = hs_lknc[x];
      lnk = (int32_t)(v & 0xffffu);
      nc = (int32_t)(v >> 16);
    } else {
      fc = A->first_child[off + x];
      nc = A->n_child[off + x];
      lnk = A->link[off + x];
    }
  }
};

// Lane geometry of the last chunk (see the row layout above).
template <int PER>
struct RowShape {
  int32_t last_idx;  // element held by this lane in the last chunk
  bool last_ok;      // false for lanes repeating an element of chunk PER-2 (or past V+1)
  __device__ explicit RowShape(int32_t V1) {
    const int lane = __lane_id();
    if (PER > 1) {
      last_idx = V1 - 64 + lane;
      last_ok = last_idx >= 64 * (PER - 1);
    } else {
      last_ok = lane < V1;
      last_idx = last_ok ? lane : V1 - 1;
    }
  }
};

template <class Ld, int PER>
__device__ __forceinline__ void load_row(float* dst, const typename Ld::T* row,
                                         const RowShape<PER>& rs) {
  const int lane = __lane_id();
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) dst[j] = Ld::get(row, 64 * j + lane);
  dst[PER - 1] = Ld::get(row, rs.last_idx);
}

// The boosted step from state x on the row in zrow (LDS), given the row's best
// root move. All lanes take part; the result is uniform.
template <int PER>
__device__ __forceinline__ Answer eval_state(const Graph& G, const Tables<PER>& tb,
                                             const float* zrow, uint8_t* stamps, uint32_t& tag,
                                             int32_t x, float zb, float r1_y, int32_t r1_tok,
                                             int32_t r1_dst, int32_t r1_cls, int32_t V) {
  const int lane = __lane_id();
  if (++tag == 256u) {  // 8-bit tags: clear the table on wrap
    uint32_t* w = reinterpret_cast<uint32_t*>(stamps);
    for (int32_t i = lane; i < 16 * PER; i += 64) w[i] = 0u;
    tag = 1;
  }
  const uint8_t tg = (uint8_t)tag;
  const float phi_x = G.phi(x);

  float lk = kNegInf;
  int32_t lt = INT_MAX, lns = 0;
  float lpsi = 0.f;
  for (int32_t c = x; c != 0;) {
    int32_t fc, nc, lnk;
    G.rec(c, fc, nc, lnk);
    const bool hot_kids = fc + nc <= G.nhot;
    for (int32_t j0 = 0; j0 < nc; j0 += 64) {
      const int32_t j = j0 + lane;
      if (j < nc) {
        const int32_t y = fc + j;
        const int32_t lab = hot_kids ? (int32_t)G.hs_label[y] : G.A->label[G.off + y];
        if (stamps[lab] != tg) {
          stamps[lab] = tg;
          const float py = hot_kids ? G.hs_psi[y] : G.A->psi[G.off + y];
          const int32_t m0 = tb.cls_ptr[lab], m1 = tb.cls_ptr[lab + 1];
          for (int32_t q = m0; q < m1; ++q) {
            const int32_t tok = tb.cls_tok[q];
            const float k = zrow[tok] + py;
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
      const int32_t c = tb.cls[v];
      if (c != 0xffff && stamps[c] == tg) continue;
      const float k = zrow[v] + tb.rpsi[v];
      if (better(k, v, k2, t2)) { k2 = k; t2 = v; d2 = tb.rdst[v]; }
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
    a.b = G.psi(r_ns) - phi_x;
  }
  if (a.tok != V) a.zv = zrow[a.tok];
  return a;
}

// One complete step on a row held in registers (raw[j] as loaded). rp holds
// this lane's root-move psi (-inf for blank and masked lanes). Returns the
// answer and the row's normaliser.
template <int PER>
__device__ __forceinline__ Answer full_step(const Graph& G, const Tables<PER>& tb, float* zrow,
                                            uint8_t* stamps, uint32_t& tag, const float* raw,
                                            const float* rp, const RowShape<PER>& rs, int32_t s,
                                            int mode, int32_t V, float& lse) {
  const int lane = __lane_id();
  float cur[PER];
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) {
    zrow[64 * j + lane] = raw[j];
    cur[j] = raw[j];
  }
  zrow[rs.last_idx] = raw[PER - 1];  // repeated lanes rewrite equal values
  cur[PER - 1] = rs.last_ok ? raw[PER - 1] : kNegInf;
  const float zb = rlf(raw[PER - 1], PER > 1 ? 63 : V);
  asm volatile("" ::: "memory");

  // best root move per lane: strict > keeps the lowest chunk, hence the lowest index
  float zmax = kNegInf, yb = kNegInf;
  int32_t jb = 0;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    zmax = zmax > cur[j] ? zmax : cur[j];
    const float yj = cur[j] + rp[j];
    const bool gt = yj > yb;
    yb = gt ? yj : yb;
    jb = gt ? j : jb;
  }
  const int32_t idx = (jb == PER - 1) ? rs.last_idx : 64 * jb + lane;
  zmax = wave_max_dpp(zmax);
  float ymax;
  int32_t r1_tok;
  wave_argmax_dpp(yb, idx, ymax, r1_tok);
  if (r1_tok >= V) r1_tok = 0;  // only with -inf / nan logits: keep indices in range
  const float mL = zmax * kLog2e;
  float se = 0.f;
#pragma unroll
  for (int j = 0; j < PER; ++j) se += __builtin_amdgcn_exp2f(__builtin_fmaf(cur[j], kLog2e, -mL));
  se = wave_sum_dpp(se);
  lse = zmax + __logf(se);
  Answer a;
  if (mode != 1) {
    const bool blank = !better(ymax, r1_tok, zb, V);
    a.tok = blank ? V : r1_tok;
    a.ns = s;
    a.b = 0.f;
    a.zv = blank ? zb : ymax;
    return a;
  }
  const int32_t c16 = tb.cls[r1_tok];
  return eval_state<PER>(G, tb, zrow, stamps, tag, s, zb, ymax, r1_tok, tb.rdst[r1_tok],
                         c16 == 0xffff ? -1 : c16, V);
}

// Root row and class tables of model m (mode 1) into LDS; NT threads.
template <int PER, int NT>
__device__ __forceinline__ void fill_tables(Tables<PER>& tb, const ArenaView& A, int32_t m,
                                            int mode) {
  const int32_t V1 = A.V1, V = V1 - 1;
  const float* gpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* gdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;
#pragma unroll
  for (int k = 0; k < (64 * PER + NT - 1) / NT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < 64 * PER) {
      tb.rpsi[i] = (i < V) ? (mode == 1 ? gpsi[i] : 0.f) : kNegInf;
      tb.rdst[i] = (i < V && mode == 1) ? gdst[i] : 0;
      const int32_t c = (i < V1) ? A.class_map[i] : -1;
      tb.cls[i] = c < 0 ? (uint16_t)0xffff : (uint16_t)c;
      tb.cls_ptr[i] = (i < V1) ? (uint16_t)A.cls_ptr[i] : (uint16_t)0;
      tb.cls_tok[i] = (i < V) ? (uint16_t)A.cls_tok[i] : (uint16_t)0;
    }
  }
}

// This lane's root-move psi per chunk, from the LDS tables.
template <int PER>
__device__ __forceinline__ void root_psi_regs(float* rp, const Tables<PER>& tb,
                                              const RowShape<PER>& rs) {
  const int lane = __lane_id();
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) rp[j] = tb.rpsi[64 * j + lane];
  rp[PER - 1] = rs.last_ok ? tb.rpsi[rs.last_idx] : kNegInf;
}

template <class Ld, int PER>
__global__ __launch_bounds__(Shape<PER>::NT) void greedy_seg_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  constexpr int W = Shape<PER>::W;
  constexpr int NT = Shape<PER>::NT;
  constexpr int HOT = SegLds<PER>::HOT;
  __shared__ SegLds<PER> S;
  const int32_t V1 = A.V1, V = V1 - 1;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int32_t b = blockIdx.x % B;
  const int32_t g = blockIdx.x / B;

  const int32_t m = model_ids[b];
  const int32_t s0 = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s0, off, n);
  fill_tables<PER, NT>(S.tab, A, m, mode);
  const int32_t nhot = (mode == 1) ? (n < HOT ? n : HOT) : 0;
#pragma unroll
  for (int k = 0; k < (HOT + NT - 1) / NT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < nhot) {
      S.hs_fc[i] = A.first_child[off + i];
      S.hs_lknc[i] = (uint32_t)A.link[off + i] | ((uint32_t)A.n_child[off + i] << 16);
      S.hs_phi[i] = A.phi[off + i];
      S.hs_psi[i] = A.psi[off + i];
      const int32_t lab = A.label[off + i];
      S.hs_label[i] = (uint16_t)(lab < 0 ? 0 : lab);
    }
  }
  for (int32_t i = threadIdx.x; i < (int32_t)sizeof(S.stamps) / 4; i += NT)
    reinterpret_cast<uint32_t*>(&S.stamps[0][0])[i] = 0u;
  if (threadIdx.x < W) {
    S.fin_ready[threadIdx.x] = 0;
    S.fin_state[threadIdx.x] = 0;
  }
  if (threadIdx.x == 0) S.abort_flag = 0;
  __syncthreads();

  Graph Gr;
  Gr.A = &A;
  Gr.off = off;
  Gr.nhot = nhot;
  Gr.hs_fc = S.hs_fc;
  Gr.hs_lknc = S.hs_lknc;
  Gr.hs_phi = S.hs_phi;
  Gr.hs_psi = S.hs_psi;
  Gr.hs_label = S.hs_label;
  float* zrow = S.zbuf[w];
  uint8_t* stamps = S.stamps[w];
  uint32_t tag = 0;
  const RowShape<PER> rs(V1);
  float rp[PER];
  root_psi_regs<PER>(rp, S.tab, rs);

  const int32_t unbiased_state = (mode == 0) ? TB_STATE_NONE : TB_STATE_INVALID;
  const int32_t segi = g * W + w;
  const int32_t t0 = segi * L;
  const int32_t t1 = (t0 + L < T) ? t0 + L : T;
  const bool exact_start = (segi == 0) || mode != 1;
  const int32_t start = (mode == 1) ? (segi == 0 ? s0 : 0) : unbiased_state;
  const int32_t tw = exact_start ? t0 : (t0 - kWarm > 0 ? t0 - kWarm : 0);

  // ---- main pass over the segment (with warm-up rows)
  int32_t s = start;
  int32_t assumed = start;
  if (t0 < t1) {
    // Two row buffers used in turn; the prefetch is unconditional (the last
    // row of the segment is read again at the end) so that the wait for the
    // current row can leave the next row's loads in flight.
    float ra[PER], rb[PER];
    int32_t o_tok = 0, o_st = 0;
    float o_sc = 0.f;
    auto step = [&](const float* cur, float* nxt, int32_t t) {
      const int32_t tn = (t + 1 < t1) ? t + 1 : t;
      load_row<Ld, PER>(nxt, logits + ((int64_t)tn * B + b) * stride, rs);
      if (t == t0) assumed = s;
      float lse;
      const Answer a = full_step<PER>(Gr, S.tab, zrow, stamps, tag, cur, rp, rs, s, mode, V, lse);
      if (t >= t0) {
        const int32_t i = t - t0;
        const int32_t ln = i & 63;
        const bool mine = lane == ln;
        o_tok = mine ? a.tok : o_tok;
        o_st = mine ? a.ns : o_st;
        o_sc = mine ? (a.zv - lse) + a.b : o_sc;
        if (i < kTraj && lane == 0) S.traj[w][i] = a.ns;
        if (ln == 63 || t == t1 - 1) {
          if (lane <= ln) {
            const int64_t oi = (int64_t)(t - ln + lane) * B + b;
            out_tok[oi] = o_tok;
            out_state[oi] = o_st;
            out_score[oi] = o_sc;
          }
        }
      }
      s = __builtin_amdgcn_readfirstlane(a.ns);
    };
    load_row<Ld, PER>(ra, logits + ((int64_t)tw * B + b) * stride, rs);
    for (int32_t t = tw; t < t1; t += 2) {
      step(ra, rb, t);
      if (t + 1 < t1) step(rb, ra, t + 1);
    }
  }

  // ---- hand the exact state along the segments of this workgroup
  int32_t fin = s;
  if (w > 0) {
    uint32_t spins = 0;
    while (lds_ld(&S.fin_ready[w - 1]) == 0) {
      if (lds_ld(&S.abort_flag) || ++spins > kSpinLimit) {
        lds_st(&S.abort_flag, 1);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    asm volatile("" ::: "memory");
    const int32_t exact = __builtin_amdgcn_readfirstlane(lds_ld(&S.fin_state[w - 1]));
    if (lds_ld(&S.abort_flag)) {
      for (int32_t t = t0 + lane; t < t1; t += 64) out_state[(int64_t)t * B + b] = kStateTimeout;
    } else if (t0 >= t1) {
      fin = exact;  // empty segment: pass the state on
    } else if (exact != assumed) {
      // recompute from the exact state until the trajectories meet
      int32_t x = exact;
      bool met = false;
      for (int32_t t = t0; t < t1; ++t) {
        float cur[PER];
        load_row<Ld, PER>(cur, logits + ((int64_t)t * B + b) * stride, rs);
        float lse;
        const Answer a =
            full_step<PER>(Gr, S.tab, zrow, stamps, tag, cur, rp, rs, x, mode, V, lse);
        const int32_t i = t - t0;
        const int32_t old = (i < kTraj) ? __builtin_amdgcn_readfirstlane(S.traj[w][i]) : INT_MIN;
        if (lane == (i & 63)) {  // the lane that wrote this row in the main pass
          const int64_t oi = (int64_t)t * B + b;
          out_tok[oi] = a.tok;
          out_state[oi] = a.ns;
          out_score[oi] = (a.zv - lse) + a.b;
        }
        x = __builtin_amdgcn_readfirstlane(a.ns);
        if (x == old) {
          met = true;
          break;
        }
      }
      fin = met ? s : x;
    }
  }
  if (lane == 0) {
    lds_st(&S.fin_state[w], fin);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    lds_st(&S.fin_ready[w], 1);
    // with several workgroups per stream the fix-up kernel writes the carry
    if (G == 1 && w == W - 1) states[b] = lds_ld(&S.abort_flag) ? kStateTimeout : fin;
  }
}

// Repairs the workgroup boundaries of each stream after greedy_seg_kernel
// (one wave per stream, boundaries in order): from the exact state before a
// boundary, recompute until the stored trajectory is met. Writes the carry.
template <class Ld, int PER>
__global__ __launch_bounds__(64) void greedy_fix_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, int32_t W, const int32_t* __restrict__ model_ids,
    int32_t* __restrict__ states, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  __shared__ Tables<PER> tb;
  __shared__ float zrow[64 * PER];
  __shared__ uint8_t stamps[64 * PER];
  const int32_t V1 = A.V1, V = V1 - 1;
  const int lane = __lane_id();
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  // The carried state was consumed by the main kernel; streams that are not
  // biased, or whose carried state was invalid, have exact (unboosted)
  // segment starts and need no repair.
  const bool biased = m >= 0 && m < A.n_models;
  bool timed_out = false;
  if (biased) {
    const int32_t off = A.model_off[m], n = A.model_n[m];
    fill_tables<PER, 64>(tb, A, m, 1);
    for (int32_t i = lane; i < 16 * PER; i += 64) reinterpret_cast<uint32_t*>(stamps)[i] = 0u;
    __syncthreads();
    Graph Gr;
    Gr.A = &A;
    Gr.off = off;
    Gr.nhot = 0;
    Gr.hs_fc = nullptr;
    Gr.hs_lknc = nullptr;
    Gr.hs_phi = nullptr;
    Gr.hs_psi = nullptr;
    Gr.hs_label = nullptr;
    uint32_t tag = 0;
    const RowShape<PER> rs(V1);
    float rp[PER];
    root_psi_regs<PER>(rp, tb, rs);
    int32_t t = 0;
    for (int32_t gg = 1; gg < G; ++gg) {
      const int32_t tb0 = gg * W * L;
      if (tb0 >= T) break;
      if (t > tb0) continue;  // an earlier repair already ran past this boundary
      t = tb0;
      int32_t x = __builtin_amdgcn_readfirstlane(out_state[(int64_t)(t - 1) * B + b]);
      if (x < 0 || x >= n) {  // invalid carried state (-2) or a timed-out main kernel (-3)
        timed_out = x == kStateTimeout;
        break;
      }
      for (; t < T; ++t) {
        float cur[PER];
        load_row<Ld, PER>(cur, logits + ((int64_t)t * B + b) * stride, rs);
        float lse;
        const Answer a = full_step<PER>(Gr, tb, zrow, stamps, tag, cur, rp, rs, x, 1, V, lse);
        const int64_t oi = (int64_t)t * B + b;
        const int32_t old = __builtin_amdgcn_readfirstlane(out_state[oi]);
        if (lane == 0) {
          out_tok[oi] = a.tok;
          out_state[oi] = a.ns;
          out_score[oi] = (a.zv - lse) + a.b;
        }
        x = __builtin_amdgcn_readfirstlane(a.ns);
        if (x == old) {
          ++t;
          break;
        }
      }
    }
  }
  if (lane == 0) states[b] = timed_out ? kStateTimeout : out_state[(int64_t)(T - 1) * B + b];
}

// Launch geometry: workgroups per stream G and segment length L.
template <int PER>
inline void seg_geometry(int32_t T, int32_t B, int32_t& G, int32_t& L) {
  constexpr int W = Shape<PER>::W;
  // enough workgroups to cover the 256 CUs, but segments of at least kMinSeg rows
  G = (256 + B - 1) / B;
  const int32_t gmax = (T + W * kMinSeg - 1) / (W * kMinSeg);
  if (G > gmax) G = gmax;
  if (G < 1) G = 1;
  L = (T + G * W - 1) / (G * W);
  if (L < kMinSeg) L = kMinSeg;
  // every workgroup must own rows (an empty one would not hand on a state)
  while (G > 1 && (G - 1) * W * L >= T) --G;
}

template <class Ld, int PER>
hipError_t launch_seg(const ArenaView& A, const void* logits, int32_t T, int32_t B,
                      int64_t stride, const int32_t* model_ids, int32_t* states, int32_t* out_tok,
                      int32_t* out_state, float* out_score, hipStream_t st) {
  typedef typename Ld::T TT;
  static_assert(sizeof(SegLds<PER>) <= Shape<PER>::kBudget + 1024, "LDS budget");
  static_assert(SegLds<PER>::HOT >= 64, "room for hot states");
  int32_t G, L;
  seg_geometry<PER>(T, B, G, L);
  hipLaunchKernelGGL((greedy_seg_kernel<Ld, PER>), dim3(B * G), dim3(Shape<PER>::NT), 0, st, A,
                     static_cast<const TT*>(logits), T, B, stride, G, L, model_ids, states,
                     out_tok, out_state, out_score);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || G == 1) return e;
  hipLaunchKernelGGL((greedy_fix_kernel<Ld, PER>), dim3(B), dim3(64), 0, st, A,
                     static_cast<const TT*>(logits), T, B, stride, G, L, Shape<PER>::W,
                     model_ids, states, out_tok, out_state, out_score);
  return hipGetLastError();
}

// Launchers for chunk counts in [lo, hi], one translation unit per range.
typedef hipError_t (*SegLaunch)(const ArenaView&, const void*, int32_t, int32_t, int64_t,
                                const int32_t*, int32_t*, int32_t*, int32_t*, float*,
                                hipStream_t);
SegLaunch seg_launcher_1_8(int per, int32_t dtype);
SegLaunch seg_launcher_9_16(int per, int32_t dtype);
SegLaunch seg_launcher_17_24(int per, int32_t dtype);
SegLaunch seg_launcher_25_32(int per, int32_t dtype);

}  // namespace seg
}  // namespace tbias
