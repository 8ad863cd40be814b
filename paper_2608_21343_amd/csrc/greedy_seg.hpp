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
// Per-wave LDS: the row and a bitmap marking the classes that are overridden
// in the state being evaluated. Shared LDS: the model's root row, the class
// tables, and the packed records of the model's first (shallowest) states
// with its psi and phi value tables: every state of a model of a few
// thousand states, so that a step reads LDS only.
#pragma once

#include <climits>

#include "device.hpp"
#include "launch.hpp"

namespace tbias {
namespace seg {

constexpr int kWarm = 4;    // warm-up rows of a guessed segment start
constexpr int kTraj = 64;   // trajectory states kept per segment
constexpr int kMinSeg = 8;  // shortest segment worth a wave
constexpr int kScalarKids = 8;  // arena children walked one at a time up to this many
// Polls of the hand-off wait before it gives up (rows then get
// TB_STATE_TIMEOUT). The waves of a workgroup are resident together and a
// wave never waits for a later one, so the wait always ends well before this.
constexpr uint32_t kSpinLimit = 1u << 26;
constexpr int32_t kStateTimeout = TB_STATE_TIMEOUT;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;

// State-independent facts of one row: blank logit, best root move (key,
// token, its class, target state, target psi and logit) and normaliser.
struct RowSum {
  float zb, ymax, lse, r1_psi, r1_z;
  int32_t r1_tok, r1_cls, r1_dst;
};

// A lane's two best root moves (token ids; kNoTok when the lane has none),
// tracked only by the short-call kernel.
constexpr int32_t kNoTok = 0xffff;
struct LaneTop {
  int32_t i1, i2;
  float k1, k2;
};

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
  static constexpr int kMarkWords = 2 * PER;  // one bit per token id / class id
  float zbuf[W][64 * PER];  // row of the step each wave evaluates
  uint32_t marks[W][kMarkWords];
  Tables<PER> tab;
  int32_t traj[W][kTraj];  // state after each of the first kTraj steps
  RowSum rsum[W];          // short calls: summary of row w
  uint32_t ltop[W][64];    // short calls: each lane's two best root moves of row w
  int32_t spec_ns[2][W];   // short calls: state after row w's step from its guess (by round)
  int32_t spec_x[W];       // short calls: row w's final guess and its answer
  int4 spec_ans[W];
  float lse[W];            // short calls: normaliser of row w
  int32_t fin_state[W];    // exact state after each segment
  int32_t fin_ready[W];
  int32_t abort_flag;
};

// Records of the first HOT states of a model (BFS order: the shallowest, the
// most visited) held in LDS: one 16-byte state record and the 8-byte record
// of the arc into the state (its class and first three members, as arc_mem).
template <int HOT>
struct alignas(16) HotRecords {
  int4 rec[HOT];   // first child, link | n_child << 16, phi bits, psi bits
  uint2 mem[HOT];  // arc member record
};

constexpr int kHotRecordBytes = 16 + 8;

// Packed records (see state_rec in tbias.h) of the first HOT states of a
// model and the model's psi and phi value tables, held in LDS by the greedy
// kernels.
template <int HOT>
struct alignas(16) StateHot {
  uint32_t w0[HOT];
  uint32_t w1[HOT];
  uint32_t w2[HOT];
  float vpsi[256];
  float vphi[256];
};
constexpr int kStateHotBytes = 12;

template <int PER>
constexpr int hot_states() {
  const int room =
      (Shape<PER>::kBudget - (int)sizeof(FixedLds<PER>) - 2048) / kStateHotBytes;
  const int h = (room / 64) * 64;
  return h > 8192 ? 8192 : h;
}

template <int PER>
struct alignas(16) SegLds : FixedLds<PER> {
  static constexpr int HOT = hot_states<PER>();
  StateHot<HOT> hot;
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

// Read-only load through the scalar cache (uniform address). It waits on the
// scalar counter, not behind the vector loads of the prefetched rows.
template <class T>
__device__ __forceinline__ T sload(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}

// A read through an explicitly global pointer: keeps the compiler from merging
// it with an LDS read of the other branch into one generic (flat) load.
template <class T>
__device__ __forceinline__ T gload(const T* p) {
  return *(const __attribute__((address_space(1))) T*)(p);
}

__device__ __forceinline__ uint4 sload4(const uint4* p) {
  const uint32_t* q = reinterpret_cast<const uint32_t*>(p);
  return make_uint4(sload(q), sload(q + 1), sload(q + 2), sload(q + 3));
}

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

// Graph records: from LDS for states < nhot, else from the arena by scalar
// loads (the arena is immutable while a step runs; state ids are uniform).
struct Graph {
  const ArenaView* A;
  int32_t off, nhot;
  const int4* hrec;
  const uint2* hmem;
  template <int HOT>
  __device__ __forceinline__ Graph(const ArenaView& a, int32_t o, int32_t nh,
                                   const HotRecords<HOT>& h)
      : A(&a), off(o), nhot(nh), hrec(h.rec), hmem(h.mem) {}
  __device__ __forceinline__ float phi_of(int32_t x) const {
    return x < nhot ? __int_as_float(hrec[x].z) : sload(A->phi + off + x);
  }
  __device__ __forceinline__ float psi_of(int32_t x) const {
    return x < nhot ? __int_as_float(hrec[x].w) : sload(A->psi + off + x);
  }
  // first child, child count, suffix link and phi of state x (uniform)
  __device__ __forceinline__ void rec(int32_t x, int32_t& fc, int32_t& nc, int32_t& lnk,
                                      float& phi) const {
    if (x < nhot) {
      const int4 r = hrec[x];
      fc = r.x;
      lnk = (int32_t)((uint32_t)r.y & 0xffffu);
      nc = (int32_t)((uint32_t)r.y >> 16);
      phi = __int_as_float(r.z);
    } else {
      fc = sload(A->first_child + off + x);
      nc = sload(A->n_child + off + x);
      lnk = sload(A->link + off + x);
      phi = sload(A->phi + off + x);
    }
  }
};

// Graph records for the greedy kernels: the packed record of a state from LDS
// for states < nhot; with FAR, the others from the arena's packed records
// (the arena is immutable while a step runs); the plain arena arrays for a
// record that is not usable (flagged) and, without FAR, for states >= nhot.
template <bool FAR>
struct SGraphT {
  static constexpr bool kFar = FAR;
  const ArenaView* A;
  int32_t off, nhot;
  const uint32_t* w0;
  const uint32_t* w1;
  const uint32_t* w2;
  const float* vpsi;
  const float* vphi;
  const uint16_t* cls_tok;  // class members (LDS copy of the arena's cls_tok)
  template <int HOT, int PER>
  __device__ __forceinline__ SGraphT(const ArenaView& a, int32_t o, int32_t nh,
                                     const StateHot<HOT>& h, const Tables<PER>& tb)
      : A(&a), off(o), nhot(nh), w0(h.w0), w1(h.w1), w2(h.w2), vpsi(h.vpsi), vphi(h.vphi),
        cls_tok(tb.cls_tok) {}
  // first child, child count, suffix link and phi of state x from its packed
  // record (uniform); false when there is no usable one (see above), or when
  // the value tables are not in LDS (no hot states)
  __device__ __forceinline__ bool srec(int32_t x, int32_t& fc, int32_t& nc, int32_t& lnk,
                                       float& phi) const {
    uint32_t a, b, c;
    if (x < nhot) {
      // the three words are read together (one LDS round trip), then checked
      const uint32_t a0 = w0[x], b0 = w1[x], c0 = w2[x];
      c = __builtin_amdgcn_readfirstlane(c0);
      a = __builtin_amdgcn_readfirstlane(a0);
      b = __builtin_amdgcn_readfirstlane(b0);
    } else if constexpr (FAR) {
      if (nhot == 0) return false;  // no value tables in LDS
      const uint32_t* g = A->state_rec + 3 * ((int64_t)off + x);
      const uint32_t a0 = gload(g), b0 = gload(g + 1), c0 = gload(g + 2);
      c = __builtin_amdgcn_readfirstlane(c0);
      a = __builtin_amdgcn_readfirstlane(a0);
      b = __builtin_amdgcn_readfirstlane(b0);
    } else {
      return false;
    }
    if (c >> 31) return false;
    fc = (int32_t)(a & 0xffffu);
    nc = (int32_t)((a >> 16) & 0xffu);
    lnk = (int32_t)(b & 0xffffu);
    phi = vphi[(c >> 8) & 0xffu];
    return true;
  }
  // psi of state x (uniform): from its LDS record when usable, else the arena
  __device__ __forceinline__ float psi_of(int32_t x) const {
    if (x < nhot) {
      const uint32_t a0 = w0[x], c0 = w2[x];
      const uint32_t c = __builtin_amdgcn_readfirstlane(c0);
      // the value index is the record's top byte: an unsigned shift
      if (!(c >> 31)) return vpsi[(uint32_t)__builtin_amdgcn_readfirstlane(a0) >> 24];
    }
    return sload(A->psi + off + x);
  }
  // the same, from the arena when x has no usable LDS record
  __device__ __forceinline__ void rec(int32_t x, int32_t& fc, int32_t& nc, int32_t& lnk,
                                      float& phi) const {
    if (!srec(x, fc, nc, lnk, phi)) {
      fc = sload(A->first_child + off + x);
      nc = sload(A->n_child + off + x);
      lnk = sload(A->link + off + x);
      phi = sload(A->phi + off + x);
    }
  }
};
using SGraph = SGraphT<false>;

// Arc member record fields.
__device__ __forceinline__ int32_t arc_class(uint2 m) { return (int32_t)((m.y >> 16) & 0x7fffu); }
__device__ __forceinline__ bool arc_more(uint2 m) { return (m.y >> 31) != 0u; }

// Records of states [0, nhot) of the model at off into LDS; NT threads.
template <int HOT, int NT>
__device__ __forceinline__ void fill_hot(HotRecords<HOT>& h, const ArenaView& A, int32_t off,
                                         int32_t nhot) {
#pragma unroll
  for (int k = 0; k < (HOT + NT - 1) / NT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < nhot) {
      int4 r;
      r.x = A.first_child[off + i];
      r.y = (int32_t)((uint32_t)A.link[off + i] | ((uint32_t)A.n_child[off + i] << 16));
      r.z = __float_as_int(A.phi[off + i]);
      r.w = __float_as_int(A.psi[off + i]);
      h.rec[i] = r;
      const int64_t q = 2 * ((int64_t)off + i);
      h.mem[i] = make_uint2(A.arc_mem[q], A.arc_mem[q + 1]);
    }
  }
}

// Packed records of states [0, nhot) of the model at off and its value
// tables (model m) into LDS; NT threads.
template <int HOT, int NT>
__device__ __forceinline__ void fill_state_hot(StateHot<HOT>& h, const ArenaView& A, int32_t m,
                                               int32_t off, int32_t nhot) {
  const uint32_t* src = A.state_rec + 3 * (int64_t)off;
#pragma unroll
  for (int k = 0; k < (HOT + NT - 1) / NT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < nhot) {
      h.w0[i] = src[3 * i];
      h.w1[i] = src[3 * i + 1];
      h.w2[i] = src[3 * i + 2];
    }
  }
  if (nhot > 0) {
    const float* vt = A.value_tab + 512 * (int64_t)m;
    for (int32_t i = threadIdx.x; i < 512; i += NT) {
      if (i < 256) h.vpsi[i] = vt[i];
      else h.vphi[i - 256] = vt[i];
    }
  }
}

template <class Ld, int PER>
__device__ __forceinline__ void load_row(float* dst, const typename Ld::T* row,
                                         const RowShape<PER>& rs) {
  const int lane = __lane_id();
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) dst[j] = Ld::get(row, 64 * j + lane);
  dst[PER - 1] = Ld::get(row, rs.last_idx);
}

// Bumps the 8-bit tag of a wave's class-mark table, clearing it on wrap.
template <int PER>
__device__ __forceinline__ uint8_t next_tag(uint8_t* stamps, uint32_t& tag) {
  if (++tag == 256u) {
    uint32_t* w = reinterpret_cast<uint32_t*>(stamps);
    for (int32_t i = __lane_id(); i < 16 * PER; i += 64) w[i] = 0u;
    tag = 1;
  }
  return (uint8_t)tag;
}

// Class-mark bitmaps (one bit per class id) of the greedy kernels. Marks are
// set with LDS atomics and read by the same wave afterwards; a wave's LDS
// operations complete in order.
template <int PER>
__device__ __forceinline__ void marks_clear(uint32_t* bits) {
  if (__lane_id() < 2 * PER) bits[__lane_id()] = 0u;
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void mark(uint32_t* bits, int32_t c) {
  __hip_atomic_fetch_or(bits + (c >> 5), 1u << (c & 31), __ATOMIC_RELAXED,
                        __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ bool is_marked(const uint32_t* bits, int32_t c) {
  return (bits[c >> 5] >> (c & 31)) & 1u;
}
__device__ __forceinline__ void marks_fence() { asm volatile("" ::: "memory"); }

// Per-lane best override candidate.
struct Cand {
  float k, z, psi;
  int32_t tok, ns;
  __device__ __forceinline__ void offer(float kk, int32_t t, float zz, int32_t y, float py) {
    if (better(kk, t, k, tok)) { k = kk; tok = t; z = zz; ns = y; psi = py; }
  }
};

// Members of the arc class m into state y (psi py) offered by this lane.
template <int PER>
__device__ __forceinline__ void offer_members(Cand& c, const Tables<PER>& tb, const float* zrow,
                                              uint2 m, int32_t y, float py) {
  if (!arc_more(m)) {  // up to three members, ascending (repeats when fewer)
    const int32_t t0 = (int32_t)(m.x & 0xffffu), t1 = (int32_t)(m.x >> 16);
    const int32_t t2 = (int32_t)(m.y & 0xffffu);
    const float z0 = zrow[t0], z1 = zrow[t1], z2 = zrow[t2];
    c.offer(z0 + py, t0, z0, y, py);
    c.offer(z1 + py, t1, z1, y, py);
    c.offer(z2 + py, t2, z2, y, py);
  } else {
    const int32_t lab = arc_class(m);
    for (int32_t q = tb.cls_ptr[lab]; q < tb.cls_ptr[lab + 1]; ++q) {
      const int32_t t = tb.cls_tok[q];
      const float z = zrow[t];
      c.offer(z + py, t, z, y, py);
    }
  }
}

// Arc record and psi of child y (hot: LDS; else one vector load each).
__device__ __forceinline__ void child_rec(const Graph& G, int32_t y, uint2& m, float& py) {
  if (y < G.nhot) {
    m = G.hmem[y];
    py = __int_as_float(G.hrec[y].w);
  } else {
    const int64_t q = 2 * ((int64_t)G.off + y);
    m = make_uint2(G.A->arc_mem[q], G.A->arc_mem[q + 1]);
    py = G.A->psi[G.off + y];
  }
}

// Arc record (as arc_mem) and psi of child y: rebuilt from its LDS record
// when it has a usable one, else read from the arena.
template <bool F>
__device__ __forceinline__ void child_rec(const SGraphT<F>& G, int32_t y, uint2& m, float& py) {
  if (y < G.nhot) {
    const uint32_t a = G.w0[y], b = G.w1[y], c = G.w2[y];
    if (!(c >> 31)) {
      const int32_t mc = (int32_t)(c & 0xffu), ms = (int32_t)(b >> 16);
      const uint32_t t0 = G.cls_tok[ms];
      const uint32_t t1 = G.cls_tok[ms + (mc > 1 ? 1 : 0)];
      const uint32_t t2 = G.cls_tok[ms + (mc > 2 ? 2 : (mc > 1 ? 1 : 0))];
      m = make_uint2(t0 | (t1 << 16), t2 | (c & 0x7fff0000u) | (mc > 3 ? 0x80000000u : 0u));
      py = G.vpsi[a >> 24];
      return;
    }
  }
  const int64_t q = 2 * ((int64_t)G.off + y);
  m = make_uint2(gload(G.A->arc_mem + q), gload(G.A->arc_mem + q + 1));
  py = gload(G.A->psi + G.off + y);
}

// Marks the classes of the children [fc, fc+nc).
template <bool F>
__device__ __forceinline__ void mark_children(const SGraphT<F>& G, uint32_t* marks, int32_t fc,
                                              int32_t nc) {
  for (int32_t j = __lane_id(); j < nc; j += 64) {
    uint2 m;
    float py;
    child_rec(G, fc + j, m, py);
    mark(marks, arc_class(m));
  }
  marks_fence();
}

// Best root move whose class is not marked, from every lane's two best root
// moves: a lane whose best is marked offers its runner-up. Returns false when
// some lane's best two are both marked and its further moves could still
// reach the result.
template <int PER>
__device__ __forceinline__ bool root_excluding(const Tables<PER>& tb, const float* zrow,
                                               const uint32_t* marks, LaneTop top, float& rk,
                                               int32_t& rt) {
  const bool h1 = top.i1 != kNoTok, h2 = top.i2 != kNoTok;
  const int32_t i1 = h1 ? top.i1 : 0, i2 = h2 ? top.i2 : 0;
  const int32_t c1 = tb.cls[i1], c2 = tb.cls[i2];
  const float k1 = zrow[i1] + tb.rpsi[i1], k2 = zrow[i2] + tb.rpsi[i2];
  const bool o1 = h1 && c1 != 0xffff && is_marked(marks, c1);
  const bool o2 = h2 && c2 != 0xffff && is_marked(marks, c2);
  const bool use1 = h1 && !o1, use2 = !use1 && h2 && !o2;
  const float k = use1 ? k1 : (use2 ? k2 : kNegInf);
  const int32_t t = use1 ? i1 : (use2 ? i2 : INT_MAX);
  wave_argmax_dpp(k, t, rk, rt);
  // A lane whose best two are both marked holds further moves with keys at
  // most its runner-up's; they matter only if that key reaches the result
  // (equal keys included: a lower index would win the tie).
  return __ballot(o1 && o2 && !(k2 < rk)) == 0ull;
}

// Best root move whose class is not marked, over the whole row (unrolled
// over the row's chunks so that the table reads of several chunks issue
// together).
template <int PER>
__device__ __forceinline__ void root_scan(const Tables<PER>& tb, const float* zrow,
                                          const uint32_t* marks, const RowShape<PER>& rs,
                                          float& rk, int32_t& rt) {
  const int lane = __lane_id();
  float k2 = kNegInf;
  int32_t t2 = INT_MAX;
#pragma unroll 6
  for (int j = 0; j < PER; ++j) {
    const int32_t v = (j < PER - 1) ? 64 * j + lane : rs.last_idx;
    const int32_t cv = tb.cls[v];
    const bool ok_lane = (j < PER - 1) || rs.last_ok;
    const float k = zrow[v] + tb.rpsi[v];  // -inf for the blank
    const bool ov = cv != 0xffff && is_marked(marks, cv);
    if (ok_lane && !ov && k > k2) { k2 = k; t2 = v; }
  }
  wave_argmax_dpp(k2, t2, rk, rt);
}

// The boosted step from state x on the row in zrow (LDS), given the row's
// summary. All lanes take part; the result is uniform.
//
// The children of the states on x's suffix chain override the root move of
// their class, deeper states first; every other token takes its root move
// (the row's best of those is r.r1 unless its class is overridden); the blank
// keeps the state. Class marks are needed only when the chain has more than
// one state (to let deeper states win) or when r.r1's class is overridden.
template <int PER, class GR>
__device__ __forceinline__ Answer eval_general(const GR& G, const Tables<PER>& tb,
                                               const float* zrow, uint32_t* marks,
                                               const RowShape<PER>& rs, int32_t x, const RowSum& r,
                                               const LaneTop* top, int32_t V) {
  const int lane = __lane_id();
  int32_t fc, nc, lnk;
  float phi_x;
  G.rec(x, fc, nc, lnk, phi_x);
  const int32_t fc0 = fc, nc0 = nc;
  const bool multi = lnk != 0;
  if (multi) marks_clear<PER>(marks);

  Cand c;
  c.k = kNegInf;
  c.tok = INT_MAX;
  c.z = 0.f;
  c.psi = 0.f;
  c.ns = 0;
  bool over = false;
  for (int32_t lvl = 0; x != 0; ++lvl) {
    if (fc + nc <= G.nhot || nc > kScalarKids) {
      // one child per lane
      for (int32_t j0 = 0; j0 < nc; j0 += 64) {
        const int32_t j = j0 + lane;
        if (j < nc) {
          const int32_t y = fc + j;
          uint2 m;
          float py;
          child_rec(G, y, m, py);
          const int32_t lab = arc_class(m);
          bool take = true;
          if (multi) {
            take = lvl == 0 || !is_marked(marks, lab);
            if (take) mark(marks, lab);
          }
          if (take) {
            over |= lab == r.r1_cls;
            offer_members<PER>(c, tb, zrow, m, y, py);
          }
        }
      }
    } else {
      // a few children in the arena: one child at a time by scalar loads,
      // its members across the lanes
      for (int32_t j = 0; j < nc; ++j) {
        const int32_t y = fc + j;
        const int64_t q = 2 * ((int64_t)G.off + y);
        const uint2 m = make_uint2(sload(G.A->arc_mem + q), sload(G.A->arc_mem + q + 1));
        const float py = sload(G.A->psi + G.off + y);
        const int32_t lab = arc_class(m);
        bool take = true;
        if (multi) {
          take = lvl == 0 || !is_marked(marks, lab);  // uniform
          if (take) mark(marks, lab);
          marks_fence();
        }
        if (take) {
          over |= lab == r.r1_cls;
          int32_t t = -1;
          if (!arc_more(m)) {
            if (lane < 3) t = (int32_t)(lane == 0 ? (m.x & 0xffffu) : lane == 1 ? (m.x >> 16) : (m.y & 0xffffu));
          } else {
            const int32_t qq = tb.cls_ptr[lab] + lane;
            if (qq < tb.cls_ptr[lab + 1]) t = tb.cls_tok[qq];
          }
          if (t >= 0) {
            const float z = zrow[t];
            c.offer(z + py, t, z, y, py);
          }
        }
      }
    }
    marks_fence();  // the next level reads this level's marks
    if (lnk == 0) break;
    float phi_unused;
    G.rec(lnk, fc, nc, lnk, phi_unused);
  }
  float ok;
  int32_t ot;
  const int32_t wl = wave_argmax_dpp(c.k, c.tok, ok, ot);
  const int32_t o_ns = rl(c.ns, wl);
  const float o_psi = rlf(c.psi, wl);
  const float o_z = rlf(c.z, wl);

  // best root move whose class is not overridden
  float rk = r.ymax;
  int32_t rt = r.r1_tok, r_ns = r.r1_dst;
  float r_psi = r.r1_psi, r_z = r.r1_z;
  if (__ballot(over) != 0ull) {
    if (!multi) {
      marks_clear<PER>(marks);
      mark_children(G, marks, fc0, nc0);
    }
    if (!(top && root_excluding<PER>(tb, zrow, marks, *top, rk, rt)))
      root_scan<PER>(tb, zrow, marks, rs, rk, rt);
    const int32_t rv = (rt < V) ? rt : 0;
    r_ns = tb.rdst[rv];
    r_psi = tb.rpsi[rv];
    r_z = zrow[rv];
  }
  Answer a;
  a.tok = V;
  a.ns = x;
  a.b = 0.f;
  a.zv = r.zb;
  float bk = r.zb + phi_x;  // blank keeps the state
  int32_t bt = V;
  if (better(ok, ot, bk, bt)) {
    bk = ok;
    bt = ot;
    a.tok = ot;
    a.ns = o_ns;
    a.b = o_psi - phi_x;
    a.zv = o_z;
  }
  if (better(rk, rt, bk, bt)) {
    a.tok = rt;
    a.ns = r_ns;
    a.b = r_psi - phi_x;
    a.zv = r_z;
  }
  return a;
}

// The step from state x given the first children and child counts of its
// suffix chain (x first, levels non-root states, kChainMax at most): up to
// 64*NS children, NS per lane (slot 64*i + lane in the lane's i-th register),
// provided the children of every level but the shallowest fit in the first 64
// slots (the shadowing scan reads them by readlane). Returns false, with no
// output, on any other shape.
constexpr int kChainMax = 8;

template <int PER, int NS, class GR>
__device__ __forceinline__ bool eval_chain_wide(const GR& G, const Tables<PER>& tb,
                                                const float* zrow, uint32_t* marks,
                                                const RowShape<PER>& rs, int32_t x, float phi_x,
                                                const int32_t (&fl)[kChainMax],
                                                const int32_t (&nl)[kChainMax], int32_t levels,
                                                const RowSum& r, const LaneTop* top, int32_t V,
                                                Answer& a) {
  constexpr int kLv = kChainMax;
  const int lane = __lane_id();
  int32_t st[kLv + 1];  // first slot of every level
  st[0] = 0;
#pragma unroll
  for (int i = 0; i < kLv; ++i) st[i + 1] = st[i] + nl[i];
  const int32_t total = st[kLv];
  int32_t last = 0;  // first slot of the shallowest level
#pragma unroll
  for (int i = 1; i < kLv; ++i) last = (i < levels) ? st[i] : last;
  if (total > 64 * NS || last > 64) return false;

  // a slot's child: its level, state record and best member
  auto slot = [&](int32_t q, int32_t& lv, int32_t& y, int32_t& lab, float& py, float& kb,
                  float& zb, int32_t& tk, bool& in, bool& bad) {
    in = q < total;
    // level and child index without indexing the level arrays (they stay in
    // scalar registers): y = q + (fl[lv] - st[lv]), summed level by level
    lv = 0;
    int32_t yy = q + fl[0];
#pragma unroll
    for (int i = 1; i < kLv; ++i) {
      const bool past = q >= st[i];
      lv += past ? 1 : 0;
      yy += past ? (fl[i] - st[i]) - (fl[i - 1] - st[i - 1]) : 0;
    }
    y = in ? yy : 0;
    uint32_t c0 = 0u, c1 = 0u, c2 = 0x80000000u;
    if (in && y < G.nhot) {
      c0 = G.w0[y];
      c1 = G.w1[y];
      c2 = G.w2[y];
    } else if constexpr (GR::kFar) {
      if (in && G.nhot > 0) {  // the arena's packed record
        const uint32_t* g = G.A->state_rec + 3 * ((int64_t)G.off + y);
        c0 = gload(g);
        c1 = gload(g + 1);
        c2 = gload(g + 2);
      }
    }
    const int32_t mc = (int32_t)(c2 & 0xffu);
    bad = in && ((c2 >> 31) != 0u || mc > 3);
    lab = (int32_t)((c2 >> 16) & 0x7fffu);
    const int32_t ms = in ? (int32_t)(c1 >> 16) : 0;
    py = G.vpsi[c0 >> 24];
    const int32_t t0 = tb.cls_tok[ms];
    const int32_t t1 = tb.cls_tok[ms + (mc > 1 ? 1 : 0)];
    const int32_t t2 = tb.cls_tok[ms + (mc > 2 ? 2 : (mc > 1 ? 1 : 0))];
    const float z0 = zrow[t0], z1 = zrow[t1], z2 = zrow[t2];
    kb = z0 + py;
    zb = z0;
    tk = t0;
    const float k1 = z1 + py, k2 = z2 + py;
    if (k1 > kb) { kb = k1; tk = t1; zb = z1; }  // members ascend: ties keep the lower
    if (k2 > kb) { kb = k2; tk = t2; zb = z2; }
  };
  int32_t lvS[NS], yS[NS], labS[NS], tkS[NS];
  float pyS[NS], kS[NS], zS[NS];
  bool inS[NS];
  bool anybad = false;
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    bool bad;
    slot(64 * i + lane, lvS[i], yS[i], labS[i], pyS[i], kS[i], zS[i], tkS[i], inS[i], bad);
    anybad = anybad || bad;
  }
  if (__ballot(anybad) != 0ull) return false;
  // A class that a deeper chain state (a lower level) also has is shadowed;
  // the deeper levels' slots are all below 64 (lane = slot). The best of all
  // children is the answer unless it is shadowed (a shadowing child has the
  // same tokens; see eval_walk), which is checked on the winner alone.
  // the winner's class, level, child, psi and logit (uniform)
  int32_t w_lab = 0, w_lv = 0, w_y = 0;
  float w_py = 0.f, w_z = 0.f;
  auto best = [&](const bool (&take)[NS], float& ok, int32_t& ot) {
    float bk = kNegInf;
    int32_t bt = INT_MAX, blab = 0, blv = 0, by = 0;
    float bpy = 0.f, bz = 0.f;
#pragma unroll
    for (int i = 0; i < NS; ++i) {  // strict: ties keep the lower slot
      const float k = take[i] ? kS[i] : kNegInf;
      const int32_t t = take[i] ? tkS[i] : INT_MAX;
      if (better(k, t, bk, bt)) {
        bk = k;
        bt = t;
        blab = labS[i];
        blv = lvS[i];
        by = yS[i];
        bpy = pyS[i];
        bz = zS[i];
      }
    }
    const int32_t wl = wave_argmax_dpp(bk, bt, ok, ot);
    w_lab = rl(blab, wl);
    w_lv = rl(blv, wl);
    w_y = rl(by, wl);
    w_py = rlf(bpy, wl);
    w_z = rlf(bz, wl);
  };
  float ok = kNegInf;
  int32_t ot = INT_MAX;
  best(inS, ok, ot);
  {
    const int32_t lw = w_lab, vw = w_lv;
    bool sh = false;
#pragma unroll
    for (int i = 0; i < NS; ++i) sh = sh || (inS[i] && labS[i] == lw && lvS[i] < vw);
    if (__ballot(sh) != 0ull) {
      bool take[NS];
#pragma unroll
      for (int i = 0; i < NS; ++i) take[i] = inS[i];
      for (int32_t j = 0; j < last; ++j) {
        const int32_t cj = __builtin_amdgcn_readlane(labS[0], j);
        const int32_t lvj = __builtin_amdgcn_readlane(lvS[0], j);
#pragma unroll
        for (int i = 0; i < NS; ++i) take[i] = take[i] && !(lvj < lvS[i] && cj == labS[i]);
      }
      best(take, ok, ot);
    }
  }
  const int32_t o_ns = w_y;
  const float o_psi = w_py, o_z = w_z;
  // every chain child's class overrides its root move; the remaining root
  // moves have keys at most r.ymax, so when the best child or the blank is
  // above it no root move can win
  bool h = false;
#pragma unroll
  for (int i = 0; i < NS; ++i) h = h || (inS[i] && labS[i] == r.r1_cls);
  const bool hit = __ballot(h) != 0ull;
  const bool root_lost = hit && (ok > r.ymax || r.zb + phi_x > r.ymax);
  const bool over = hit && !root_lost;
  if (over) {
    marks_clear<PER>(marks);
#pragma unroll
    for (int i = 0; i < NS; ++i)
      if (inS[i]) mark(marks, labS[i]);
    marks_fence();
  }

  // best root move whose class is not overridden
  float rk = root_lost ? kNegInf : r.ymax;
  int32_t rt = r.r1_tok, r_ns = r.r1_dst;
  float r_psi = r.r1_psi, r_z = r.r1_z;
  if (over) {
    if (!(top && root_excluding<PER>(tb, zrow, marks, *top, rk, rt)))
      root_scan<PER>(tb, zrow, marks, rs, rk, rt);
    const int32_t rv = (rt < V) ? rt : 0;
    r_ns = tb.rdst[rv];
    r_psi = tb.rpsi[rv];
    r_z = zrow[rv];
  }
  a.tok = V;
  a.ns = x;
  a.b = 0.f;
  a.zv = r.zb;
  float bk = r.zb + phi_x;  // blank keeps the state
  int32_t bt = V;
  if (better(ok, ot, bk, bt)) {
    bk = ok;
    bt = ot;
    a.tok = ot;
    a.ns = o_ns;
    a.b = o_psi - phi_x;
    a.zv = o_z;
  }
  if (better(rk, rt, bk, bt)) {
    a.tok = rt;
    a.ns = r_ns;
    a.b = r_psi - phi_x;
    a.zv = r_z;
  }
  return true;
}

// eval_chain_wide with two children per lane, or four (when NSMAX allows it)
// when the chain has more than 128.
template <int PER, int NSMAX = 2, class GR = SGraph>
__device__ __forceinline__ bool eval_chain_any(const GR& G, const Tables<PER>& tb,
                                               const float* zrow, uint32_t* marks,
                                               const RowShape<PER>& rs, int32_t x, float phi_x,
                                               const int32_t (&fl)[kChainMax],
                                               const int32_t (&nl)[kChainMax], int32_t levels,
                                               const RowSum& r, const LaneTop* top, int32_t V,
                                               Answer& a) {
  int32_t total = 0;
#pragma unroll
  for (int i = 0; i < kChainMax; ++i) total += nl[i];
  if (NSMAX < 4 || total <= 128)
    return eval_chain_wide<PER, 2, GR>(G, tb, zrow, marks, rs, x, phi_x, fl, nl, levels, r, top,
                                       V, a);
  return eval_chain_wide<PER, 4, GR>(G, tb, zrow, marks, rs, x, phi_x, fl, nl, levels, r, top, V,
                                     a);
}


// The step from state x from the packed state records in LDS. The children of
// the states on x's suffix chain (x, link(x), ... up to four non-root states,
// at most 64 children in all) are the override candidates, one per lane; a
// child is dropped when a deeper chain state has a child on the same class.
// Every other token takes its root move: the row's best root move unless its
// class is overridden, else the best unmarked one from the lanes' two best
// root moves (top) or a masked scan of the row. The blank keeps the state.
// Returns false, with no output, on any other shape (a state or child without
// a usable record, a class of more than three members, too many children);
// longer is set when the reason is a chain of more than four states.
template <int PER, int NSMAX = 2, class GR = SGraph>
__device__ __forceinline__ bool eval_walk(const GR& G, const Tables<PER>& tb,
                                          const float* zrow, uint32_t* marks,
                                          const RowShape<PER>& rs, int32_t x, const RowSum& r,
                                          const LaneTop* top, int32_t V, Answer& a,
                                          bool& longer) {
  const int lane = __lane_id();
  int32_t fc, nc, lnk;
  float phi_x;
  if (!G.srec(x, fc, nc, lnk, phi_x)) return false;
  int32_t f0 = 0, f1 = 0, f2 = 0, f3 = 0, n0 = 0, n1 = 0, n2 = 0, n3 = 0, levels = 0;
  if (x != 0) {  // the root's children are the dense root row
    f0 = fc;
    n0 = nc;
    levels = 1;
    while (lnk != 0) {
      if (levels == 4) {
        longer = true;
        return false;
      }
      float phi_unused;
      if (!G.srec(lnk, fc, nc, lnk, phi_unused)) return false;
      if (levels == 1) { f1 = fc; n1 = nc; }
      else if (levels == 2) { f2 = fc; n2 = nc; }
      else { f3 = fc; n3 = nc; }
      ++levels;
    }
  }
  const int32_t s1 = n0, s2 = s1 + n1, s3 = s2 + n2, total = s3 + n3;
  if (total > 64) {  // more children than lanes: two per lane
    const int32_t fl[kChainMax] = {f0, f1, f2, f3, 0, 0, 0, 0};
    const int32_t nl[kChainMax] = {n0, n1, n2, n3, 0, 0, 0, 0};
    return eval_chain_any<PER, NSMAX, GR>(G, tb, zrow, marks, rs, x, phi_x, fl, nl, levels, r, top,
                                      V, a);
  }

  // best override candidate (none when the chain has no children)
  float ok = kNegInf, o_psi = 0.f, o_z = 0.f;
  int32_t ot = INT_MAX, o_ns = 0;
  bool over = false, root_lost = false;
  if (total > 0) {
    const bool in = lane < total;
    const int32_t lv = (lane >= s1) + (lane >= s2) + (lane >= s3);
    const int32_t fb = lv == 0 ? f0 : lv == 1 ? f1 : lv == 2 ? f2 : f3;
    const int32_t sb = lv == 0 ? 0 : lv == 1 ? s1 : lv == 2 ? s2 : s3;
    const int32_t y = in ? fb + (lane - sb) : 0;
    uint32_t c0 = 0u, c1 = 0u, c2 = 0x80000000u;
    if (in && y < G.nhot) {
      c0 = G.w0[y];
      c1 = G.w1[y];
      c2 = G.w2[y];
    } else if constexpr (GR::kFar) {
      if (in && G.nhot > 0) {  // the arena's packed record
        const uint32_t* g = G.A->state_rec + 3 * ((int64_t)G.off + y);
        c0 = gload(g);
        c1 = gload(g + 1);
        c2 = gload(g + 2);
      }
    }
    const int32_t mc = (int32_t)(c2 & 0xffu);
    if (__ballot(in && ((c2 >> 31) != 0u || mc > 3)) != 0ull) return false;
    const int32_t lab = (int32_t)((c2 >> 16) & 0x7fffu);
    const int32_t ms = in ? (int32_t)(c1 >> 16) : 0;
    const float py = G.vpsi[c0 >> 24];
    const int32_t t0 = tb.cls_tok[ms];
    const int32_t t1 = tb.cls_tok[ms + (mc > 1 ? 1 : 0)];
    const int32_t t2 = tb.cls_tok[ms + (mc > 2 ? 2 : (mc > 1 ? 1 : 0))];
    const float z0 = zrow[t0], z1 = zrow[t1], z2 = zrow[t2];
    float kb = z0 + py, zb_ = z0;
    int32_t tk = t0;
    const float k1 = z1 + py, k2 = z2 + py;
    if (k1 > kb) { kb = k1; tk = t1; zb_ = z1; }  // members ascend: ties keep the lower
    if (k2 > kb) { kb = k2; tk = t2; zb_ = z2; }
    // A class that a deeper chain state (a lower level) also has is shadowed.
    // The best of all children is the answer unless it is shadowed: a
    // shadowing child has the same tokens, and among equal keys and tokens
    // the lowest lane (the deepest level) wins the argmax. Only a shadowed
    // winner needs the class-by-class resolution.
    int32_t wl = wave_argmax_dpp(in ? kb : kNegInf, in ? tk : INT_MAX, ok, ot);
    if (levels > 1) {
      const int32_t lw = rl(lab, wl), vw = rl(lv, wl);
      if (__ballot(in && lab == lw && lv < vw) != 0ull) {
        const int32_t last = levels == 2 ? s1 : (levels == 3 ? s2 : s3);
        bool take = in;
        for (int32_t j = 0; j < last; ++j) {
          const int32_t cj = __builtin_amdgcn_readlane(lab, j);
          const int32_t lvj = (j >= s1) + (j >= s2) + (j >= s3);
          take = take && !(lvj < lv && cj == lab);
        }
        wl = wave_argmax_dpp(take ? kb : kNegInf, take ? tk : INT_MAX, ok, ot);
      }
    }
    o_ns = rl(y, wl);
    o_psi = rlf(py, wl);
    o_z = rlf(zb_, wl);
    // every chain child's class overrides its root move (a shadowed class is
    // also a deeper child's)
    over = __ballot(in && lab == r.r1_cls) != 0ull;
    // the remaining root moves have keys at most r.ymax: when the best child
    // or the blank is above it, no root move can win
    if (over && (ok > r.ymax || r.zb + phi_x > r.ymax)) {
      over = false;
      root_lost = true;
    }
    if (over) {
      marks_clear<PER>(marks);
      if (in) mark(marks, lab);
      marks_fence();
    }
  }

  // best root move whose class is not overridden
  float rk = root_lost ? kNegInf : r.ymax;
  int32_t rt = r.r1_tok, r_ns = r.r1_dst;
  float r_psi = r.r1_psi, r_z = r.r1_z;
  if (over) {
    if (!(top && root_excluding<PER>(tb, zrow, marks, *top, rk, rt)))
      root_scan<PER>(tb, zrow, marks, rs, rk, rt);
    const int32_t rv = (rt < V) ? rt : 0;
    r_ns = tb.rdst[rv];
    r_psi = tb.rpsi[rv];
    r_z = zrow[rv];
  }
  a.tok = V;
  a.ns = x;
  a.b = 0.f;
  a.zv = r.zb;
  float bk = r.zb + phi_x;  // blank keeps the state
  int32_t bt = V;
  if (better(ok, ot, bk, bt)) {
    bk = ok;
    bt = ot;
    a.tok = ot;
    a.ns = o_ns;
    a.b = o_psi - phi_x;
    a.zv = o_z;
  }
  if (better(rk, rt, bk, bt)) {
    a.tok = rt;
    a.ns = r_ns;
    a.b = r_psi - phi_x;
    a.zv = r_z;
  }
  return true;
}

// eval_walk for chains of up to kChainMax non-root states (and the child
// sets of eval_chain_wide). Returns false, with no output, on any other shape.
template <int PER, int NSMAX = 2, class GR = SGraph>
__device__ __forceinline__ bool eval_walk2(const GR& G, const Tables<PER>& tb,
                                           const float* zrow, uint32_t* marks,
                                           const RowShape<PER>& rs, int32_t x, const RowSum& r,
                                           const LaneTop* top, int32_t V, Answer& a) {
  constexpr int kLv = kChainMax;
  int32_t fc, nc, lnk;
  float phi_x;
  if (x == 0 || !G.srec(x, fc, nc, lnk, phi_x)) return false;
  int32_t fl[kLv], nl[kLv];
  fl[0] = fc;
  nl[0] = nc;
  int32_t levels = 1;
#pragma unroll
  for (int i = 1; i < kLv; ++i) {
    fl[i] = 0;
    nl[i] = 0;
    if (lnk != 0) {
      float phi_unused;
      if (!G.srec(lnk, fc, nc, lnk, phi_unused)) return false;
      fl[i] = fc;
      nl[i] = nc;
      ++levels;
    }
  }
  if (lnk != 0) return false;
  return eval_chain_any<PER, NSMAX, GR>(G, tb, zrow, marks, rs, x, phi_x, fl, nl, levels, r, top,
                                    V, a);
}

// The boosted step from state x: from the LDS records when they apply, else
// the general path.
template <int PER, int NSMAX = 2, class GR = SGraph>
__device__ __forceinline__ Answer eval_state(const GR& G, const Tables<PER>& tb,
                                             const float* zrow, uint32_t* marks,
                                             const RowShape<PER>& rs, int32_t x, const RowSum& r,
                                             const LaneTop* top, int32_t V) {
  Answer a;
  bool longer = false;
  if (eval_walk<PER, NSMAX, GR>(G, tb, zrow, marks, rs, x, r, top, V, a, longer)) return a;
  // only a longer chain is a shape eval_walk2 takes that eval_walk does not
  if (longer && eval_walk2<PER, NSMAX, GR>(G, tb, zrow, marks, rs, x, r, top, V, a)) return a;
  return eval_general<PER, GR>(G, tb, zrow, marks, rs, x, r, top, V);
}

// log(sum(exp(z))) of a row from this lane's elements and their maximum:
// max over the wave, then the sum of exp2 terms over the wave.
template <int PER>
__device__ __forceinline__ float lse_of(const float* cur, float zmax) {
  zmax = wave_max_dpp(zmax);
  const float mL = zmax * kLog2e;
  float se = 0.f;
#pragma unroll
  for (int j = 0; j < PER; ++j) se += __builtin_amdgcn_exp2f(__builtin_fmaf(cur[j], kLog2e, -mL));
  se = wave_sum_dpp(se);
  return zmax + __logf(se);
}

// State-independent part of a step on a row held in registers (raw[j] as
// loaded): copies the row to zrow (LDS) and summarises it. rp holds this
// lane's root-move psi (-inf for blank and masked lanes).
template <int PER, bool kTop2 = false>
__device__ __forceinline__ RowSum row_summary(float* zrow, const Tables<PER>& tb, const float* raw,
                                              const float* rp, const RowShape<PER>& rs, int32_t V,
                                              bool need_lse, LaneTop* top = nullptr) {
  const int lane = __lane_id();
  float cur[PER];
#pragma unroll
  for (int j = 0; j < PER - 1; ++j) {
    zrow[64 * j + lane] = raw[j];
    cur[j] = raw[j];
  }
  zrow[rs.last_idx] = raw[PER - 1];  // repeated lanes rewrite equal values
  cur[PER - 1] = rs.last_ok ? raw[PER - 1] : kNegInf;
  RowSum r;
  r.zb = rlf(raw[PER - 1], PER > 1 ? 63 : V);
  asm volatile("" ::: "memory");

  // best root move per lane: strict > keeps the lowest chunk, hence the lowest index
  float zmax = kNegInf, yb = kNegInf, y2 = kNegInf;
  int32_t jb = 0, j2 = -1;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    zmax = __builtin_fmaxf(zmax, cur[j]);
    const float yj = cur[j] + rp[j];
    const bool gt = yj > yb;
    if (kTop2) {  // the runner-up, in the same (key, index) order
      const bool gt2 = yj > y2;
      y2 = gt ? yb : (gt2 ? yj : y2);
      j2 = gt ? (yb > kNegInf ? jb : -1) : (gt2 ? j : j2);
    }
    yb = gt ? yj : yb;
    jb = gt ? j : jb;
  }
  const int32_t idx = (jb == PER - 1) ? rs.last_idx : 64 * jb + lane;
  if (kTop2) {
    top->i1 = (yb > kNegInf) ? idx : kNoTok;
    top->i2 = (j2 < 0 || !(y2 > kNegInf)) ? kNoTok : ((j2 == PER - 1) ? rs.last_idx : 64 * j2 + lane);
    top->k1 = yb;
    top->k2 = y2;
  }
  wave_argmax_dpp(yb, idx, r.ymax, r.r1_tok);
  if (r.r1_tok >= V) r.r1_tok = 0;  // only with -inf / nan logits: keep indices in range
  const int32_t c16 = tb.cls[r.r1_tok];
  r.r1_cls = c16 == 0xffff ? -1 : c16;
  r.r1_dst = tb.rdst[r.r1_tok];
  r.r1_psi = tb.rpsi[r.r1_tok];
  r.r1_z = zrow[r.r1_tok];
  r.lse = need_lse ? lse_of<PER>(cur, zmax) : 0.f;  // warm-up rows only need the state
  return r;
}

// The row's normaliser from this lane's elements in row_summary's layout
// (from registers as loaded, or from the row in LDS).
template <int PER>
__device__ __forceinline__ float row_lse(const float* raw, const RowShape<PER>& rs) {
  float cur[PER];
  float zmax = kNegInf;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    cur[j] = (j < PER - 1 || rs.last_ok) ? raw[j] : kNegInf;
    zmax = __builtin_fmaxf(zmax, cur[j]);
  }
  return lse_of<PER>(cur, zmax);
}

template <int PER>
__device__ __forceinline__ float row_lse_lds(const float* zrow, const RowShape<PER>& rs) {
  const int lane = __lane_id();
  float raw[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) raw[j] = zrow[(j < PER - 1) ? 64 * j + lane : rs.last_idx];
  return row_lse<PER>(raw, rs);
}

// The step from state s on a summarised row (zrow in LDS).
template <int PER, int NSMAX = 2, class GR = SGraph>
__device__ __forceinline__ Answer step_from(const GR& G, const Tables<PER>& tb,
                                            const float* zrow, uint32_t* marks,
                                            const RowShape<PER>& rs, const RowSum& r, int32_t s,
                                            int mode, int32_t V, const LaneTop* top = nullptr) {
  if (mode != 1) {
    Answer a;
    const bool blank = !better(r.ymax, r.r1_tok, r.zb, V);
    a.tok = blank ? V : r.r1_tok;
    a.ns = s;
    a.b = 0.f;
    a.zv = blank ? r.zb : r.ymax;
    return a;
  }
  return eval_state<PER, NSMAX, GR>(G, tb, zrow, marks, rs, s, r, top, V);
}

// One complete step on a row held in registers.
template <int PER>
__device__ __forceinline__ Answer full_step(const SGraph& G, const Tables<PER>& tb, float* zrow,
                                            uint32_t* marks, const float* raw,
                                            const float* rp, const RowShape<PER>& rs, int32_t s,
                                            int mode, int32_t V, bool need_lse, float& lse) {
  const RowSum r = row_summary<PER>(zrow, tb, raw, rp, rs, V, need_lse);
  lse = r.lse;
  return step_from<PER>(G, tb, zrow, marks, rs, r, s, mode, V);
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

// The LDS tables of fill_tables and fill_state_hot in two halves: the loads
// into registers, then the stores. A kernel issues the loads before its
// logit rows, so that the stores (loads complete in issue order) wait for the
// tables only, not for the rows coming from HBM.
template <int PER, int NT, int HOT>
struct FillRegs {
  static constexpr int KT = (64 * PER + NT - 1) / NT;
  static constexpr int KH = (HOT + NT - 1) / NT;
  float rpsi[KT];
  int32_t rdst[KT], cls[KT], cptr[KT], ctok[KT];
  uint32_t w0[KH], w1[KH], w2[KH];
  float vt;
};

template <int PER, int NT, int HOT>
__device__ __forceinline__ void fill_gather(FillRegs<PER, NT, HOT>& f, const ArenaView& A,
                                            int32_t m, int mode) {
  const int32_t V1 = A.V1, V = V1 - 1;
  const float* gpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* gdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;
#pragma unroll
  for (int k = 0; k < f.KT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    f.rpsi[k] = (i < V) ? (mode == 1 ? gpsi[i] : 0.f) : kNegInf;
    f.rdst[k] = (i < V && mode == 1) ? gdst[i] : 0;
    f.cls[k] = (i < V1) ? A.class_map[i] : -1;
    f.cptr[k] = (i < V1) ? A.cls_ptr[i] : 0;
    f.ctok[k] = (i < V) ? A.cls_tok[i] : 0;
  }
}

// The state records of the first nhot states of the model at off, and its
// psi / phi value tables.
template <int PER, int NT, int HOT>
__device__ __forceinline__ void fill_gather_hot(FillRegs<PER, NT, HOT>& f, const ArenaView& A,
                                                int32_t m, int32_t off, int32_t nhot) {
  const uint32_t* src = A.state_rec + 3 * (int64_t)off;
#pragma unroll
  for (int k = 0; k < f.KH; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    const bool in = i < nhot;
    f.w0[k] = in ? src[3 * i] : 0u;
    f.w1[k] = in ? src[3 * i + 1] : 0u;
    f.w2[k] = in ? src[3 * i + 2] : 0u;
  }
  f.vt = (nhot > 0 && threadIdx.x < 512) ? A.value_tab[512 * (int64_t)m + threadIdx.x] : 0.f;
}

template <int PER, int NT, int HOT>
__device__ __forceinline__ void fill_scatter(const FillRegs<PER, NT, HOT>& f, Tables<PER>& tb) {
#pragma unroll
  for (int k = 0; k < f.KT; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < 64 * PER) {
      tb.rpsi[i] = f.rpsi[k];
      tb.rdst[i] = f.rdst[k];
      tb.cls[i] = f.cls[k] < 0 ? (uint16_t)0xffff : (uint16_t)f.cls[k];
      tb.cls_ptr[i] = (uint16_t)f.cptr[k];
      tb.cls_tok[i] = (uint16_t)f.ctok[k];
    }
  }
}

template <int PER, int NT, int HOT>
__device__ __forceinline__ void fill_scatter_hot(const FillRegs<PER, NT, HOT>& f,
                                                 StateHot<HOT>& h, int32_t nhot) {
#pragma unroll
  for (int k = 0; k < f.KH; ++k) {
    const int32_t i = k * NT + (int32_t)threadIdx.x;
    if (i < nhot) {
      h.w0[i] = f.w0[k];
      h.w1[i] = f.w1[k];
      h.w2[i] = f.w2[k];
    }
  }
  if (nhot > 0 && threadIdx.x < 512) {
    if (threadIdx.x < 256) h.vpsi[threadIdx.x] = f.vt;
    else h.vphi[threadIdx.x - 256] = f.vt;
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

// Sequential recompute from state x over rows [t, t_end), stopping after the
// first row whose new state equals old_state(t): from there on the stored
// outputs already follow the exact trajectory. With b2 given, rows are
// prefetched two ahead in three buffers (b0, b1 hold or are loading rows t and
// t+1, clamped to t_end - 1); with b2 null, one ahead in two buffers (b0 holds
// row t). emit(t, answer, lse) writes a row. Returns true when the
// trajectories met; x is the exact state after the last recomputed row.
template <class Ld, int PER, bool kTwoAhead, class OldFn, class EmitFn>
__device__ __forceinline__ bool repair_run(const SGraph& G, const Tables<PER>& tb, float* zrow,
                                           uint32_t* marks, const float* rp,
                                           const RowShape<PER>& rs,
                                           const typename Ld::T* col, int64_t tstride,
                                           int32_t t, int32_t t_end, int32_t& x, int mode,
                                           int32_t V, float* b0, float* b1, float* b2,
                                           OldFn old_state, EmitFn emit) {
  constexpr int kAhead = kTwoAhead ? 2 : 1;
  auto sub = [&](const float* cur, float* pf, int32_t tt) -> bool {
    const int32_t tn = (tt + kAhead < t_end) ? tt + kAhead : t_end - 1;
    load_row<Ld, PER>(pf, col + (int64_t)tn * tstride, rs);
    float lse;
    const Answer a = full_step<PER>(G, tb, zrow, marks, cur, rp, rs, x, mode, V, true, lse);
    const int32_t old = old_state(tt);
    emit(tt, a, lse);
    x = __builtin_amdgcn_readfirstlane(a.ns);
    return x == old;
  };
  if constexpr (kTwoAhead) {
    for (; t < t_end; t += 3) {
      if (sub(b0, b2, t)) return true;
      if (t + 1 >= t_end) break;
      if (sub(b1, b0, t + 1)) return true;
      if (t + 2 >= t_end) break;
      if (sub(b2, b1, t + 2)) return true;
    }
  } else {
    for (; t < t_end; t += 2) {
      if (sub(b0, b1, t)) return true;
      if (t + 1 >= t_end) break;
      if (sub(b1, b0, t + 1)) return true;
    }
  }
  return false;
}

template <class Ld, int PER>
__global__ __launch_bounds__(Shape<PER>::NT) void greedy_seg_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score, uint32_t spin_limit) {
  constexpr int W = Shape<PER>::W;
  constexpr int NT = Shape<PER>::NT;
  constexpr int HOT = SegLds<PER>::HOT;
  __shared__ SegLds<PER> S;
  lds_poison(&S, sizeof(S));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int32_t b = blockIdx.x % B;
  const int32_t g = blockIdx.x / B;
  const typename Ld::T* col = logits + (int64_t)b * stride;  // row t of stream b: col + t*tstride
  const int64_t tstride = (int64_t)B * stride;

  const int32_t m = model_ids[b];
  const int32_t s0 = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s0, off, n);

  const RowShape<PER> rs(V1);
  const int32_t segi = g * W + w;
  const int32_t t0 = segi * L;
  const int32_t t1 = (t0 + L < T) ? t0 + L : T;
  const bool exact_start = (segi == 0) || mode != 1;
  const int32_t tw = exact_start ? t0 : (t0 - kWarm > 0 ? t0 - kWarm : 0);
  // the first row is in flight while the tables are filled
  float ra[PER], rb[PER];
  if (t0 < t1) load_row<Ld, PER>(ra, col + (int64_t)tw * tstride, rs);

  fill_tables<PER, NT>(S.tab, A, m, mode);
  const int32_t nhot = (mode == 1) ? (n < HOT ? n : HOT) : 0;
  fill_state_hot<HOT, NT>(S.hot, A, m, off, nhot);
  if (threadIdx.x < W) {
    S.fin_ready[threadIdx.x] = 0;
    S.fin_state[threadIdx.x] = 0;
  }
  if (threadIdx.x == 0) S.abort_flag = 0;
  __syncthreads();

  const SGraph Gr(A, off, nhot, S.hot, S.tab);
  float* zrow = S.zbuf[w];
  uint32_t* marks = S.marks[w];
  float rp[PER];
  root_psi_regs<PER>(rp, S.tab, rs);

  const int32_t start = (mode == 1) ? (segi == 0 ? s0 : 0)
                                    : unbiased_state(mode, s0 == TB_STATE_TIMEOUT);

  // ---- main pass over the segment (with warm-up rows)
  int32_t s = start;
  int32_t assumed = start;
  if (t0 < t1) {
    // Two row buffers used in turn; the prefetch is unconditional (the last
    // row of the segment is read again at the end) so that the wait for the
    // current row can leave the next row's loads in flight.
    int32_t o_tok = 0, o_st = 0;
    float o_sc = 0.f;
    auto step = [&](const float* cur, float* nxt, int32_t t) {
      const int32_t tn = (t + 1 < t1) ? t + 1 : t;
      load_row<Ld, PER>(nxt, col + (int64_t)tn * tstride, rs);
      if (t == t0) assumed = s;
      float lse;
      const Answer a =
          full_step<PER>(Gr, S.tab, zrow, marks, cur, rp, rs, s, mode, V, t >= t0, lse);
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
    for (int32_t t = tw; t < t1; t += 2) {
      step(ra, rb, t);
      if (t + 1 < t1) step(rb, ra, t + 1);
    }
  }

  // ---- hand the exact state along the segments of this workgroup
  // The first row a repair would need is loaded while waiting.
  const bool may_repair = w > 0 && t0 < t1 && mode == 1;
  if (may_repair) load_row<Ld, PER>(ra, col + (int64_t)t0 * tstride, rs);
  int32_t fin = s;
  if (w > 0) {
    uint32_t spins = 0;
    while (lds_ld(&S.fin_ready[w - 1]) == 0) {
      if (lds_ld(&S.abort_flag) || ++spins > spin_limit) {
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
      // Stored states: LDS for the first kTraj rows, else read back by the
      // lane that wrote them in the main pass (row i of the segment: lane i & 63).
      auto old_state = [&](int32_t t) -> int32_t {
        const int32_t i = t - t0;
        if (i < kTraj) return __builtin_amdgcn_readfirstlane(S.traj[w][i]);
        return rl(out_state[(int64_t)t * B + b], i & 63);
      };
      auto emit = [&](int32_t t, const Answer& a, float lse) {
        if (lane == ((t - t0) & 63)) {
          const int64_t oi = (int64_t)t * B + b;
          out_tok[oi] = a.tok;
          out_state[oi] = a.ns;
          out_score[oi] = (a.zv - lse) + a.b;
        }
      };
      int32_t x = exact;
      const bool met =
          repair_run<Ld, PER, false>(Gr, S.tab, zrow, marks, rp, rs, col, tstride, t0, t1,
                                     x, mode, V, ra, rb, nullptr, old_state, emit);
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

// Repairs the workgroup boundaries of each stream after greedy_seg_kernel,
// boundaries in order: from the exact state before a boundary, recompute
// until the stored trajectory is met. Four waves fill the tables, wave 0
// repairs. Writes the carry.
constexpr int kFixThreads = 256;
constexpr int kFixHot = 6144;

template <int PER>
struct alignas(16) FixLds {
  Tables<PER> tab;
  float zrow[64 * PER];
  uint32_t marks[2 * PER];
  StateHot<kFixHot> hot;
};

template <class Ld, int PER>
__global__ __launch_bounds__(kFixThreads) void greedy_fix_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    int32_t G, int32_t L, int32_t W, const int32_t* __restrict__ model_ids,
    int32_t* __restrict__ states, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  __shared__ FixLds<PER> S;
  lds_poison(&S, sizeof(S));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int lane = __lane_id();
  const int32_t b = blockIdx.x;
  const int32_t m = model_ids[b];
  const typename Ld::T* col = logits + (int64_t)b * stride;
  const int64_t tstride = (int64_t)B * stride;
  // The carried state was consumed by the main kernel; streams that are not
  // biased, or whose carried state was invalid, have exact (unboosted)
  // segment starts and need no repair.
  const bool biased = m >= 0 && m < A.n_models;
  bool timed_out = false;
  if (biased) {
    const RowShape<PER> rs(V1);
    float ra[PER], rb[PER], rc[PER];
    const int32_t first = W * L;  // the first workgroup boundary (< T)
    if (threadIdx.x < 64) {
      load_row<Ld, PER>(ra, col + (int64_t)first * tstride, rs);
      load_row<Ld, PER>(rb, col + (int64_t)(first + 1 < T ? first + 1 : first) * tstride, rs);
    }
    const int32_t off = A.model_off[m], n = A.model_n[m];
    const int32_t nhot = n < kFixHot ? n : kFixHot;
    fill_tables<PER, kFixThreads>(S.tab, A, m, 1);
    fill_state_hot<kFixHot, kFixThreads>(S.hot, A, m, off, nhot);
    __syncthreads();
    if (threadIdx.x >= 64) return;  // no barrier follows
    const SGraph Gr(A, off, nhot, S.hot, S.tab);
    float rp[PER];
    root_psi_regs<PER>(rp, S.tab, rs);
    auto old_state = [&](int32_t t) -> int32_t {
      return __builtin_amdgcn_readfirstlane(out_state[(int64_t)t * B + b]);
    };
    auto emit = [&](int32_t t, const Answer& a, float lse) {
      if (lane == 0) {
        const int64_t oi = (int64_t)t * B + b;
        out_tok[oi] = a.tok;
        out_state[oi] = a.ns;
        out_score[oi] = (a.zv - lse) + a.b;
      }
    };
    int32_t done = 0;  // rows before this are exact
    for (int32_t gg = 1; gg < G; ++gg) {
      const int32_t tb0 = gg * W * L;
      if (tb0 >= T) break;
      if (done > tb0) continue;  // an earlier repair already ran past this boundary
      if (gg > 1) {
        load_row<Ld, PER>(ra, col + (int64_t)tb0 * tstride, rs);
        load_row<Ld, PER>(rb, col + (int64_t)(tb0 + 1 < T ? tb0 + 1 : tb0) * tstride, rs);
      }
      int32_t x = __builtin_amdgcn_readfirstlane(out_state[(int64_t)(tb0 - 1) * B + b]);
      if (x < 0 || x >= n) {
        // a timed-out main kernel (-3): no exact state reaches this boundary,
        // so none of the following rows can be repaired; they are marked
        timed_out = x == kStateTimeout;
        if (timed_out)
          for (int32_t t = tb0 + lane; t < T; t += 64) out_state[(int64_t)t * B + b] = kStateTimeout;
        break;
      }
      // the rows up to the meeting point are recomputed; find where it was
      int32_t t_stop = tb0;
      auto emit_track = [&](int32_t t, const Answer& a, float lse) {
        emit(t, a, lse);
        t_stop = t + 1;
      };
      repair_run<Ld, PER, true>(Gr, S.tab, S.zrow, S.marks, rp, rs, col, tstride, tb0, T,
                                x, 1, V, ra, rb, rc, old_state, emit_track);
      done = t_stop;
    }
  }
  if (lane == 0 && threadIdx.x < 64)
    states[b] = timed_out ? kStateTimeout : out_state[(int64_t)(T - 1) * B + b];
}

// Short calls (T <= W steps, a streaming chunk). Wave w owns row w: it
// summarises the row (best root moves, row copy in LDS), then evaluates the
// step of row w from a guessed start state x_w, all rows in parallel:
//
//   x_0 = the carried state (exact);
//   x_w (w >= 1) starts as the target of row w-1's best root move, the move
//   taken from most states; after each of kSpecRounds rounds, x_w <- the
//   state reached by row w-1's step from x_{w-1} (rows whose guess did not
//   change are not evaluated again).
//
// Wave 0 then walks the rows in order from the exact carried state: a row
// whose guess equals the exact state keeps its answer (and so does the run of
// rows after it whose guesses follow the answers), any other row is
// evaluated again from the exact state. Mostly the guesses hold, so the
// sequential part is a few comparisons plus the rows inside long phrase
// matches. Every round costs about one evaluation and saves about one
// walker evaluation in the stream with the longest match: three rounds
// measured best on 128 streams of 16-row chunks (two and four were slower).
// While wave 0 walks, the other waves take the rows' normalisers.
//
// FAR: for arenas whose models are larger than the LDS records on average,
// states beyond them are read from the arena's packed records and suffix
// chains with up to 256 children (four per lane) stay on the fast path; the
// other instance, which every model that fits runs, reads such states through
// the general path. Both give the same results.
constexpr int kSpecRounds = 3;

template <class Ld, int PER, bool FAR>
__global__ __launch_bounds__(Shape<PER>::NT) void greedy_chunk_kernel(
    ArenaView A, const typename Ld::T* __restrict__ logits, int32_t T, int32_t B, int64_t stride,
    const int32_t* __restrict__ model_ids, int32_t* __restrict__ states,
    int32_t* __restrict__ out_tok, int32_t* __restrict__ out_state,
    float* __restrict__ out_score) {
  constexpr int NT = Shape<PER>::NT;
  constexpr int HOT = SegLds<PER>::HOT;
  constexpr int NSMAX = FAR ? 4 : 2;
  __shared__ SegLds<PER> S;
  lds_poison(&S, sizeof(S));
  const int32_t V1 = A.V1, V = V1 - 1;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = __lane_id();
  const int32_t b = blockIdx.x;
  const typename Ld::T* col = logits + (int64_t)b * stride;
  const int64_t tstride = (int64_t)B * stride;

  const int32_t m = model_ids[b];
  const int32_t s0 = states[b];
  int32_t off = 0, n = 0;
  const int mode = resolve_stream(A, m, s0, off, n);
  const RowShape<PER> rs(V1);
  const bool own = w < T;  // this wave has a row
  const int32_t nhot = (mode == 1) ? (n < HOT ? n : HOT) : 0;
  // the tables' loads, then the row's (from HBM, the slowest), then the
  // tables' stores while the row is still on its way
  FillRegs<PER, NT, HOT> fr;
  fill_gather<PER, NT, HOT>(fr, A, m, mode);
  fill_gather_hot<PER, NT, HOT>(fr, A, m, off, nhot);
  asm volatile("" ::: "memory");
  float raw[PER];
  if (own) load_row<Ld, PER>(raw, col + (int64_t)w * tstride, rs);
  fill_scatter<PER, NT, HOT>(fr, S.tab);
  fill_scatter_hot<PER, NT, HOT>(fr, S.hot, nhot);
  __syncthreads();

  RowSum r = {};
  LaneTop top = {kNoTok, kNoTok, kNegInf, kNegInf};
  if (own) {
    float rp[PER];
    root_psi_regs<PER>(rp, S.tab, rs);
    // the normaliser is taken later, off the sequential part
    r = row_summary<PER, true>(S.zbuf[w], S.tab, raw, rp, rs, V, false, &top);
    if (lane == 0) S.rsum[w] = r;
    S.ltop[w][lane] = (uint32_t)top.i1 | ((uint32_t)top.i2 << 16);
  }
  __syncthreads();

  const SGraphT<FAR> Gr(A, off, nhot, S.hot, S.tab);
  const int32_t fixed = unbiased_state(mode, s0 == TB_STATE_TIMEOUT);
  int32_t x;  // guessed start state of row w
  if (mode != 1) {
    x = fixed;  // unbiased rows: the step does not depend on the state
  } else if (w == 0) {
    x = s0;
  } else {
    x = own ? __builtin_amdgcn_readfirstlane(S.rsum[w - 1].r1_dst) : 0;
  }
  Answer a = {0, 0, 0.f, 0.f};
  bool need = own;
#pragma unroll
  for (int round = 0; round < kSpecRounds; ++round) {
    if (need)
      a = step_from<PER, NSMAX>(Gr, S.tab, S.zbuf[w], S.marks[w], rs, r, x, mode, V, &top);
    if (own && lane == 0) lds_st(&S.spec_ns[round & 1][w], a.ns);
    __syncthreads();
    if (round + 1 < kSpecRounds) {
      int32_t xn = x;
      if (own && w > 0 && mode == 1)
        xn = __builtin_amdgcn_readfirstlane(lds_ld(&S.spec_ns[round & 1][w - 1]));
      need = xn != x;
      x = xn;
    }
  }
  if (own && lane == 0) {
    S.spec_x[w] = x;
    S.spec_ans[w] = make_int4(a.tok, a.ns, __float_as_int(a.b), __float_as_int(a.zv));
  }
  __syncthreads();
  if (w != 0) {
    // the normalisers while wave 0 walks: every other wave its own row (from
    // registers), the last wave also row 0 (from LDS)
    if (own) {
      const float l = row_lse<PER>(raw, rs);
      if (lane == 0) S.lse[w] = l;
    }
    if (w == Shape<PER>::W - 1 && T > 0) {
      const float l = row_lse_lds<PER>(S.zbuf[0], rs);
      if (lane == 0) S.lse[0] = l;
    }
    __syncthreads();
    return;
  }

  // The walk is the sequential part: its instructions go first on this SIMD
  // (the other waves' normalisers take the cycles it leaves idle).
  __builtin_amdgcn_s_setprio(3);
  // Lane t holds row t's guess, answer and summary. A run of rows whose
  // guesses follow each other's answers is exact as soon as its first guess
  // is: link says that row t's answer is row t+1's guess, and the walk jumps
  // over such runs. Any other row is evaluated again from the exact state.
  int4 ans = make_int4(0, 0, 0, 0);
  int32_t gx = INT_MIN;
  RowSum rl_ = {};
  if (lane < T) {
    ans = S.spec_ans[lane];
    gx = S.spec_x[lane];
    rl_ = S.rsum[lane];
  }
  const int32_t gx_next = __shfl_down(gx, 1, 64);
  const uint64_t stop = ~__ballot(lane + 1 < T && gx_next == ans.y);  // bit T-1 is set
  int32_t s = (mode == 1) ? s0 : fixed;
  int32_t t = 0;
  while (t < T) {
    if (rl(gx, t) == s) {
      const int32_t u = t + (int32_t)__builtin_ctzll(stop >> t);
      s = rl(ans.y, u);
      t = u + 1;
      continue;
    }
    const uint32_t tp = S.ltop[t][lane];
    RowSum rt;
    rt.zb = rlf(rl_.zb, t);
    rt.ymax = rlf(rl_.ymax, t);
    rt.lse = 0.f;
    rt.r1_psi = rlf(rl_.r1_psi, t);
    rt.r1_z = rlf(rl_.r1_z, t);
    rt.r1_tok = rl(rl_.r1_tok, t);
    rt.r1_cls = rl(rl_.r1_cls, t);
    rt.r1_dst = rl(rl_.r1_dst, t);
    const LaneTop tt = {(int32_t)(tp & 0xffffu), (int32_t)(tp >> 16), 0.f, 0.f};
    const Answer e =
        step_from<PER, NSMAX>(Gr, S.tab, S.zbuf[t], S.marks[0], rs, rt, s, mode, V, &tt);
    if (lane == t) ans = make_int4(e.tok, e.ns, __float_as_int(e.b), __float_as_int(e.zv));
    s = __builtin_amdgcn_readfirstlane(e.ns);
    ++t;
  }
  __syncthreads();  // the normalisers
  if (lane < T) {
    const int64_t oi = (int64_t)lane * B + b;
    out_tok[oi] = ans.x;
    out_state[oi] = ans.y;
    out_score[oi] = (__int_as_float(ans.w) - S.lse[lane]) + __int_as_float(ans.z);
  }
  if (lane == 0) states[b] = s;
}

// Launch geometry: workgroups per stream G and segment length L. Short calls
// (a streaming chunk) use one workgroup per stream and segments of a few
// rows; long calls use enough workgroups to cover the 256 CUs, with segments
// of at least kMinSeg rows.
template <int PER>
inline void seg_geometry(int32_t T, int32_t B, int32_t& G, int32_t& L) {
  constexpr int W = Shape<PER>::W;
  if (T <= W * kMinSeg) {
    G = 1;
    L = (T + W - 1) / W;
    if (L < 2) L = 2;
    return;
  }
  G = (256 + B - 1) / B;
  const int32_t gmax = T / (W * kMinSeg);
  if (G > gmax) G = gmax;
  if (G < 1) G = 1;
  L = (T + G * W - 1) / (G * W);
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
  if (T <= Shape<PER>::W) {
    const bool far = A.n_states > (int64_t)SegLds<PER>::HOT * A.n_models;
    if (far)
      hipLaunchKernelGGL((greedy_chunk_kernel<Ld, PER, true>), dim3(B), dim3(Shape<PER>::NT), 0,
                         st, A, static_cast<const TT*>(logits), T, B, stride, model_ids, states,
                         out_tok, out_state, out_score);
    else
      hipLaunchKernelGGL((greedy_chunk_kernel<Ld, PER, false>), dim3(B), dim3(Shape<PER>::NT), 0,
                         st, A, static_cast<const TT*>(logits), T, B, stride, model_ids, states,
                         out_tok, out_state, out_score);
    return hipGetLastError();
  }
  int32_t G, L;
  seg_geometry<PER>(T, B, G, L);
  const uint32_t spin = debug_spin_limit();
  hipLaunchKernelGGL((greedy_seg_kernel<Ld, PER>), dim3(B * G), dim3(Shape<PER>::NT), 0, st, A,
                     static_cast<const TT*>(logits), T, B, stride, G, L, model_ids, states,
                     out_tok, out_state, out_score, spin ? spin : kSpinLimit);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || G == 1) return e;
  hipLaunchKernelGGL((greedy_fix_kernel<Ld, PER>), dim3(B), dim3(kFixThreads), 0, st, A,
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
