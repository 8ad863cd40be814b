// Pieces shared by the wide-vocabulary step kernels (V+1 > 2048): a row is
// spread over one workgroup of kThreads threads, thread i holding tokens
// v = i + kThreads * j (j < TPV) with their class and root move in registers,
// and the classes overridden in the current state go to an LDS tag table.
#pragma once

#include <climits>

#include "device.hpp"

namespace tbias {
namespace wide {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kNegInf = -__builtin_huge_valf();

// Read-only load through the scalar cache (uniform address).
template <class T>
__device__ __forceinline__ T sld(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}

// The row length passes through an empty asm each time it is used, so that
// the compiler keeps the per-slot bounds tests where they are used instead of
// hoisting 2*TPV lane masks out of the row loop (they would not fit in SGPRs).
__device__ __forceinline__ int32_t opaque(int32_t x) {
  asm volatile("" : "+s"(x));
  return x;
}

// The workgroup's view of one stream's model: arena and the LDS tag table.
struct Ctx {
  const ArenaView* A;
  int32_t off;       // first global state of the model
  int mode;          // 1 biased, 0 model -1, -1 invalid model or state
  int32_t fixed;     // state written for unbiased streams
  int32_t cap;       // override list capacity
  uint32_t* omark;   // [V]: tag << 16 | list slot of an overridden class
  int32_t* olist_y;  // [cap] target state of an override
  float* olist_psi;  // [cap] its psi
  int32_t* nlist;    // list fill counter (LDS)
  uint32_t tag;
};

// Bytes of dynamic LDS a workgroup needs: the tag table and the override list.
__host__ __device__ inline size_t lds_bytes(const ArenaView& A) {
  const int32_t cap = A.max_override > 0 ? A.max_override : 1;
  return 4 * (size_t)(A.V1 - 1) + 8 * (size_t)cap;
}

__device__ __forceinline__ Ctx make_ctx(const ArenaView& A, int32_t off, int mode, int32_t fixed,
                                        int32_t* nlist, unsigned char* dyn) {
  const int32_t V = A.V1 - 1;
  Ctx C;
  C.A = &A;
  C.off = off;
  C.mode = mode;
  C.fixed = fixed;
  C.cap = A.max_override > 0 ? A.max_override : 1;
  C.omark = reinterpret_cast<uint32_t*>(dyn);
  C.olist_y = reinterpret_cast<int32_t*>(dyn + 4 * (size_t)V);
  C.olist_psi = reinterpret_cast<float*>(dyn + 4 * (size_t)V + 4 * (size_t)C.cap);
  C.nlist = nlist;
  C.tag = 0u;
  for (int32_t c = threadIdx.x; c < V; c += kThreads) C.omark[c] = 0u;
  return C;
}

// Per-thread registers of its tokens v = tid + kThreads * j. The blank and the
// positions past the row have root psi -inf, so they never win as tokens; the
// blank is scored on its own (zb, held by the thread that owns it).
template <int TPV>
struct Own {
  float z[TPV];
  float zb;          // the blank's logit (thread V mod kThreads only)
  int32_t cls[TPV];  // class of v (-1: none, blank or past the row)
  float rps[TPV];    // psi of v's root move (0 when unbiased; -inf: blank, past the row)
  int32_t rds[TPV];  // target of v's root move (the fixed state when unbiased)
};

template <class Ld, int TPV>
__device__ __forceinline__ void load_row(float (&z)[TPV], float& zb, const typename Ld::T* row,
                                         int32_t V1x) {
  const int32_t V1 = opaque(V1x);
  const int32_t V = V1 - 1;
#pragma unroll
  for (int j = 0; j < TPV; ++j) {
    const int32_t v = (int32_t)threadIdx.x + kThreads * j;
    z[j] = (v < V1) ? Ld::get(row, v) : kNegInf;
  }
  zb = ((int32_t)threadIdx.x == V % kThreads) ? Ld::get(row, V) : kNegInf;
}

template <int TPV>
__device__ __forceinline__ void own_tables(Own<TPV>& o, const ArenaView& A, int32_t m, int mode,
                                           int32_t fixed) {
  const int32_t V1 = A.V1, V = V1 - 1;
  const float* gpsi = A.root_psi + (int64_t)(mode == 1 ? m : 0) * V1;
  const int32_t* gdst = A.root_dst + (int64_t)(mode == 1 ? m : 0) * V1;
#pragma unroll
  for (int j = 0; j < TPV; ++j) {
    const int32_t v = (int32_t)threadIdx.x + kThreads * j;
    const bool tok = v < V;
    o.cls[j] = tok ? A.class_map[v] : -1;
    o.rps[j] = tok ? (mode == 1 ? gpsi[v] : 0.f) : kNegInf;
    o.rds[j] = (mode == 1) ? (tok ? gdst[v] : 0) : fixed;
  }
}

// The classes overridden in state s: the children of the states on s's
// suffix chain (s, link(s), ..., the root excluded), the deepest state first,
// go to the tag table and the override list, level by level. Returns whether
// any chain was walked (s != 0 for a biased stream); phi_s gets phi[s].
// Contains workgroup barriers (uniform s): all threads must call it.
__device__ __forceinline__ bool build_overrides(Ctx& C, int32_t s, float& phi_s) {
  const ArenaView& A = *C.A;
  const int32_t V = A.V1 - 1;
  const int tid = threadIdx.x;
  phi_s = 0.f;
  if (C.mode != 1) return false;
  phi_s = sld(A.phi + C.off + s);
  if (s == 0) return false;
  if (++C.tag == 65536u) {  // uniform: clear the tags and restart
    for (int32_t c = tid; c < V; c += kThreads) C.omark[c] = 0u;
    C.tag = 1u;
  }
  if (tid == 0) *C.nlist = 0;
  __syncthreads();
  for (int32_t x = s; x != 0;) {
    const int32_t fc = sld(A.first_child + C.off + x);
    const int32_t nc = sld(A.n_child + C.off + x);
    const int32_t lk = sld(A.link + C.off + x);
    for (int32_t j = tid; j < nc; j += kThreads) {
      const int32_t y = fc + j;
      const int32_t c = A.label[C.off + y];
      // a class already listed by a deeper chain state keeps that move
      if ((C.omark[c] >> 16) != C.tag) {
        const int32_t slot = atomicAdd(C.nlist, 1);
        if (slot < C.cap) {
          C.olist_y[slot] = y;
          C.olist_psi[slot] = A.psi[C.off + y];
          C.omark[c] = (C.tag << 16) | (uint32_t)slot;
        }
      }
    }
    __syncthreads();
    x = lk;
  }
  return true;
}

// Calls visit(j, p, ns) for every token slot j of this thread with the psi p
// of its move and the state ns it moves to: the override when its class is in
// the table (chain), else its root move. Tag reads of 8 tokens are issued
// together, then their list entries (slot 0 when not overridden).
template <int TPV, class F>
__device__ __forceinline__ void for_each_move(const Ctx& C, const Own<TPV>& o, bool chain,
                                              F&& visit) {
  if (chain) {
    constexpr int kG = 8;
#pragma unroll
    for (int g0 = 0; g0 < TPV; g0 += kG) {
      uint32_t e[kG];
#pragma unroll
      for (int i = 0; i < kG; ++i)
        if (g0 + i < TPV) e[i] = C.omark[o.cls[g0 + i] > 0 ? o.cls[g0 + i] : 0];
      float po[kG];
      int32_t yo[kG];
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        if (g0 + i < TPV) {
          const bool ov = o.cls[g0 + i] >= 0 && (e[i] >> 16) == C.tag;
          const int32_t slot = ov ? (int32_t)(e[i] & 0xffffu) : 0;
          po[i] = C.olist_psi[slot];
          yo[i] = C.olist_y[slot];
          e[i] = ov ? 1u : 0u;
        }
      }
#pragma unroll
      for (int i = 0; i < kG; ++i) {
        if (g0 + i < TPV) {
          const int j = g0 + i;
          visit(j, e[i] ? po[i] : o.rps[j], e[i] ? yo[i] : o.rds[j]);
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < TPV; ++j) visit(j, o.rps[j], o.rds[j]);
  }
}

}  // namespace wide
}  // namespace tbias
