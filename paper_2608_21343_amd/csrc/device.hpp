// Device-side view of the arena and small wave64 helpers (gfx950).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/tbias.h"

namespace tbias {

// Raw device pointers into one arena image (see tb_arena_layout).
struct ArenaView {
  const int32_t* model_off;
  const int32_t* model_n;
  const int32_t* first_child;
  const int32_t* n_child;
  const int32_t* link;
  const int32_t* label;
  const float* phi;
  const float* psi;
  const float* root_psi;
  const int32_t* root_dst;
  const int32_t* class_map;
  const int32_t* cls_ptr;
  const int32_t* cls_tok;
  const uint32_t* arc_mem;  // two words per state (see tb_arena_layout)
  const float* value_tab;      // per model: 256 psi values, 256 phi values
  const uint32_t* state_rec;   // three words per state (see tb_arena_layout)
  int64_t n_states;      // over all models
  int32_t n_models;
  int32_t V1;            // V + 1
  int32_t max_override;  // most tokens any state overrides
};

inline ArenaView make_view(const tb_arena& a) {
  const unsigned char* b = static_cast<const unsigned char*>(a.base);
  const tb_arena_layout& L = a.layout;
  ArenaView v;
  v.model_off = reinterpret_cast<const int32_t*>(b + L.off_model_off);
  v.model_n = reinterpret_cast<const int32_t*>(b + L.off_model_n);
  v.first_child = reinterpret_cast<const int32_t*>(b + L.off_first_child);
  v.n_child = reinterpret_cast<const int32_t*>(b + L.off_n_child);
  v.link = reinterpret_cast<const int32_t*>(b + L.off_link);
  v.label = reinterpret_cast<const int32_t*>(b + L.off_label);
  v.phi = reinterpret_cast<const float*>(b + L.off_phi);
  v.psi = reinterpret_cast<const float*>(b + L.off_psi);
  v.root_psi = reinterpret_cast<const float*>(b + L.off_root_psi);
  v.root_dst = reinterpret_cast<const int32_t*>(b + L.off_root_dst);
  v.class_map = reinterpret_cast<const int32_t*>(b + L.off_class_map);
  v.cls_ptr = reinterpret_cast<const int32_t*>(b + L.off_cls_ptr);
  v.cls_tok = reinterpret_cast<const int32_t*>(b + L.off_cls_tok);
  v.arc_mem = reinterpret_cast<const uint32_t*>(b + L.off_arc_mem);
  v.value_tab = reinterpret_cast<const float*>(b + L.off_value_tab);
  v.state_rec = reinterpret_cast<const uint32_t*>(b + L.off_state_rec);
  v.n_states = L.n_states;
  v.n_models = L.n_models;
  v.V1 = L.v_plus_blank;
  v.max_override = L.max_override;
  return v;
}

// Element loaders: float32 as is, bfloat16 widened exactly.
struct LoadF32 {
  typedef float T;
  __device__ static inline float get(const float* p, int64_t i) { return p[i]; }
  // streaming read of a logit row: read once, not kept in the caches
  __device__ static inline float get_nt(const float* p, int64_t i) {
    return __builtin_nontemporal_load(p + i);
  }
};
struct LoadBF16 {
  typedef uint16_t T;
  __device__ static inline float get(const uint16_t* p, int64_t i) {
    return __uint_as_float(((uint32_t)p[i]) << 16);
  }
  __device__ static inline float get_nt(const uint16_t* p, int64_t i) {
    return __uint_as_float(((uint32_t)__builtin_nontemporal_load(p + i)) << 16);
  }
};

// (key, index) order used by every selection: larger key first, then lower index.
__device__ inline bool better(float ka, int32_t ia, float kb, int32_t ib) {
  return ka > kb || (ka == kb && ia < ib);
}

// ---- wave64 reductions on DPP (row shifts within rows of 16 lanes, then the
// gfx9 row broadcasts); every lane of the wave must be active. The result is
// the value of lane 63, returned uniform.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_i(int old, int src) {
  return __builtin_amdgcn_update_dpp(old, src, CTRL, ROW_MASK, 0xf, false);
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float old, float src) {
  return __int_as_float(dpp_i<CTRL, ROW_MASK>(__float_as_int(old), __float_as_int(src)));
}
__device__ __forceinline__ float bcast63_f(float v) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

__device__ __forceinline__ float wave_max_dpp(float v) {
  const float id = -__builtin_huge_valf();
  v = fmaxf(v, dpp_f<0x111, 0xf>(id, v));
  v = fmaxf(v, dpp_f<0x112, 0xf>(id, v));
  v = fmaxf(v, dpp_f<0x114, 0xf>(id, v));
  v = fmaxf(v, dpp_f<0x118, 0xf>(id, v));
  v = fmaxf(v, dpp_f<0x142, 0xa>(id, v));
  v = fmaxf(v, dpp_f<0x143, 0xc>(id, v));
  return bcast63_f(v);
}

__device__ __forceinline__ float wave_sum_dpp(float v) {
  v = v + dpp_f<0x111, 0xf>(0.f, v);
  v = v + dpp_f<0x112, 0xf>(0.f, v);
  v = v + dpp_f<0x114, 0xf>(0.f, v);
  v = v + dpp_f<0x118, 0xf>(0.f, v);
  v = v + dpp_f<0x142, 0xa>(0.f, v);
  v = v + dpp_f<0x143, 0xc>(0.f, v);
  return bcast63_f(v);
}

__device__ __forceinline__ int32_t wave_min_i32_dpp(int32_t v) {
  const int32_t id = 0x7fffffff;
  v = min(v, dpp_i<0x111, 0xf>(id, v));
  v = min(v, dpp_i<0x112, 0xf>(id, v));
  v = min(v, dpp_i<0x114, 0xf>(id, v));
  v = min(v, dpp_i<0x118, 0xf>(id, v));
  v = min(v, dpp_i<0x142, 0xa>(id, v));
  v = min(v, dpp_i<0x143, 0xc>(id, v));
  return __builtin_amdgcn_readlane(v, 63);
}

// Wave argmax of (key, idx): larger key, then lower idx. Returns the winner
// (uniform) and the first lane holding it.
__device__ __forceinline__ int32_t wave_argmax_dpp(float key, int32_t idx, float& bk, int32_t& bi) {
  const float m = wave_max_dpp(key);
  const uint64_t hit = __ballot(key == m);
  int32_t lane;
  if (__builtin_popcountll(hit) == 1) {
    lane = (int32_t)__builtin_ctzll(hit);
    bi = __builtin_amdgcn_readlane(idx, lane);
  } else {
    bi = wave_min_i32_dpp(key == m ? idx : 0x7fffffff);
    const uint64_t own = __ballot(key == m && idx == bi);
    lane = own ? (int32_t)__builtin_ctzll(own) : 0;
  }
  bk = m;
  return lane;
}

__device__ inline float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

__device__ inline float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__device__ inline double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

__device__ inline void wave_argmax(float& k, int32_t& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float k2 = __shfl_xor(k, o, 64);
    int32_t i2 = __shfl_xor(i, o, 64);
    if (better(k2, i2, k, i)) { k = k2; i = i2; }
  }
}

// e^x for x <= 0 in float64 (x = -inf and x < -745 give 0): e^x = 2^k e^r with
// k = rint(x / ln 2) and r = x - k ln 2, ln 2 split in a high part with
// trailing zero bits (k * ln2_hi is exact for |k| < 2^11) and a low part
// (Cody and Waite's reduction); e^r is summed as its Taylor series to degree
// 12, whose truncation error for |r| <= ln(2)/2 is below 2e-16 relative.
__device__ __forceinline__ double exp_nonpos(double x) {
  const double kInvLn2 = 1.4426950408889634074;
  const double kLn2Hi = 6.93147180369123816490e-01;
  const double kLn2Lo = 1.90821492927058770002e-10;
  const bool tiny = !(x >= -745.0);
  x = tiny ? -745.0 : x;  // keeps k finite; the result is selected below
  const double k = __builtin_rint(x * kInvLn2);
  const double r = __builtin_fma(-k, kLn2Lo, __builtin_fma(-k, kLn2Hi, x));
  double p = 1.0 / 479001600.0;  // 1/12!
  p = __builtin_fma(p, r, 1.0 / 39916800.0);
  p = __builtin_fma(p, r, 1.0 / 3628800.0);
  p = __builtin_fma(p, r, 1.0 / 362880.0);
  p = __builtin_fma(p, r, 1.0 / 40320.0);
  p = __builtin_fma(p, r, 1.0 / 5040.0);
  p = __builtin_fma(p, r, 1.0 / 720.0);
  p = __builtin_fma(p, r, 1.0 / 120.0);
  p = __builtin_fma(p, r, 1.0 / 24.0);
  p = __builtin_fma(p, r, 1.0 / 6.0);
  p = __builtin_fma(p, r, 0.5);
  p = __builtin_fma(p, r, 1.0);
  p = __builtin_fma(p, r, 1.0);
  return tiny ? 0.0 : __builtin_ldexp(p, (int)k);
}

// Debug builds (TB_POISON_LDS): a kernel first fills its LDS with all bits
// set (a NaN, -1, 0xffff: no table or candidate holds that pattern as data),
// so a read of a word the kernel did not write first changes its results.
// Every thread of the workgroup calls it (a barrier follows).
__device__ __forceinline__ void lds_poison(void* p, size_t bytes) {
#ifdef TB_POISON_LDS
  uint32_t* w = static_cast<uint32_t*>(p);
  for (size_t i = threadIdx.x; i < bytes / 4; i += blockDim.x) w[i] = 0xffffffffu;
  __syncthreads();
#else
  (void)p;
  (void)bytes;
#endif
}

// The state written for a stream decoded without biasing (mode != 1 below):
// -1 for model -1; a carried TB_STATE_TIMEOUT stays TB_STATE_TIMEOUT (the
// stream's earlier outputs are unreliable until it is reset); any other
// out-of-range model id or carried state gives TB_STATE_INVALID.
__device__ __forceinline__ int32_t unbiased_state(int mode, bool carried_timeout) {
  if (mode == 0) return TB_STATE_NONE;
  return carried_timeout ? TB_STATE_TIMEOUT : TB_STATE_INVALID;
}

// Resolve a (model id, carried state) pair.
//   returns 1 and sets off/n when the stream is biased with a valid state,
//   0 for model -1, -1 for an out-of-range model id or carried state.
__device__ inline int resolve_stream(const ArenaView& A, int32_t m, int32_t s, int32_t& off,
                                     int32_t& n) {
  if (m == -1) return 0;
  if (m < -1 || m >= A.n_models) return -1;
  off = A.model_off[m];
  n = A.model_n[m];
  if (s < 0 || s >= n) return -1;
  return 1;
}

}  // namespace tbias
