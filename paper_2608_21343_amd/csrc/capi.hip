// C ABI shim: synchronous argument checks, then asynchronous launches.
#include <atomic>
#include <cstring>
#include <string>

#include "internal.hpp"
#include "launch.hpp"

using namespace tbias;

namespace {

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

int check_arena(const tb_arena* a) {
  if (!a) return fail(TB_EINVAL, "arena is NULL");
  if (!a->base) return fail(TB_EINVAL, "arena base is NULL");
  if (!aligned(a->base, 256)) return fail(TB_EINVAL, "arena base not 256-byte aligned");
  const tb_arena_layout& L = a->layout;
  if (L.n_models < 1 || L.v_plus_blank < 2 || L.n_states < L.n_models || L.total_bytes <= 0)
    return fail(TB_EINVAL, "arena layout is not initialised");
  if (L.v_plus_blank > kMaxV1)
    return fail(TB_EINVAL, "v_plus_blank " + std::to_string(L.v_plus_blank) +
                               " exceeds the supported maximum " + std::to_string(kMaxV1));
  return TB_OK;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(TB_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

int check_i32(const void* p, const char* name) {
  if (!p) return fail(TB_EINVAL, std::string(name) + " is NULL");
  if (!aligned(p, 4)) return fail(TB_EINVAL, std::string(name) + " not 4-byte aligned");
  return TB_OK;
}

int check_logits(const void* logits, int32_t dtype, int64_t row_stride, int32_t V1) {
  if (dtype != TB_F32 && dtype != TB_BF16) return fail(TB_EINVAL, "unknown dtype");
  if (!logits) return fail(TB_EINVAL, "logits is NULL");
  if (!aligned(logits, dtype == TB_F32 ? 4 : 2)) return fail(TB_EINVAL, "logits misaligned");
  if (row_stride < V1)
    return fail(TB_EINVAL, "row_stride " + std::to_string(row_stride) + " < V+1 = " +
                               std::to_string(V1));
  return TB_OK;
}

std::atomic<int32_t> g_greedy_kernel{kGreedyAuto};
std::atomic<int32_t> g_beam_kernel{kBeamAuto};
std::atomic<uint32_t> g_spin_limit{0u};

}  // namespace

namespace tbias {
int32_t debug_greedy_kernel() { return g_greedy_kernel.load(std::memory_order_relaxed); }
int32_t debug_beam_kernel() { return g_beam_kernel.load(std::memory_order_relaxed); }
uint32_t debug_spin_limit() { return g_spin_limit.load(std::memory_order_relaxed); }
}  // namespace tbias

extern "C" int tb_debug_select_kernels(int32_t greedy, int32_t beam) {
  if (greedy < kGreedyAuto || greedy > kGreedyRef) return fail(TB_EINVAL, "unknown greedy kernel");
  if (beam < kBeamAuto || beam > kBeamNoPipe) return fail(TB_EINVAL, "unknown beam kernel");
  g_greedy_kernel.store(greedy, std::memory_order_relaxed);
  g_beam_kernel.store(beam, std::memory_order_relaxed);
  return TB_OK;
}

extern "C" int tb_debug_set_spin_limit(uint32_t polls) {
  g_spin_limit.store(polls, std::memory_order_relaxed);
  return TB_OK;
}

extern "C" int tb_debug_launch_empty(int32_t grid, int32_t block, int32_t lds_bytes,
                                     void* hip_stream) {
  if (grid < 1 || block < 1 || block > 1024 || lds_bytes < 0 || lds_bytes > 160 * 1024)
    return fail(TB_EINVAL, "launch shape out of range");
  hipError_t e = launch_empty(grid, block, lds_bytes, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "empty kernel launch");
  return TB_OK;
}

extern "C" int tb_graphs_upload(const tb_graphs* g, void* dev_base, int64_t bytes,
                                void* hip_stream, tb_arena* out) {
  if (!g || !dev_base || !out) return fail(TB_EINVAL, "NULL argument");
  if (!aligned(dev_base, 256)) return fail(TB_EINVAL, "dev_base not 256-byte aligned");
  if (bytes < g->layout.total_bytes) return fail(TB_ENOMEM, "device buffer too small");
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  hipError_t e = hipMemcpyAsync(dev_base, g->image.data(), (size_t)g->layout.total_bytes,
                                hipMemcpyHostToDevice, st);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync");
  e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  out->base = dev_base;
  out->layout = g->layout;
  return TB_OK;
}

extern "C" int tb_init_states(const tb_arena* a, int32_t B, int32_t K, const int32_t* model_ids,
                              int32_t* states, float* scores, void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (K < 1 || K > TB_MAX_BEAM) return fail(TB_EINVAL, "K outside [1, TB_MAX_BEAM]");
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if (scores && !aligned(scores, 4)) return fail(TB_EINVAL, "scores not 4-byte aligned");
  hipError_t e = launch_init_states(make_view(*a), B, K, model_ids, states, scores,
                                    static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "init_states launch");
  return TB_OK;
}

extern "C" int tb_init_beam_stream(const tb_arena* a, int32_t B, int32_t K,
                                   const int32_t* model_ids, int32_t* states, float* scores,
                                   tb_hyp* hyps, int32_t* tree_len, void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (K < 1 || K > TB_MAX_BEAM) return fail(TB_EINVAL, "K outside [1, TB_MAX_BEAM]");
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if ((r = check_i32(scores, "scores"))) return r;
  if ((r = check_i32(tree_len, "tree_len"))) return r;
  if (!hyps || !aligned(hyps, 8)) return fail(TB_EINVAL, "hyps NULL or not 8-byte aligned");
  hipError_t e = launch_init_beam_stream(make_view(*a), B, K, model_ids, states, scores, hyps,
                                         tree_len, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "init_beam_stream launch");
  return TB_OK;
}

extern "C" int tb_reset_stream(const tb_arena* a, int32_t B, int32_t b, int32_t new_model_id,
                               int32_t K, int32_t* model_ids, int32_t* states, float* scores,
                               void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (b < 0 || b >= B) return fail(TB_EINVAL, "stream index outside [0, B)");
  if (K < 1 || K > TB_MAX_BEAM) return fail(TB_EINVAL, "K outside [1, TB_MAX_BEAM]");
  if (new_model_id < -1 || new_model_id >= a->layout.n_models)
    return fail(TB_ERANGE, "model id " + std::to_string(new_model_id) + " outside [-1, " +
                               std::to_string(a->layout.n_models) + ")");
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if (scores && !aligned(scores, 4)) return fail(TB_EINVAL, "scores not 4-byte aligned");
  hipError_t e = launch_reset_stream(b, new_model_id, K, model_ids, states, scores,
                                     static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "reset_stream launch");
  return TB_OK;
}

extern "C" int tb_boost_step_greedy(const tb_arena* a, const void* logits, int32_t dtype,
                                    int32_t T, int32_t B, int64_t row_stride,
                                    const int32_t* model_ids, int32_t* states, int32_t* out_tok,
                                    int32_t* out_state, float* out_score, void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (T < 0) return fail(TB_EINVAL, "T must be >= 0");
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (T == 0) return TB_OK;  // no-op: buffers are not touched (and may be NULL)
  if ((r = check_logits(logits, dtype, row_stride, a->layout.v_plus_blank))) return r;
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if ((r = check_i32(out_tok, "out_tok"))) return r;
  if ((r = check_i32(out_state, "out_state"))) return r;
  if ((r = check_i32(out_score, "out_score"))) return r;
  hipError_t e = launch_greedy(make_view(*a), logits, dtype, T, B, row_stride, model_ids, states,
                               out_tok, out_state, out_score,
                               static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "greedy launch");
  return TB_OK;
}

extern "C" int tb_boost_step_beam(const tb_arena* a, const void* logits, int32_t dtype, int32_t T,
                                  int32_t B, int32_t K, int64_t row_stride,
                                  const int32_t* model_ids, int32_t* states, float* scores,
                                  int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                                  float* out_step, float* out_cum, void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (T < 0) return fail(TB_EINVAL, "T must be >= 0");
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (K < 1 || K > TB_MAX_BEAM) return fail(TB_EINVAL, "K outside [1, TB_MAX_BEAM]");
  if (K > a->layout.v_plus_blank) return fail(TB_EINVAL, "K exceeds V+1");
  if (T == 0) return TB_OK;  // no-op: buffers are not touched (and may be NULL)
  if ((r = check_logits(logits, dtype, row_stride, a->layout.v_plus_blank))) return r;
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if ((r = check_i32(scores, "scores"))) return r;
  if ((r = check_i32(out_tok, "out_tok"))) return r;
  if ((r = check_i32(out_parent, "out_parent"))) return r;
  if ((r = check_i32(out_state, "out_state"))) return r;
  if ((r = check_i32(out_step, "out_step"))) return r;
  if ((r = check_i32(out_cum, "out_cum"))) return r;
  hipError_t e = launch_beam(make_view(*a), logits, dtype, T, B, K, row_stride, model_ids, states,
                             scores, out_tok, out_parent, out_state, out_step, out_cum,
                             static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "beam launch");
  return TB_OK;
}

extern "C" int tb_boost_step_beam_stream(const tb_arena* a, const void* logits, int32_t dtype,
                                         int32_t T, int32_t B, int32_t K, int64_t row_stride,
                                         const int32_t* model_ids, int32_t* states, float* scores,
                                         tb_hyp* hyps, int32_t* tree, int32_t tree_cap,
                                         int32_t* tree_len, int32_t recombine, int32_t* out_tok,
                                         int32_t* out_parent, int32_t* out_state, float* out_step,
                                         float* out_cum, void* hip_stream) {
  int r;
  if ((r = check_arena(a))) return r;
  if (T < 0) return fail(TB_EINVAL, "T must be >= 0");
  if (B < 1) return fail(TB_EINVAL, "B must be >= 1");
  if (K < 1 || K > TB_MAX_BEAM) return fail(TB_EINVAL, "K outside [1, TB_MAX_BEAM]");
  if (K > a->layout.v_plus_blank) return fail(TB_EINVAL, "K exceeds V+1");
  if (tree_cap < 0) return fail(TB_EINVAL, "tree_cap must be >= 0");
  if (T == 0) return TB_OK;  // no-op: buffers are not touched (and may be NULL)
  if ((r = check_logits(logits, dtype, row_stride, a->layout.v_plus_blank))) return r;
  if ((r = check_i32(model_ids, "model_ids"))) return r;
  if ((r = check_i32(states, "states"))) return r;
  if ((r = check_i32(scores, "scores"))) return r;
  if ((r = check_i32(tree_len, "tree_len"))) return r;
  if (!hyps || !aligned(hyps, 8)) return fail(TB_EINVAL, "hyps NULL or not 8-byte aligned");
  if (tree_cap > 0 && (r = check_i32(tree, "tree"))) return r;
  if ((r = check_i32(out_tok, "out_tok"))) return r;
  if ((r = check_i32(out_parent, "out_parent"))) return r;
  if ((r = check_i32(out_state, "out_state"))) return r;
  if ((r = check_i32(out_step, "out_step"))) return r;
  if ((r = check_i32(out_cum, "out_cum"))) return r;
  hipError_t e = launch_beam_stream(make_view(*a), logits, dtype, T, B, K, row_stride, model_ids,
                                    states, scores, hyps, tree, tree_cap, tree_len, recombine,
                                    out_tok, out_parent, out_state, out_step, out_cum,
                                    static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return hip_fail(e, "streaming beam launch");
  return TB_OK;
}
