// Host launchers of the device kernels (argument checks happen in the C ABI).
#pragma once

#include <hip/hip_runtime.h>

#include "device.hpp"

namespace tbias {

hipError_t launch_init_states(const ArenaView& A, int32_t B, int32_t K, const int32_t* model_ids,
                              int32_t* states, float* scores, hipStream_t st);
hipError_t launch_empty(int32_t grid, int32_t block, int32_t lds_bytes, hipStream_t st);
hipError_t launch_reset_stream(int32_t b, int32_t m, int32_t K, int32_t* model_ids,
                               int32_t* states, float* scores, hipStream_t st);

// Greedy: T steps for B streams. Requires V1 <= kMaxV1.
hipError_t launch_greedy(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                         int32_t B, int64_t row_stride, const int32_t* model_ids, int32_t* states,
                         int32_t* out_tok, int32_t* out_state, float* out_score, hipStream_t st);

hipError_t launch_beam(const ArenaView& A, const void* logits, int32_t dtype, int32_t T, int32_t B,
                       int32_t K, int64_t row_stride, const int32_t* model_ids, int32_t* states,
                       float* scores, int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                       float* out_step, float* out_cum, hipStream_t st);

// Streaming beam (recombination and tree): launch_init_beam_stream starts the
// carry; launch_beam_stream returns hipErrorNotSupported for rows or arenas
// its kernel does not serve (beam_stream_supported tells in advance).
hipError_t launch_init_beam_stream(const ArenaView& A, int32_t B, int32_t K,
                                   const int32_t* model_ids, int32_t* states, float* scores,
                                   tb_hyp* hyps, int32_t* tree_len, hipStream_t st);
bool beam_stream_supported(int32_t v_plus_blank, int32_t max_override, int32_t K);
hipError_t launch_beam_stream(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int32_t K, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, float* scores, tb_hyp* hyps, int32_t* tree,
                              int32_t tree_cap, int32_t* tree_len, int32_t recombine,
                              int32_t* out_tok, int32_t* out_parent, int32_t* out_state,
                              float* out_step, float* out_cum, hipStream_t st);

// Segmented greedy kernel (plus its boundary fix-up); hipErrorNotSupported
// when V+1 is too large for it.
hipError_t launch_greedy_seg(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                             int32_t B, int64_t row_stride, const int32_t* model_ids,
                             int32_t* states, int32_t* out_tok, int32_t* out_state,
                             float* out_score, hipStream_t st);

// Segmented greedy kernel for wide vocabularies (V+1 > 2048, one workgroup
// per segment); hipErrorNotSupported outside its range.
hipError_t launch_greedy_wide(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                              int32_t B, int64_t row_stride, const int32_t* model_ids,
                              int32_t* states, int32_t* out_tok, int32_t* out_state,
                              float* out_score, hipStream_t st);

// Largest V+1 the step kernels accept: the compiler's limit (the reference
// kernels' per-class LDS table, 4 B and one bit per class, fits up to it).
constexpr int32_t kMaxV1 = 32768;

// Test hooks (tb_debug_select_kernels, tb_debug_set_spin_limit): kernel
// choices forced by tests, and the poll limit of the greedy hand-off wait
// (0 = the kernel's default). Plain process-wide values, read per call.
enum { kGreedyAuto = 0, kGreedyRef = 1 };
enum { kBeamAuto = 0, kBeamRef = 1, kBeamNoPipe = 2 };
int32_t debug_greedy_kernel();
int32_t debug_beam_kernel();
uint32_t debug_spin_limit();

}  // namespace tbias
