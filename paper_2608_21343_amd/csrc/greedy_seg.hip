// Dispatch of the segmented greedy kernel by chunk count (see greedy_seg.hpp).
#include "greedy_seg.hpp"
#include "launch.hpp"

namespace tbias {

// Returns hipErrorNotSupported when the vocabulary is too large for this kernel.
hipError_t launch_greedy_seg(const ArenaView& A, const void* logits, int32_t dtype, int32_t T,
                             int32_t B, int64_t row_stride, const int32_t* model_ids,
                             int32_t* states, int32_t* out_tok, int32_t* out_state,
                             float* out_score, hipStream_t st) {
  const int32_t V1 = A.V1;
  if (V1 > 64 * 32 || V1 < 2) return hipErrorNotSupported;
  const int per = (V1 + 63) / 64;
  seg::SegLaunch f = per <= 8    ? seg::seg_launcher_1_8(per, dtype)
                     : per <= 16 ? seg::seg_launcher_9_16(per, dtype)
                     : per <= 24 ? seg::seg_launcher_17_24(per, dtype)
                                 : seg::seg_launcher_25_32(per, dtype);
  if (!f) return hipErrorNotSupported;
  return f(A, logits, T, B, row_stride, model_ids, states, out_tok, out_state, out_score, st);
}

}  // namespace tbias
