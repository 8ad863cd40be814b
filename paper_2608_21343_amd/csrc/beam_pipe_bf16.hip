// Wide-row beam kernel with helper waves, bfloat16 logits.
#include "beam_pipe.hpp"

namespace tbias {
namespace bpipe {

PipeLaunch pipe_launcher_bf16(int32_t V1, int32_t K) {
  if (K > kSlots || V1 <= 2048) return nullptr;
  if (V1 <= 128 * 17) return &launch_pipe_t<LoadBF16, 17>;
  if (V1 <= 128 * 33) return &launch_pipe_t<LoadBF16, 33>;
  if (V1 <= 128 * 65) return &launch_pipe_t<LoadBF16, 65>;
  return nullptr;
}

}  // namespace bpipe
}  // namespace tbias
