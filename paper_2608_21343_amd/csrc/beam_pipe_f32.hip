// Wide-row beam kernel with helper waves, float32 logits.
#include "beam_pipe.hpp"

namespace tbias {
namespace bpipe {

PipeLaunch pipe_launcher_f32(int32_t V1, int32_t K) {
  if (K > kSlots || V1 <= 2048) return nullptr;
  if (V1 <= 128 * 17) return &launch_pipe_t<LoadF32, 17>;
  if (V1 <= 128 * 33) return &launch_pipe_t<LoadF32, 33>;
  return nullptr;
}

}  // namespace bpipe
}  // namespace tbias
