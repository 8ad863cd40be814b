// Wide-vocabulary beam kernel, float32 logits.
#include "beam_wide.hpp"

namespace tbias {
namespace wide {

BeamWideLaunch beam_wide_launcher_f32(int tpv, int maxk) {
  return beam_wide_launcher<LoadF32>(tpv, maxk);
}

}  // namespace wide
}  // namespace tbias
