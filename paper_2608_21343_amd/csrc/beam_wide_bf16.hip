// Wide-vocabulary beam kernel, bfloat16 logits.
#include "beam_wide.hpp"

namespace tbias {
namespace wide {

BeamWideLaunch beam_wide_launcher_bf16(int tpv, int maxk) {
  return beam_wide_launcher<LoadBF16>(tpv, maxk);
}

}  // namespace wide
}  // namespace tbias
