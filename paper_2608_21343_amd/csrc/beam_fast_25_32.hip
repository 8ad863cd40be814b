// Beam kernel, instantiated for rows of 1537..2048 logits (chunk counts 25..32) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamLaunch beam_launcher_25_32(int per, int maxk, int32_t dtype) {
  switch (per) {
#define TB_BEAM_CASE(P)                                                                   \
  case P:                                                                                \
    if (maxk == 2) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 2> : &launch_beam_fast_t<LoadBF16, P, 2>; \
    if (maxk == 4) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 4> : &launch_beam_fast_t<LoadBF16, P, 4>; \
    return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 8> : &launch_beam_fast_t<LoadBF16, P, 8>;
     TB_BEAM_CASE(25) TB_BEAM_CASE(26) TB_BEAM_CASE(27) TB_BEAM_CASE(28) TB_BEAM_CASE(29) TB_BEAM_CASE(30) TB_BEAM_CASE(31) TB_BEAM_CASE(32)
#undef TB_BEAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
