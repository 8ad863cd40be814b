// Beam kernel, instantiated for rows of 1..512 logits (chunk counts 1..8) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamLaunch beam_launcher_1_8(int per, int maxk, int32_t dtype) {
  switch (per) {
#define TB_BEAM_CASE(P)                                                                   \
  case P:                                                                                \
    if (maxk == 2) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 2> : &launch_beam_fast_t<LoadBF16, P, 2>; \
    if (maxk == 4) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 4> : &launch_beam_fast_t<LoadBF16, P, 4>; \
    return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 8> : &launch_beam_fast_t<LoadBF16, P, 8>;
     TB_BEAM_CASE(1) TB_BEAM_CASE(2) TB_BEAM_CASE(3) TB_BEAM_CASE(4) TB_BEAM_CASE(5) TB_BEAM_CASE(6) TB_BEAM_CASE(7) TB_BEAM_CASE(8)
#undef TB_BEAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
