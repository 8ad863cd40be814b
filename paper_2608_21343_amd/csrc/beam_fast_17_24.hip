// Beam kernel, instantiated for rows of 1025..1536 logits (chunk counts 17..24) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamLaunch beam_launcher_17_24(int per, int maxk, int32_t dtype) {
  switch (per) {
#define TB_BEAM_CASE(P)                                                                   \
  case P:                                                                                \
    if (maxk == 2) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 2> : &launch_beam_fast_t<LoadBF16, P, 2>; \
    if (maxk == 4) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 4> : &launch_beam_fast_t<LoadBF16, P, 4>; \
    return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 8> : &launch_beam_fast_t<LoadBF16, P, 8>;
     TB_BEAM_CASE(17) TB_BEAM_CASE(18) TB_BEAM_CASE(19) TB_BEAM_CASE(20) TB_BEAM_CASE(21) TB_BEAM_CASE(22) TB_BEAM_CASE(23) TB_BEAM_CASE(24)
#undef TB_BEAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
