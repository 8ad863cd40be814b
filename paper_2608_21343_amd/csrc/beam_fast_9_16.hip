// Beam kernel, instantiated for rows of 513..1024 logits (chunk counts 9..16) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamLaunch beam_launcher_9_16(int per, int maxk, int32_t dtype) {
  switch (per) {
#define TB_BEAM_CASE(P)                                                                   \
  case P:                                                                                \
    if (maxk == 2) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 2> : &launch_beam_fast_t<LoadBF16, P, 2>; \
    if (maxk == 4) return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 4> : &launch_beam_fast_t<LoadBF16, P, 4>; \
    return dtype == TB_F32 ? &launch_beam_fast_t<LoadF32, P, 8> : &launch_beam_fast_t<LoadBF16, P, 8>;
     TB_BEAM_CASE(9) TB_BEAM_CASE(10) TB_BEAM_CASE(11) TB_BEAM_CASE(12) TB_BEAM_CASE(13) TB_BEAM_CASE(14) TB_BEAM_CASE(15) TB_BEAM_CASE(16)
#undef TB_BEAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
