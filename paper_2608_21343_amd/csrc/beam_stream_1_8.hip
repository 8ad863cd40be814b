// Streaming beam kernel (hypothesis recombination and tree), instantiated for
// rows of 1..512 logits (chunk counts 1..8) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamStreamLaunch beam_stream_launcher_1_8(int per, int32_t dtype) {
  switch (per) {
#define TB_STREAM_CASE(P) \
  case P:                 \
    return dtype == TB_F32 ? &launch_beam_stream_t<LoadF32, P> : &launch_beam_stream_t<LoadBF16, P>;
    TB_STREAM_CASE(1) TB_STREAM_CASE(2) TB_STREAM_CASE(3) TB_STREAM_CASE(4) TB_STREAM_CASE(5) TB_STREAM_CASE(6) TB_STREAM_CASE(7) TB_STREAM_CASE(8)
#undef TB_STREAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
