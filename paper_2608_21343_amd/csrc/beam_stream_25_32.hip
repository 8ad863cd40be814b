// Streaming beam kernel (hypothesis recombination and tree), instantiated for
// rows of 1537..2048 logits (chunk counts 25..32) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamStreamLaunch beam_stream_launcher_25_32(int per, int32_t dtype) {
  switch (per) {
#define TB_STREAM_CASE(P) \
  case P:                 \
    return dtype == TB_F32 ? &launch_beam_stream_t<LoadF32, P> : &launch_beam_stream_t<LoadBF16, P>;
    TB_STREAM_CASE(25) TB_STREAM_CASE(26) TB_STREAM_CASE(27) TB_STREAM_CASE(28) TB_STREAM_CASE(29) TB_STREAM_CASE(30) TB_STREAM_CASE(31) TB_STREAM_CASE(32)
#undef TB_STREAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
