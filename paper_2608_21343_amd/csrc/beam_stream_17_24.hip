// Streaming beam kernel (hypothesis recombination and tree), instantiated for
// rows of 1025..1536 logits (chunk counts 17..24) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamStreamLaunch beam_stream_launcher_17_24(int per, int32_t dtype) {
  switch (per) {
#define TB_STREAM_CASE(P) \
  case P:                 \
    return dtype == TB_F32 ? &launch_beam_stream_t<LoadF32, P> : &launch_beam_stream_t<LoadBF16, P>;
    TB_STREAM_CASE(17) TB_STREAM_CASE(18) TB_STREAM_CASE(19) TB_STREAM_CASE(20) TB_STREAM_CASE(21) TB_STREAM_CASE(22) TB_STREAM_CASE(23) TB_STREAM_CASE(24)
#undef TB_STREAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
