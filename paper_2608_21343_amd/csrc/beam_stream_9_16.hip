// Streaming beam kernel (hypothesis recombination and tree), instantiated for
// rows of 513..1024 logits (chunk counts 9..16) and K <= 8.
#include "beam_fast.hpp"

namespace tbias {
namespace beamk {

BeamStreamLaunch beam_stream_launcher_9_16(int per, int32_t dtype) {
  switch (per) {
#define TB_STREAM_CASE(P) \
  case P:                 \
    return dtype == TB_F32 ? &launch_beam_stream_t<LoadF32, P> : &launch_beam_stream_t<LoadBF16, P>;
    TB_STREAM_CASE(9) TB_STREAM_CASE(10) TB_STREAM_CASE(11) TB_STREAM_CASE(12) TB_STREAM_CASE(13) TB_STREAM_CASE(14) TB_STREAM_CASE(15) TB_STREAM_CASE(16)
#undef TB_STREAM_CASE
    default:
      return nullptr;
  }
}

}  // namespace beamk
}  // namespace tbias
