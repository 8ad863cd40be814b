// Segmented greedy kernel, instantiated for rows of 513..1024 logits (chunk counts 9..16).
#include "greedy_seg.hpp"

namespace tbias {
namespace seg {

SegLaunch seg_launcher_9_16(int per, int32_t dtype) {
  switch (per) {
#define TB_SEG_CASE(P) \
  case P:            \
    return dtype == TB_F32 ? &launch_seg<LoadF32, P> : &launch_seg<LoadBF16, P>;
     TB_SEG_CASE(9) TB_SEG_CASE(10) TB_SEG_CASE(11) TB_SEG_CASE(12) TB_SEG_CASE(13) TB_SEG_CASE(14) TB_SEG_CASE(15) TB_SEG_CASE(16)
#undef TB_SEG_CASE
    default:
      return nullptr;
  }
}

}  // namespace seg
}  // namespace tbias
