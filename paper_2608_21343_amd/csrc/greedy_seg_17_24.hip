// Segmented greedy kernel, instantiated for rows of 1025..1536 logits (chunk counts 17..24).
#include "greedy_seg.hpp"

namespace tbias {
namespace seg {

SegLaunch seg_launcher_17_24(int per, int32_t dtype) {
  switch (per) {
#define TB_SEG_CASE(P) \
  case P:            \
    return dtype == TB_F32 ? &launch_seg<LoadF32, P> : &launch_seg<LoadBF16, P>;
     TB_SEG_CASE(17) TB_SEG_CASE(18) TB_SEG_CASE(19) TB_SEG_CASE(20) TB_SEG_CASE(21) TB_SEG_CASE(22) TB_SEG_CASE(23) TB_SEG_CASE(24)
#undef TB_SEG_CASE
    default:
      return nullptr;
  }
}

}  // namespace seg
}  // namespace tbias
