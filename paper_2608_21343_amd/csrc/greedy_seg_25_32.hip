// Segmented greedy kernel, instantiated for rows of 1537..2048 logits (chunk counts 25..32).
#include "greedy_seg.hpp"

namespace tbias {
namespace seg {

SegLaunch seg_launcher_25_32(int per, int32_t dtype) {
  switch (per) {
#define TB_SEG_CASE(P) \
  case P:            \
    return dtype == TB_F32 ? &launch_seg<LoadF32, P> : &launch_seg<LoadBF16, P>;
     TB_SEG_CASE(25) TB_SEG_CASE(26) TB_SEG_CASE(27) TB_SEG_CASE(28) TB_SEG_CASE(29) TB_SEG_CASE(30) TB_SEG_CASE(31) TB_SEG_CASE(32)
#undef TB_SEG_CASE
    default:
      return nullptr;
  }
}

}  // namespace seg
}  // namespace tbias
