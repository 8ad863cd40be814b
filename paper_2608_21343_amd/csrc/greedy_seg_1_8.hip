// Segmented greedy kernel, instantiated for rows of 1..512 logits (chunk counts 1..8).
#include "greedy_seg.hpp"

namespace tbias {
namespace seg {

SegLaunch seg_launcher_1_8(int per, int32_t dtype) {
  switch (per) {
#define TB_SEG_CASE(P) \
  case P:            \
    return dtype == TB_F32 ? &launch_seg<LoadF32, P> : &launch_seg<LoadBF16, P>;
     TB_SEG_CASE(1) TB_SEG_CASE(2) TB_SEG_CASE(3) TB_SEG_CASE(4) TB_SEG_CASE(5) TB_SEG_CASE(6) TB_SEG_CASE(7) TB_SEG_CASE(8)
#undef TB_SEG_CASE
    default:
      return nullptr;
  }
}

}  // namespace seg
}  // namespace tbias
