// Host-side tables of the compiled rotary axis maps: which compile-time map a
// prcr_rope selects, and the axis of each rotary pair under it.
#include "prcr_internal.h"

namespace prcr {

AxisMapId axis_map_id(const prcr_rope &rope) {
  const int *s = rope.section;
  // Every pair on the t axis (plain 1-D rotary at position t) is the same map
  // whether the sections are read as blocks or interleaved.
  if (s[1] == 0 && s[2] == 0) {
    if (rope.head_dim == 64 && s[0] == 32) return AxisMapId::kS_32_0_0;
    if (rope.head_dim == 128 && s[0] == 64) return AxisMapId::kS_64_0_0;
  }
  if (rope.head_dim == 64) {
    if (!rope.interleaved && s[0] == 8 && s[1] == 12 && s[2] == 12) return AxisMapId::kS_8_12_12;
    if (rope.interleaved && s[0] == 11 && s[1] == 11 && s[2] == 10) return AxisMapId::kI_11_11_10;
  } else if (rope.head_dim == 128) {
    if (!rope.interleaved && s[0] == 16 && s[1] == 24 && s[2] == 24) return AxisMapId::kS_16_24_24;
    if (rope.interleaved && s[0] == 22 && s[1] == 21 && s[2] == 21) return AxisMapId::kI_22_21_21;
    if (rope.interleaved && s[0] == 24 && s[1] == 20 && s[2] == 20) return AxisMapId::kI_24_20_20;
  }
  return AxisMapId::kUnsupported;
}

int axis_of_pair(AxisMapId id, int i) {
  switch (id) {
    case AxisMapId::kS_8_12_12: return Sectioned<8, 12, 12>::axis(i);
    case AxisMapId::kI_11_11_10: return Interleaved<11, 11, 10>::axis(i);
    case AxisMapId::kS_16_24_24: return Sectioned<16, 24, 24>::axis(i);
    case AxisMapId::kI_22_21_21: return Interleaved<22, 21, 21>::axis(i);
    case AxisMapId::kI_24_20_20: return Interleaved<24, 20, 20>::axis(i);
    case AxisMapId::kS_32_0_0: return Sectioned<32, 0, 0>::axis(i);
    case AxisMapId::kS_64_0_0: return Sectioned<64, 0, 0>::axis(i);
    default: return -1;
  }
}

}  // namespace prcr
