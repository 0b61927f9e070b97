// Host dispatch of the decode launch and occupancy queries to the
// translation unit that holds each score mode's kernels.
#include "pot_launch.hpp"

namespace potattn {

int decode_occupancy(int mode, int G, int mant_bits, int vf, bool pool) {
  switch (mode) {
    case kScorePot:
      return vf == 1 ? occupancy_mode_vf<kScorePot, 1>(G, mant_bits, pool)
             : vf == 2 ? occupancy_mode_vf<kScorePot, 2>(G, mant_bits, pool)
                       : occupancy_mode_vf<kScorePot, 0>(G, mant_bits, pool);
    case kScoreDs4a:
      return vf == 1 ? occupancy_mode_vf<kScoreDs4a, 1>(G, mant_bits, pool)
             : vf == 2 ? occupancy_mode_vf<kScoreDs4a, 2>(G, mant_bits, pool)
                       : occupancy_mode_vf<kScoreDs4a, 0>(G, mant_bits, pool);
    case kScoreInt8: return occupancy_mode_vf<kScoreInt8, 0>(G, 0, pool);
    case kScoreFp16: return occupancy_mode_vf<kScoreFp16, 0>(G, 0, pool);
    default: return 0;
  }
}

hipError_t launch_decode(int mode, int G, int mant_bits, bool debug, int vf,
                         const DecodeArgs& a, hipStream_t stream, hipEvent_t ev_begin,
                         hipEvent_t ev_end) {
  if (vf < 0 || vf > 2) return hipErrorInvalidValue;
  switch (mode) {
    case kScorePot:
      return vf == 1 ? launch_mode_vf<kScorePot, 1>(G, mant_bits, debug, a, stream, ev_begin, ev_end)
             : vf == 2
                 ? launch_mode_vf<kScorePot, 2>(G, mant_bits, debug, a, stream, ev_begin, ev_end)
                 : launch_mode_vf<kScorePot, 0>(G, mant_bits, debug, a, stream, ev_begin, ev_end);
    case kScoreDs4a:
      if (vf != 0 && mant_bits != 0) return hipErrorInvalidValue;
      return vf == 1 ? launch_mode_vf<kScoreDs4a, 1>(G, 0, debug, a, stream, ev_begin, ev_end)
             : vf == 2
                 ? launch_mode_vf<kScoreDs4a, 2>(G, 0, debug, a, stream, ev_begin, ev_end)
                 : launch_mode_vf<kScoreDs4a, 0>(G, mant_bits, debug, a, stream, ev_begin, ev_end);
    case kScoreInt8:
      if (vf != 0) return hipErrorInvalidValue;
      return launch_mode_vf<kScoreInt8, 0>(G, 0, debug, a, stream, ev_begin, ev_end);
    case kScoreFp16:
      if (vf != 0) return hipErrorInvalidValue;
      return launch_mode_vf<kScoreFp16, 0>(G, 0, debug, a, stream, ev_begin, ev_end);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace potattn
