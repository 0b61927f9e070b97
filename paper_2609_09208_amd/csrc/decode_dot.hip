// Decode kernels: codes decoded to integer weights on the dot unit (every value format).
#include "decode_kernel.hpp"

namespace potattn {

template hipError_t launch_mode_vf<kScoreDs4a, 0>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScoreDs4a, 0>(int, int, bool);
template hipError_t launch_mode_vf<kScoreDs4a, 1>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScoreDs4a, 1>(int, int, bool);
template hipError_t launch_mode_vf<kScoreDs4a, 2>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScoreDs4a, 2>(int, int, bool);

}  // namespace potattn
