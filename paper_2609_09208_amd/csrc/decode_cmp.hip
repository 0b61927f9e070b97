// Decode kernels of the comparators: INT8 keys and fp16 keys.
#include "decode_kernel.hpp"

namespace potattn {

template hipError_t launch_mode_vf<kScoreInt8, 0>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScoreInt8, 0>(int, int, bool);
template hipError_t launch_mode_vf<kScoreFp16, 0>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScoreFp16, 0>(int, int, bool);

}  // namespace potattn
