// Decode kernels: shift-accumulate scores, INT8 values, power-of-two weights.
#include "decode_kernel.hpp"

namespace potattn {

template hipError_t launch_mode_vf<kScorePot, 2>(int, int, bool, const DecodeArgs&, hipStream_t,
                                                 hipEvent_t, hipEvent_t);
template int occupancy_mode_vf<kScorePot, 2>(int, int, bool);

}  // namespace potattn
