// ntc_decode_l2c16_h128.hip -- decode kernels of the shape family: two levels of 16 channels, 128-wide hidden layers.
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<2, 16, 0, 128>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
