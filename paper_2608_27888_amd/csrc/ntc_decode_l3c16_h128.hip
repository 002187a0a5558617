// ntc_decode_l3c16_h128.hip -- decode kernels of the shape family: three levels of 16 channels, 128-wide hidden layers (48-128-128-128-8: the wide trilinear configuration).
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<3, 16, 0, 128>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
