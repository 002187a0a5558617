// ntc_decode_l3c16.hip -- decode kernels of the shape family: three levels of 16 channels, 64-wide hidden layers.
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<3, 16, 0, 64>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
