// ntc_decode_l2c16.hip -- decode kernels of the shape family: two levels of 16 channels, 64-wide hidden layers (32-64-64-8: the single, divergent and clustered 4K configurations).
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<2, 16, 0, 64>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
