// ntc_decode_l2c16_pe.hip -- decode kernels of the shape family: two levels of 16 channels with 4 or 8 positional octaves (the Sec. 4 setup decoder).
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<2, 16, 16, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_shape<2, 16, 32, 64>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
