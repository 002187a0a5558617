// ntc_decode_l2c8.hip -- decode kernels of the shape family: two levels of 8 channels (16 features, the tiny configuration; with 4 or 8 positional octaves).
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_shape<2, 8, 0, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_shape<2, 8, 0, 128>(const DecodeArgs &, hipStream_t);
template int launch_decode_shape<2, 8, 16, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_shape<2, 8, 32, 64>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
