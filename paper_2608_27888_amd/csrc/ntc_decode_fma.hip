// ntc_decode_fma.hip -- the per-lane vector-FMA decode engine (NTC_ENGINE_FMA) of every
// shape family.
#include "ntc_decode_launch.h"

namespace ntc {

template int launch_decode_fma_shape<2, 8, 0, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 8, 0, 128>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 8, 16, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 8, 32, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 16, 0, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 16, 0, 128>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 16, 16, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<2, 16, 32, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<3, 16, 0, 64>(const DecodeArgs &, hipStream_t);
template int launch_decode_fma_shape<3, 16, 0, 128>(const DecodeArgs &, hipStream_t);

}  // namespace ntc
