// ntc_decode.hip -- shape dispatch of the decode kernels.  The kernels live in
// ntc_decode_kernels.h; each shape family is instantiated in its own
// translation unit (ntc_decode_<family>.hip).
#include "ntc_internal.h"

namespace ntc {

int launch_decode_fma(const DecodeArgs &a, int n_levels, int channels, int hidden,
                      hipStream_t stream) {
  if (a.out_dim % 8 != 0) return NTC_ERR_UNSUPPORTED;
  if (a.n_hidden < 1 || a.n_hidden > 2) return NTC_ERR_UNSUPPORTED;
  if (a.pe_octaves == 0) {
    if (hidden == 64) {
      if (n_levels == 2 && channels == 8) return launch_decode_fma_shape<2, 8, 0, 64>(a, stream);
      if (n_levels == 2 && channels == 16) return launch_decode_fma_shape<2, 16, 0, 64>(a, stream);
      if (n_levels == 3 && channels == 16) return launch_decode_fma_shape<3, 16, 0, 64>(a, stream);
    } else if (hidden == 128) {
      if (n_levels == 2 && channels == 8) return launch_decode_fma_shape<2, 8, 0, 128>(a, stream);
      if (n_levels == 2 && channels == 16) return launch_decode_fma_shape<2, 16, 0, 128>(a, stream);
      if (n_levels == 3 && channels == 16) return launch_decode_fma_shape<3, 16, 0, 128>(a, stream);
    }
  } else if (hidden == 64 && n_levels == 2 && a.n_hidden == 1) {
    if (channels == 8 && a.pe_octaves == 4) return launch_decode_fma_shape<2, 8, 16, 64>(a, stream);
    if (channels == 8 && a.pe_octaves == 8) return launch_decode_fma_shape<2, 8, 32, 64>(a, stream);
    if (channels == 16 && a.pe_octaves == 4) return launch_decode_fma_shape<2, 16, 16, 64>(a, stream);
    if (channels == 16 && a.pe_octaves == 8) return launch_decode_fma_shape<2, 16, 32, 64>(a, stream);
  }
  return NTC_ERR_UNSUPPORTED;
}

int launch_decode(const DecodeArgs &a, int n_levels, int channels, int feat, int hidden,
                  hipStream_t stream) {
  (void)feat;
  if (a.pe_octaves == 0) {
    if (hidden == 64) {
      if (n_levels == 2 && channels == 8) return launch_decode_shape<2, 8, 0, 64>(a, stream);
      if (n_levels == 2 && channels == 16) return launch_decode_shape<2, 16, 0, 64>(a, stream);
      if (n_levels == 3 && channels == 16) return launch_decode_shape<3, 16, 0, 64>(a, stream);
    } else if (hidden == 128) {
      if (n_levels == 2 && channels == 8) return launch_decode_shape<2, 8, 0, 128>(a, stream);
      if (n_levels == 2 && channels == 16) return launch_decode_shape<2, 16, 0, 128>(a, stream);
      if (n_levels == 3 && channels == 16) return launch_decode_shape<3, 16, 0, 128>(a, stream);
    }
  } else if (hidden == 64 && n_levels == 2) {
    if (channels == 8 && a.pe_octaves == 4) return launch_decode_shape<2, 8, 16, 64>(a, stream);
    if (channels == 8 && a.pe_octaves == 8) return launch_decode_shape<2, 8, 32, 64>(a, stream);
    if (channels == 16 && a.pe_octaves == 4) return launch_decode_shape<2, 16, 16, 64>(a, stream);
    if (channels == 16 && a.pe_octaves == 8) return launch_decode_shape<2, 16, 32, 64>(a, stream);
  }
  return NTC_ERR_UNSUPPORTED;
}

}  // namespace ntc
