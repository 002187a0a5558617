// ntc_gather.hip -- the feature vectors of a query stream alone: the gather
// step of the decode (bilinear samples of the texture's latent levels,
// concatenated finest first, levels blended by mip; Sec. 1 "latent pyramids or
// grids"), without the MLP.  The rows are the very values the decode's MLP
// consumes: the same device functions compute them, interpolation in packed
// fp16.
//
// One lane per query, grid stride.  Each lane loads its query, its 2x2 taps per
// level as 16-byte pieces of texel rows, interpolates, and writes its row with
// 16-byte stores (fp32 rows: the fp16 values widened, exactly).
#include "ntc_decode_kernels.h"

namespace ntc {
namespace {

template <int NL, int CH, bool MIP, bool F16>
__global__ void __launch_bounds__(kBlock) gather_rows(const DecodeArgs a) {
  constexpr int F = NL * CH;  // features per row, a multiple of 8
  const uint64_t stride = (uint64_t)gridDim.x * kBlock;
  for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < a.n; i += stride) {
    const Query qq = validate(a, load_query<NL, MIP>(a, (uint32_t)i, true));
    uint32_t x[F / 2];
    gather<NL, CH, 0, MIP>(a, qq, x);  // an invalid query samples texture 0
    if (!qq.valid) continue;
    if constexpr (F16) {
      uint4 *row = (uint4 *)((uint16_t *)a.out + i * F);
#pragma unroll
      for (int k = 0; k < F / 8; ++k)
        row[k] = make_uint4(x[4 * k], x[4 * k + 1], x[4 * k + 2], x[4 * k + 3]);
    } else {
      float4 *row = (float4 *)((float *)a.out + i * F);
#pragma unroll
      for (int k = 0; k < F / 4; ++k) {
        const half2v p = as_h2(x[2 * k]), r = as_h2(x[2 * k + 1]);
        row[k] = make_float4((float)p[0], (float)p[1], (float)r[0], (float)r[1]);
      }
    }
  }
}

template <int NL, int CH, bool MIP, bool F16>
int launch_rows(const DecodeArgs &a, hipStream_t stream) {
  uint64_t blocks = ((uint64_t)a.n + kBlock - 1) / kBlock;
  if (blocks > 65536) blocks = 65536;  // grid stride beyond
  hipLaunchKernelGGL((gather_rows<NL, CH, MIP, F16>), dim3((unsigned)blocks), dim3(kBlock), 0,
                     stream, a);
  return hip_status(hipGetLastError());
}

template <int NL, int CH>
int launch_shape(const DecodeArgs &a, bool f16, hipStream_t stream) {
  if (a.mip)
    return f16 ? launch_rows<NL, CH, true, true>(a, stream)
               : launch_rows<NL, CH, true, false>(a, stream);
  return f16 ? launch_rows<NL, CH, false, true>(a, stream)
             : launch_rows<NL, CH, false, false>(a, stream);
}

}  // namespace

int launch_gather(const DecodeArgs &a, int n_levels, int channels, bool f16, hipStream_t stream) {
  if (n_levels == 2 && channels == 8) return launch_shape<2, 8>(a, f16, stream);
  if (n_levels == 2 && channels == 16) return launch_shape<2, 16>(a, f16, stream);
  if (n_levels == 3 && channels == 16) return launch_shape<3, 16>(a, f16, stream);
  return NTC_ERR_UNSUPPORTED;
}

}  // namespace ntc
