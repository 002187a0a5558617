// ntc_divergence.hip -- distinct decoders per wave-sized block (Sec. 2).
//
// The paper's divergence map D(i,j) counts the distinct ids inside a screen
// block; its metric (Eq. normalized_ones_metric) is the mean excess of D over
// one.  Here a block is a window of `wave` consecutive entries of an order of
// the query stream (the stream itself, or the binned permutation), which is
// exactly the set of queries one wave of the decoder processes.
//
// One wave per window, grid-stride over windows; the distinct count comes from
// a ballot peel loop.  Totals are reduced per workgroup in LDS and added to the
// u64 totals with one atomic per workgroup and total.
#include "ntc_internal.h"

namespace ntc {
namespace {

__global__ void divergence_clear(uint64_t *totals) {
  if (threadIdx.x < 4) totals[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(kBlock)
divergence_windows(const uint32_t *__restrict__ tex_id, uint32_t n,
                   const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                   uint32_t n_decoders, const uint32_t *__restrict__ order, uint64_t len,
                   uint32_t wave, uint64_t n_windows, uint32_t *__restrict__ per_wave,
                   uint64_t *__restrict__ totals) {
  __shared__ uint64_t lds_sum[kWavesPerBlock][4];
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  uint64_t kept = 0, sum = 0, divergent = 0, mx = 0;  // wave-uniform
  const uint64_t stride = (uint64_t)gridDim.x * kWavesPerBlock;
  for (uint64_t win = (uint64_t)blockIdx.x * kWavesPerBlock + w; win < n_windows; win += stride) {
    const uint64_t i = win * wave + lane;
    uint32_t d = 0xFFFFFFFFu;
    if (lane < wave && i < len) {
      const uint32_t q = order ? order[i] : (uint32_t)i;
      if (q < n) {
        const uint32_t t = tex_id[q];
        if (t < n_textures) {
          const uint32_t dd = tex_to_dec[t];
          if (dd < n_decoders) d = dd;
        }
      }
    }
    uint64_t todo = ballot(d != 0xFFFFFFFFu);
    uint32_t distinct = 0;
    while (todo) {
      const uint32_t dl = read_lane(d, (uint32_t)__builtin_ctzll(todo));
      todo &= ~ballot(d == dl);
      ++distinct;
    }
    if (lane == 0) per_wave[win] = distinct;
    if (distinct) {
      kept += 1;
      sum += distinct;
      divergent += distinct > 1;
      mx = distinct > mx ? distinct : mx;
    }
  }
  if (lane == 0) {
    lds_sum[w][0] = kept;
    lds_sum[w][1] = sum;
    lds_sum[w][2] = divergent;
    lds_sum[w][3] = mx;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    uint64_t acc = 0;
    for (int k = 0; k < kWavesPerBlock; ++k) {
      const uint64_t v = lds_sum[k][threadIdx.x];
      acc = threadIdx.x == 3 ? (v > acc ? v : acc) : acc + v;
    }
    if (threadIdx.x == 3) {
      if (acc) atomicMax((unsigned long long *)&totals[3], (unsigned long long)acc);
    } else if (acc) {
      atomicAdd((unsigned long long *)&totals[threadIdx.x], (unsigned long long)acc);
    }
  }
}

}  // namespace

int launch_divergence(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                      int64_t len, int32_t wave, uint32_t *per_wave, uint64_t *totals,
                      hipStream_t stream) {
  hipLaunchKernelGGL(divergence_clear, dim3(1), dim3(kWave), 0, stream, totals);
  const uint64_t n_windows = ((uint64_t)len + wave - 1) / wave;
  if (n_windows > 0) {
    uint64_t blocks = (n_windows + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks > 2048) blocks = 2048;
    hipLaunchKernelGGL(divergence_windows, dim3((unsigned)blocks), dim3(kBlock), 0, stream,
                       tex_id, (uint32_t)n, tex_to_dec, (uint32_t)n_textures,
                       (uint32_t)n_decoders, order, (uint64_t)len, (uint32_t)wave, n_windows,
                       per_wave, totals);
  }
  return hip_status(hipGetLastError());
}

}  // namespace ntc
