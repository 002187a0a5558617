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
//
// The 2-D map takes one wave per screen block.  The block's samples are walked
// 64 at a time as one flat range (row segments back to back); each id sets its
// bit in a wave-private LDS bitmap over the decoder ids, and the lanes whose
// atomic OR found the bit clear are the first occurrences, counted with a
// ballot.  The bitmap is cleared after each block.
#include "ntc_internal.h"

namespace ntc {
namespace {

__global__ void divergence_clear(uint64_t *totals) {
  if (threadIdx.x < 4) totals[threadIdx.x] = 0;
}

// Adds this workgroup's four totals (per-wave values in lds_sum) to `totals`.
__device__ void flush_totals(uint64_t (*lds_sum)[4], uint64_t *totals) {
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
  flush_totals(lds_sum, totals);
}

__global__ void __launch_bounds__(kBlock)
divergence_map_clear(uint32_t *__restrict__ histogram, uint32_t hist_len,
                     uint64_t *__restrict__ totals) {
  for (uint32_t i = threadIdx.x; i < hist_len; i += kBlock) histogram[i] = 0;
  if (threadIdx.x < 4) totals[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(kBlock)
divergence_blocks(const uint32_t *__restrict__ tex_id, uint32_t width, uint32_t height,
                  uint32_t spp, const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                  uint32_t n_decoders, uint32_t block_w, uint32_t block_h, uint32_t blocks_x,
                  uint32_t n_blocks, uint32_t *__restrict__ map, uint32_t *__restrict__ histogram,
                  uint32_t hist_len, uint64_t *__restrict__ totals) {
  // LDS: kWavesPerBlock bitmaps of `words` words, then the workgroup histogram
  extern __shared__ uint32_t lds[];
  __shared__ uint64_t lds_sum[kWavesPerBlock][4];
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  const uint32_t words = (n_decoders + 31) / 32;
  uint32_t *bits = lds + w * words;
  uint32_t *lhist = lds + kWavesPerBlock * words;
  for (uint32_t i = threadIdx.x; i < kWavesPerBlock * words + hist_len; i += kBlock) lds[i] = 0;
  __syncthreads();
  uint64_t kept = 0, sum = 0, divergent = 0, mx = 0;  // wave-uniform
  const uint32_t stride = gridDim.x * kWavesPerBlock;
  for (uint32_t blk = blockIdx.x * kWavesPerBlock + w; blk < n_blocks; blk += stride) {
    const uint32_t bi = blk / blocks_x, bj = blk % blocks_x;
    const uint32_t x0 = bj * block_w, x1 = min(width, x0 + block_w);
    const uint32_t y0 = bi * block_h, y1 = min(height, y0 + block_h);
    const uint32_t seg = (x1 - x0) * spp;  // samples per row segment
    const uint32_t total = seg * (y1 - y0);
    uint32_t distinct = 0;
    for (uint32_t off = 0; off < total; off += kWave) {
      const uint32_t i = off + lane;
      bool fresh = false;
      if (i < total) {
        const uint32_t y = y0 + i / seg, k = i % seg;
        const uint32_t t = tex_id[((uint64_t)y * width + x0) * spp + k];
        if (t < n_textures) {
          const uint32_t d = tex_to_dec[t];
          if (d < n_decoders) {
            const uint32_t bit = 1u << (d & 31);
            fresh = (atomicOr(&bits[d >> 5], bit) & bit) == 0;
          }
        }
      }
      distinct += (uint32_t)__builtin_popcountll(ballot(fresh));
    }
    for (uint32_t k = lane; k < words; k += kWave) bits[k] = 0;
    if (lane == 0) {
      map[blk] = distinct;
      atomicAdd(&lhist[min(distinct, hist_len - 1)], 1u);
    }
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
  for (uint32_t i = threadIdx.x; i < hist_len; i += kBlock)
    if (lhist[i]) atomicAdd(&histogram[i], lhist[i]);
  flush_totals(lds_sum, totals);
}

}  // namespace

int launch_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                          const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                          int32_t block_w, int32_t block_h, uint32_t *map, uint32_t *histogram,
                          int32_t hist_len, uint64_t *totals, hipStream_t stream) {
  hipLaunchKernelGGL(divergence_map_clear, dim3(1), dim3(kBlock), 0, stream, histogram,
                     (uint32_t)hist_len, totals);
  const uint32_t bx = (uint32_t)((width + block_w - 1) / block_w);
  const uint32_t by = (uint32_t)((height + block_h - 1) / block_h);
  const uint32_t n_blocks = bx * by;
  const uint32_t words = ((uint32_t)n_decoders + 31) / 32;
  const size_t lds = ((size_t)kWavesPerBlock * words + (size_t)hist_len) * sizeof(uint32_t);
  uint64_t groups = ((uint64_t)n_blocks + kWavesPerBlock - 1) / kWavesPerBlock;
  if (groups > 2048) groups = 2048;
  hipLaunchKernelGGL(divergence_blocks, dim3((unsigned)groups), dim3(kBlock), lds, stream, tex_id,
                     (uint32_t)width, (uint32_t)height, (uint32_t)spp, tex_to_dec,
                     (uint32_t)n_textures, (uint32_t)n_decoders, (uint32_t)block_w,
                     (uint32_t)block_h, bx, n_blocks, map, histogram, (uint32_t)hist_len, totals);
  return hip_status(hipGetLastError());
}

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
