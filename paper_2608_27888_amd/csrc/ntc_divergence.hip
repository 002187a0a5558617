// ntc_divergence.hip -- distinct decoders per wave-sized block (Sec. 2).
//
// The paper's divergence map D(i,j) counts the distinct ids inside a screen
// block; its metric (Eq. normalized_ones_metric) is the mean excess of D over
// one.  Here a block is a window of `wave` consecutive entries of an order of
// the query stream (the stream itself, or the binned permutation), which is
// exactly the set of queries one wave of the decoder processes.
//
// One wave per window, grid-stride over batches of windows whose loads are all
// issued before any is counted; the distinct count comes from a ballot peel
// loop.  Totals are reduced per workgroup in LDS and added to the u64 totals
// with one atomic per workgroup and total.
//
// The 2-D map takes one wave per screen block, blocks taken in batches whose
// first 64 samples are loaded together.  The block's samples are walked
// 64 at a time as one flat range (row segments back to back), each chunk's
// distinct ids peeled with ballots.  A block of at most 64 samples is counted
// by the peel alone; in a longer one each peeled id sets its bit in a
// wave-private LDS bitmap over the decoder ids (one atomic OR from one lane),
// and the ids whose bit was clear are the first occurrences.  The bitmap is
// cleared after each such block.  (An atomic OR from every lane serialises on
// one LDS word when the block holds one decoder.)
#include "ntc_internal.h"

namespace ntc {
namespace {

// Divergence workgroups are 16 waves: each adds its totals to the four u64 outputs
// with one atomic per total, and those atomics all hit one cache line, so fewer,
// larger workgroups keep them off the kernel's critical path.
constexpr int kDivWaves = 16;
constexpr int kDivBlock = kDivWaves * kWave;
// At most one workgroup per CU: the final atomics, not the loads, set these kernels' time.
constexpr uint64_t kDivGroups = 256;

__global__ void divergence_clear(uint64_t *totals) {
  if (threadIdx.x < 4) totals[threadIdx.x] = 0;
}

// Adds this workgroup's four totals (per-wave values in lds_sum) to `totals`.
__device__ void flush_totals(uint64_t (*lds_sum)[4], uint64_t *totals) {
  if (threadIdx.x < 4) {
    uint64_t acc = 0;
    for (int k = 0; k < kDivWaves; ++k) {
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

// Windows a wave takes at once: their loads are all issued before any of them
// is counted, so the chain order -> tex_id -> map is paid once per batch.
constexpr int kWinBatch = 16;

__global__ void __launch_bounds__(kDivBlock)
divergence_windows(const uint32_t *__restrict__ tex_id, uint32_t n,
                   const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                   uint32_t n_decoders, const uint32_t *__restrict__ order, uint64_t len,
                   uint32_t wave, uint64_t n_windows, uint32_t *__restrict__ per_wave,
                   uint64_t *__restrict__ totals) {
  __shared__ uint64_t lds_sum[kDivWaves][4];
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  uint64_t kept = 0, sum = 0, divergent = 0, mx = 0;  // wave-uniform
  const uint64_t waves = (uint64_t)gridDim.x * kDivWaves;
  // Loads are unconditional, with entry 0 standing in for an entry that does not
  // count; entry 0 exists wherever it is read (n_windows > 0 means len > 0, and
  // tex_id / tex_to_dec are read only when n / n_textures are positive).
  const bool have_q = n > 0, have_t = n_textures > 0;
  for (uint64_t first = (uint64_t)blockIdx.x * kDivWaves + w; first < n_windows;
       first += waves * kWinBatch) {
    bool ok[kWinBatch];
    uint32_t v[kWinBatch];
#pragma unroll
    for (int k = 0; k < kWinBatch; ++k) {
      const uint64_t win = first + (uint64_t)k * waves;
      const uint64_t i = win * wave + lane;
      ok[k] = win < n_windows && lane < wave && i < len;
      v[k] = order ? order[ok[k] ? i : 0] : (uint32_t)i;  // the query
    }
#pragma unroll
    for (int k = 0; k < kWinBatch; ++k) {
      ok[k] = ok[k] && v[k] < n;
      v[k] = have_q ? tex_id[ok[k] ? v[k] : 0] : 0u;  // its texture
    }
#pragma unroll
    for (int k = 0; k < kWinBatch; ++k) {
      ok[k] = ok[k] && v[k] < n_textures;
      const uint32_t dd = have_t ? tex_to_dec[ok[k] ? v[k] : 0] : 0u;  // its decoder
      v[k] = ok[k] && dd < n_decoders ? dd : 0xFFFFFFFFu;
    }
#pragma unroll
    for (int k = 0; k < kWinBatch; ++k) {
      const uint64_t win = first + (uint64_t)k * waves;
      if (win < n_windows) {
        const uint32_t d = v[k];
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

// Screen blocks a wave takes at once (their first 64 samples loaded together).
constexpr int kBlkBatch = 16;

__global__ void __launch_bounds__(kDivBlock)
divergence_blocks(const uint32_t *__restrict__ tex_id, uint32_t width, uint32_t height,
                  uint32_t spp, const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                  uint32_t n_decoders, uint32_t block_w, uint32_t block_h, uint32_t blocks_x,
                  uint32_t n_blocks, uint32_t *__restrict__ map, uint32_t *__restrict__ histogram,
                  uint32_t hist_len, uint64_t *__restrict__ totals) {
  // LDS: kDivWaves bitmaps of `words` words, then the workgroup histogram
  extern __shared__ uint32_t lds[];
  __shared__ uint64_t lds_sum[kDivWaves][4];
  const uint32_t lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform
  const uint32_t words = (n_decoders + 31) / 32;
  uint32_t *bits = lds + w * words;
  uint32_t *lhist = lds + kDivWaves * words;
  for (uint32_t i = threadIdx.x; i < kDivWaves * words + hist_len; i += kDivBlock) lds[i] = 0;
  __syncthreads();
  uint64_t kept = 0, sum = 0, divergent = 0, mx = 0;  // wave-uniform
  const uint32_t stride = gridDim.x * kDivWaves;
  const bool have_t = n_textures > 0;  // tex_to_dec[0] exists
  // Frame index of sample i of block blk (row segments back to back); total =
  // the block's sample count.  Indexes past the block are never read.  The block's
  // geometry is wave-uniform (scalar); i / seg, per lane, comes from a float
  // reciprocal corrected by one step each way, exact while i < 2^20 (the estimate
  // is then within 1/4 of i / seg), else from an integer division.
  auto sample_index = [&](uint32_t blk, uint32_t i, uint32_t &total) -> uint64_t {
    const uint32_t bi = blk / blocks_x, bj = blk % blocks_x;
    const uint32_t x0 = bj * block_w, x1 = min(width, x0 + block_w);
    const uint32_t y0 = bi * block_h, y1 = min(height, y0 + block_h);
    const uint32_t seg = (x1 - x0) * spp;  // samples per row segment
    total = seg * (y1 - y0);
    uint32_t r, k;
    if (total < (1u << 20)) {
      r = (uint32_t)((float)i * (1.0f / (float)seg));
      int32_t rem = (int32_t)(i - r * seg);
      if (rem < 0) {
        --r;
        rem += (int32_t)seg;
      } else if (rem >= (int32_t)seg) {
        ++r;
        rem -= (int32_t)seg;
      }
      k = (uint32_t)rem;
    } else {
      r = i / seg;
      k = i % seg;
    }
    return ((uint64_t)(y0 + r) * width + x0) * spp + k;
  };
  constexpr uint32_t kNoDec = 0xFFFFFFFFu;
  // a wave takes kBlkBatch consecutive blocks (neighbours along a block row, which
  // share the cache lines of their row segments)
  for (uint32_t first = (blockIdx.x * kDivWaves + w) * kBlkBatch; first < n_blocks;
       first += stride * kBlkBatch) {
    // the first 64 samples of kBlkBatch blocks: every load issued before any is used
    // (sample 0 of the frame stands in for a lane past its block)
    uint32_t d0[kBlkBatch];
    bool ok[kBlkBatch];
#pragma unroll
    for (int j = 0; j < kBlkBatch; ++j) {
      const uint32_t blk = first + (uint32_t)j;
      uint32_t total = 0;
      const uint64_t at = sample_index(blk < n_blocks ? blk : 0, lane, total);
      ok[j] = blk < n_blocks && lane < total;
      d0[j] = tex_id[ok[j] ? at : 0];
    }
#pragma unroll
    for (int j = 0; j < kBlkBatch; ++j) {
      ok[j] = ok[j] && d0[j] < n_textures;
      const uint32_t dd = have_t ? tex_to_dec[ok[j] ? d0[j] : 0] : 0u;
      d0[j] = ok[j] && dd < n_decoders ? dd : kNoDec;
    }
#pragma unroll
    for (int j = 0; j < kBlkBatch; ++j) {
      const uint32_t blk = first + (uint32_t)j;
      if (blk < n_blocks) {
        uint32_t total = 0;
        (void)sample_index(blk, 0, total);
        uint32_t distinct = 0;
        for (uint32_t off = 0; off < total; off += kWave) {
          const uint32_t i = off + lane;
          uint32_t d = kNoDec;
          if (off == 0) {
            d = d0[j];
          } else if (i < total) {
            uint32_t tot_unused;
            const uint32_t t = tex_id[sample_index(blk, i, tot_unused)];
            if (t < n_textures) {
              const uint32_t dd = tex_to_dec[t];
              if (dd < n_decoders) d = dd;
            }
          }
          // peel the chunk's distinct ids; a block of one chunk needs no bitmap,
          // a longer one sets one bit per id and chunk (from one lane)
          uint64_t todo = ballot(d != kNoDec);
          while (todo) {
            const uint32_t dl = read_lane(d, (uint32_t)__builtin_ctzll(todo));
            todo &= ~ballot(d == dl);
            if (total <= (uint32_t)kWave) {
              ++distinct;
            } else {
              const uint32_t bit = 1u << (dl & 31);
              uint32_t old = 0;
              if (lane == 0) old = atomicOr(&bits[dl >> 5], bit);
              distinct += (__builtin_amdgcn_readfirstlane(old) & bit) == 0;
            }
          }
        }
        if (total > (uint32_t)kWave)
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
    }
  }
  if (lane == 0) {
    lds_sum[w][0] = kept;
    lds_sum[w][1] = sum;
    lds_sum[w][2] = divergent;
    lds_sum[w][3] = mx;
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < hist_len; i += kDivBlock)
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
  const size_t lds = ((size_t)kDivWaves * words + (size_t)hist_len) * sizeof(uint32_t);
  const uint64_t per_group = (uint64_t)kDivWaves * kBlkBatch;  // one batch per wave
  uint64_t groups = ((uint64_t)n_blocks + per_group - 1) / per_group;
  if (groups > kDivGroups) groups = kDivGroups;
  hipLaunchKernelGGL(divergence_blocks, dim3((unsigned)groups), dim3(kDivBlock), lds, stream, tex_id,
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
    const uint64_t per_group = (uint64_t)kDivWaves * kWinBatch;  // one batch per wave
    uint64_t blocks = (n_windows + per_group - 1) / per_group;
    if (blocks > kDivGroups) blocks = kDivGroups;
    hipLaunchKernelGGL(divergence_windows, dim3((unsigned)blocks), dim3(kDivBlock), 0, stream,
                       tex_id, (uint32_t)n, tex_to_dec, (uint32_t)n_textures,
                       (uint32_t)n_decoders, order, (uint64_t)len, (uint32_t)wave, n_windows,
                       per_wave, totals);
  }
  return hip_status(hipGetLastError());
}

}  // namespace ntc
