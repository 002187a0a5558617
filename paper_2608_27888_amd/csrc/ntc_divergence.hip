// ntc_divergence.hip -- distinct decoders per wave-sized block (Sec. 2).
//
// The paper's divergence map D(i,j) counts the distinct ids inside a screen
// block; its metric (Eq. normalized_ones_metric) is the mean excess of D over
// one.  Here a block is either a window of `wave` consecutive entries of an
// order of the query stream (the stream itself, or the binned permutation),
// exactly the set of queries one wave of the decoder processes, or a 2-D
// screen block.
//
// Two kernels per call.  The first writes one count per window or block (and
// its workgroup 0 clears the histogram and the totals); the second reduces
// those counts into the histogram and the totals, each of a few workgroups
// adding its share with one atomic per non-zero entry.  No workgroup of the
// counting kernel touches a shared word.
//
// Windows: one wave per window, grid-stride over batches of windows whose loads
// are all issued before any is counted; the distinct count comes from a ballot
// peel loop.
//
// Screen blocks whose row segment is a power-of-two number g <= 64 of samples
// and whose height is at most kTileRows: a wave takes tiles of 64 consecutive
// samples of a block row (64 / g neighbouring blocks), one coalesced load per
// pixel row.  Lane l holds the column of samples of its block's lane group;
// the group's distinct ids are peeled smallest first (a min over the lane's
// rows, then over the g lanes by butterfly shuffles), with vector instructions
// only.  Other geometries: one wave per block, its samples walked 64 at a time
// as one flat range (row segments back to back), each chunk's distinct ids
// peeled with ballots; in a block of more than 64 samples each peeled id sets
// its bit in a wave-private LDS bitmap over the decoder ids, and the ids whose
// bit was clear are first occurrences.
#include "ntc_internal.h"

namespace ntc {
namespace {

constexpr uint32_t kNoDec = 0xFFFFFFFFu;

// Windows: workgroups of 16 waves, at most kDivGroups of them (grid stride).
constexpr int kDivWaves = 16;
constexpr int kDivBlock = kDivWaves * kWave;
constexpr uint64_t kDivGroups = 1024;
// Windows a wave takes at once: their loads are all issued before any of them
// is counted, so the chain order -> tex_id -> map is paid once per batch.
constexpr int kWinBatch = 16;
// Screen tiles: at most this many pixel rows per block.
constexpr int kTileRows = 16;
// Reduction: entries per thread and per workgroup.
constexpr int kReduceThreads = 1024;
constexpr int kReducePerThread = 16;
constexpr uint64_t kReducePerGroup = (uint64_t)kReduceThreads * kReducePerThread;

// Cross-lane steps without LDS: DPP within rows of 16 lanes (quad exchanges,
// then the half-row and row mirrors), permlane swaps across rows.
__device__ __forceinline__ uint32_t dpp_xor1(uint32_t v) {
  return __builtin_amdgcn_update_dpp(v, v, 0xB1, 0xf, 0xf, false);  // quad_perm [1,0,3,2]
}
__device__ __forceinline__ uint32_t dpp_xor2(uint32_t v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x4E, 0xf, 0xf, false);  // quad_perm [2,3,0,1]
}
__device__ __forceinline__ uint32_t dpp_half_mirror(uint32_t v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x141, 0xf, 0xf, false);  // lane i <-> 7 - i
}
__device__ __forceinline__ uint32_t dpp_mirror(uint32_t v) {
  return __builtin_amdgcn_update_dpp(v, v, 0x140, 0xf, 0xf, false);  // lane i <-> 15 - i
}

// Minimum over the aligned group of g lanes (g a power of two <= 64), in every
// lane of the group.  After the four row steps every lane holds its group's
// (or its row's) minimum; a permlane swap then pairs rows 0/1 and 2/3, and one
// more pairs the halves of the wave.
__device__ __forceinline__ uint32_t group_min(uint32_t v, uint32_t g) {
  if (g > 1) v = min(v, dpp_xor1(v));
  if (g > 2) v = min(v, dpp_xor2(v));
  if (g > 4) v = min(v, dpp_half_mirror(v));
  if (g > 8) v = min(v, dpp_mirror(v));
  if (g > 16) {
    const auto p = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    v = min(p[0], p[1]);
  }
  if (g > 32) {
    const auto p = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    v = min(p[0], p[1]);
  }
  return v;
}

// Wave sum and maximum (every lane active), wave-uniform results.
__device__ __forceinline__ uint32_t wave_sum32(uint32_t v) {
  v += dpp_xor1(v);
  v += dpp_xor2(v);
  v += dpp_half_mirror(v);
  v += dpp_mirror(v);
  return read_lane(v, 0) + read_lane(v, 16) + read_lane(v, 32) + read_lane(v, 48);
}
__device__ __forceinline__ uint32_t wave_max32(uint32_t v) {
  v = max(v, dpp_xor1(v));
  v = max(v, dpp_xor2(v));
  v = max(v, dpp_half_mirror(v));
  v = max(v, dpp_mirror(v));
  return max(max(read_lane(v, 0), read_lane(v, 16)), max(read_lane(v, 32), read_lane(v, 48)));
}

// Workgroup 0 of a counting kernel clears what the reduction adds into.
__device__ __forceinline__ void clear_outputs(uint32_t b, uint32_t *histogram, uint32_t hist_len,
                                              uint64_t *totals) {
  if (b != 0) return;
  if (histogram)
    for (uint32_t i = threadIdx.x; i < hist_len; i += blockDim.x) histogram[i] = 0;
  if (threadIdx.x < 4) totals[threadIdx.x] = 0;
}

__global__ void __launch_bounds__(kDivBlock)
divergence_windows(const uint32_t *__restrict__ tex_id, uint32_t n,
                   const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                   uint32_t n_decoders, const uint32_t *__restrict__ order, uint64_t len,
                   uint32_t wave, uint64_t n_windows, uint32_t *__restrict__ per_wave,
                   uint64_t *__restrict__ totals) {
  clear_outputs(blockIdx.x, nullptr, 0, totals);
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
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
      v[k] = ok[k] && dd < n_decoders ? dd : kNoDec;
    }
#pragma unroll
    for (int k = 0; k < kWinBatch; ++k) {
      const uint64_t win = first + (uint64_t)k * waves;
      if (win < n_windows) {
        const uint32_t d = v[k];
        uint64_t todo = ballot(d != kNoDec);
        uint32_t distinct = 0;
        while (todo) {
          const uint32_t dl = read_lane(d, (uint32_t)__builtin_ctzll(todo));
          todo &= ~ballot(d == dl);
          ++distinct;
        }
        if (lane == 0) per_wave[win] = distinct;
      }
    }
  }
}

// Screen geometry shared by the block kernels.
struct Screen {
  uint32_t width, height, spp;
  uint32_t block_w, block_h, blocks_x, blocks_y;
};

// A wave takes kTilesPerWave tiles of 64 samples x one block row at once (their
// loads, then their map lookups, all issued before any is counted; one tile per
// wave measured fastest on the 4K frame).  g =
// block_w * spp, a power of two <= 64; ROWS >= block_h.
constexpr int kTilesPerWave = 1;

template <int ROWS>
__global__ void __launch_bounds__(kBlock)
divergence_tiles(const uint32_t *__restrict__ tex_id, Screen sc,
                 const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                 uint32_t n_decoders, uint32_t g, uint64_t tiles_x, uint64_t n_tiles,
                 uint32_t *__restrict__ map, uint32_t *__restrict__ histogram, uint32_t hist_len,
                 uint64_t *__restrict__ totals) {
  clear_outputs(blockIdx.x, histogram, hist_len, totals);
  const uint32_t lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint64_t row_samples = (uint64_t)sc.width * sc.spp;
  const uint64_t waves = (uint64_t)gridDim.x * kWavesPerBlock;
  for (uint64_t first = ((uint64_t)blockIdx.x * kWavesPerBlock + w) * kTilesPerWave;
       first < n_tiles; first += waves * kTilesPerWave) {
    uint32_t v[kTilesPerWave][ROWS];
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
      const uint64_t tile = first + t;
      const uint64_t bi = tile / tiles_x, tc = tile % tiles_x;  // block row, tile column
      const uint64_t s = tc * kWave + lane;                     // this lane's sample column
      const uint64_t y0 = bi * sc.block_h;
#pragma unroll
      for (int r = 0; r < ROWS; ++r) {
        const bool ok = tile < n_tiles && s < row_samples && (uint32_t)r < sc.block_h &&
                        y0 + r < sc.height;
        v[t][r] = tex_id[ok ? (y0 + r) * row_samples + s : 0];  // sample 0 stands in
        v[t][r] = ok ? v[t][r] : n_textures;                    // an id that maps nowhere
      }
    }
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t)
#pragma unroll
      for (int r = 0; r < ROWS; ++r) {
        const uint32_t dd = tex_to_dec[v[t][r] < n_textures ? v[t][r] : 0u];
        v[t][r] = v[t][r] < n_textures && dd < n_decoders ? dd : kNoDec;
      }
#pragma unroll
    for (int t = 0; t < kTilesPerWave; ++t) {
      const uint64_t tile = first + t;
      if (tile >= n_tiles) break;
      // peel the group's smallest remaining id until every group is empty
      uint32_t distinct = 0;
      while (true) {
        uint32_t m = v[t][0];
#pragma unroll
        for (int r = 1; r < ROWS; ++r) m = min(m, v[t][r]);
        m = group_min(m, g);
        if (ballot(m != kNoDec) == 0) break;
        distinct += m != kNoDec ? 1u : 0u;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) v[t][r] = v[t][r] == m ? kNoDec : v[t][r];
      }
      const uint64_t bi = tile / tiles_x, tc = tile % tiles_x;
      const uint64_t j = tc * (kWave / g) + lane / g;  // block column
      if (lane % g == 0 && j < sc.blocks_x) map[bi * sc.blocks_x + j] = distinct;
    }
  }
}

// One wave per block, any geometry.
__global__ void __launch_bounds__(kDivBlock)
divergence_blocks(const uint32_t *__restrict__ tex_id, Screen sc,
                  const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
                  uint32_t n_decoders, uint64_t n_blocks, uint32_t *__restrict__ map,
                  uint32_t *__restrict__ histogram, uint32_t hist_len,
                  uint64_t *__restrict__ totals) {
  clear_outputs(blockIdx.x, histogram, hist_len, totals);
  extern __shared__ uint32_t lds[];  // kDivWaves bitmaps of `words` words
  const uint32_t lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);  // uniform
  const uint32_t words = (n_decoders + 31) / 32;
  uint32_t *bits = lds + w * words;
  for (uint32_t i = lane; i < words; i += kWave) bits[i] = 0;
  // Frame index of sample i of block blk (row segments back to back); total =
  // the block's sample count.  The block's geometry is wave-uniform; i / seg, per
  // lane, comes from a float reciprocal corrected by one step each way, exact
  // while i < 2^20 (the estimate is then within 1/4 of i / seg), else from an
  // integer division.
  auto sample_index = [&](uint64_t blk, uint32_t i, uint32_t &total) -> uint64_t {
    const uint32_t bi = (uint32_t)(blk / sc.blocks_x), bj = (uint32_t)(blk % sc.blocks_x);
    const uint32_t x0 = bj * sc.block_w, x1 = min(sc.width, x0 + sc.block_w);
    const uint32_t y0 = bi * sc.block_h, y1 = min(sc.height, y0 + sc.block_h);
    const uint32_t seg = (x1 - x0) * sc.spp;  // samples per row segment
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
    return ((uint64_t)(y0 + r) * sc.width + x0) * sc.spp + k;
  };
  const uint64_t waves = (uint64_t)gridDim.x * kDivWaves;
  for (uint64_t blk = (uint64_t)blockIdx.x * kDivWaves + w; blk < n_blocks; blk += waves) {
    uint32_t total = 0;
    (void)sample_index(blk, 0, total);
    uint32_t distinct = 0;
    for (uint32_t off = 0; off < total; off += kWave) {
      const uint32_t i = off + lane;
      uint32_t d = kNoDec;
      if (i < total) {
        uint32_t unused;
        const uint32_t t = tex_id[sample_index(blk, i, unused)];
        if (t < n_textures) {
          const uint32_t dd = tex_to_dec[t];
          if (dd < n_decoders) d = dd;
        }
      }
      // peel the chunk's distinct ids; a block of one chunk needs no bitmap, a
      // longer one sets one bit per id and chunk (from one lane)
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
    if (lane == 0) map[blk] = distinct;
  }
}

// Reduces counts[0 .. m) into totals (and the histogram when given): workgroup
// g takes entries [g * kReducePerGroup, ...).  Histogram entries 0..3 (the
// common counts) are tallied in registers, larger ones with LDS atomics; each
// workgroup then adds its non-zero histogram entries and totals to the outputs.
__global__ void __launch_bounds__(kReduceThreads)
divergence_reduce(const uint32_t *__restrict__ counts, uint64_t m,
                  uint32_t *__restrict__ histogram, uint32_t hist_len,
                  uint64_t *__restrict__ totals) {
  extern __shared__ uint32_t lhist[];  // hist_len counters
  constexpr int kWaves = kReduceThreads / kWave;
  __shared__ uint64_t part[kWaves][4];
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  if (histogram)
    for (uint32_t i = threadIdx.x; i < hist_len; i += kReduceThreads) lhist[i] = 0;
  __syncthreads();
  const uint64_t beg = (uint64_t)blockIdx.x * kReducePerGroup;
  const uint64_t end = beg + kReducePerGroup < m ? beg + kReducePerGroup : m;
  // per thread at most kReducePerThread entries of at most 4096 each: 32 bits hold
  // every partial sum of the workgroup
  uint32_t kept = 0, sum = 0, divergent = 0, mx = 0, c[4] = {0, 0, 0, 0};
  // every load of the thread's entries is issued before any is used
  uint32_t vals[kReducePerThread];
  bool in[kReducePerThread];
#pragma unroll
  for (int k = 0; k < kReducePerThread; ++k) {
    const uint64_t i = beg + (uint64_t)k * kReduceThreads + threadIdx.x;
    in[k] = i < end;
    vals[k] = in[k] ? counts[i] : 0u;
  }
#pragma unroll
  for (int k = 0; k < kReducePerThread; ++k) {
    if (!in[k]) continue;
    const uint32_t v = vals[k];
    kept += v > 0;
    sum += v;
    divergent += v > 1;
    mx = max(mx, v);
    if (histogram) {
      const uint32_t bin = min(v, hist_len - 1);
      if (bin < 4) {
#pragma unroll
        for (uint32_t k = 0; k < 4; ++k) c[k] += bin == k ? 1u : 0u;
      } else {
        atomicAdd(&lhist[bin], 1u);
      }
    }
  }
  kept = wave_sum32(kept);
  sum = wave_sum32(sum);
  divergent = wave_sum32(divergent);
  mx = wave_max32(mx);
  if (histogram)
#pragma unroll
    for (uint32_t k = 0; k < 4; ++k) {
      const uint32_t ck = wave_sum32(c[k]);
      if (lane == 0 && ck && k < hist_len) atomicAdd(&lhist[k], ck);
    }
  if (lane == 0) {
    part[w][0] = kept;
    part[w][1] = sum;
    part[w][2] = divergent;
    part[w][3] = mx;
  }
  __syncthreads();
  if (threadIdx.x < 4) {
    uint64_t acc = 0;
    for (int k = 0; k < kWaves; ++k) {
      const uint64_t v = part[k][threadIdx.x];
      acc = threadIdx.x == 3 ? (v > acc ? v : acc) : acc + v;
    }
    if (acc) {
      if (threadIdx.x == 3)
        atomicMax((unsigned long long *)&totals[3], (unsigned long long)acc);
      else
        atomicAdd((unsigned long long *)&totals[threadIdx.x], (unsigned long long)acc);
    }
  }
  if (histogram)
    for (uint32_t i = threadIdx.x; i < hist_len; i += kReduceThreads)
      if (lhist[i]) atomicAdd(&histogram[i], lhist[i]);
}

int launch_reduce(const uint32_t *counts, uint64_t m, uint32_t *histogram, uint32_t hist_len,
                  uint64_t *totals, hipStream_t stream) {
  if (m == 0) return NTC_OK;
  const uint64_t groups = (m + kReducePerGroup - 1) / kReducePerGroup;
  const size_t lds = histogram ? (size_t)hist_len * sizeof(uint32_t) : 0;
  hipLaunchKernelGGL(divergence_reduce, dim3((unsigned)groups), dim3(kReduceThreads), lds, stream,
                     counts, m, histogram, hist_len, totals);
  return NTC_OK;
}

template <int ROWS>
void launch_tiles(const uint32_t *tex_id, const Screen &sc, const uint32_t *tex_to_dec,
                  uint32_t n_textures, uint32_t n_decoders, uint32_t g, uint32_t *map,
                  uint32_t *histogram, uint32_t hist_len, uint64_t *totals, hipStream_t stream) {
  const uint64_t tiles_x = ((uint64_t)sc.width * sc.spp + kWave - 1) / kWave;
  const uint64_t n_tiles = tiles_x * sc.blocks_y;
  const uint64_t per_group = (uint64_t)kWavesPerBlock * kTilesPerWave;
  uint64_t groups = (n_tiles + per_group - 1) / per_group;
  if (groups > 65535) groups = 65535;  // grid stride beyond
  hipLaunchKernelGGL(divergence_tiles<ROWS>, dim3((unsigned)groups), dim3(kBlock), 0, stream,
                     tex_id, sc, tex_to_dec, n_textures, n_decoders, g, tiles_x, n_tiles, map,
                     histogram, hist_len, totals);
}

}  // namespace

int launch_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                          const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                          int32_t block_w, int32_t block_h, uint32_t *map, uint32_t *histogram,
                          int32_t hist_len, uint64_t *totals, hipStream_t stream) {
  Screen sc;
  sc.width = (uint32_t)width;
  sc.height = (uint32_t)height;
  sc.spp = (uint32_t)spp;
  sc.block_w = (uint32_t)block_w;
  sc.block_h = (uint32_t)block_h;
  sc.blocks_x = (uint32_t)((width + block_w - 1) / block_w);
  sc.blocks_y = (uint32_t)((height + block_h - 1) / block_h);
  const uint64_t n_blocks = (uint64_t)sc.blocks_x * sc.blocks_y;
  const uint64_t g = (uint64_t)block_w * spp;  // samples per block row segment
  const uint32_t T = (uint32_t)n_textures, D = (uint32_t)n_decoders, H = (uint32_t)hist_len;
  if (g <= (uint64_t)kWave && (g & (g - 1)) == 0 && block_h <= kTileRows) {
    const uint32_t gg = (uint32_t)g;
    if (block_h <= 1)
      launch_tiles<1>(tex_id, sc, tex_to_dec, T, D, gg, map, histogram, H, totals, stream);
    else if (block_h <= 2)
      launch_tiles<2>(tex_id, sc, tex_to_dec, T, D, gg, map, histogram, H, totals, stream);
    else if (block_h <= 4)
      launch_tiles<4>(tex_id, sc, tex_to_dec, T, D, gg, map, histogram, H, totals, stream);
    else if (block_h <= 8)
      launch_tiles<8>(tex_id, sc, tex_to_dec, T, D, gg, map, histogram, H, totals, stream);
    else
      launch_tiles<16>(tex_id, sc, tex_to_dec, T, D, gg, map, histogram, H, totals, stream);
  } else {
    const uint32_t words = (D + 31) / 32;
    const size_t lds = (size_t)kDivWaves * words * sizeof(uint32_t);
    uint64_t groups = (n_blocks + kDivWaves - 1) / kDivWaves;
    if (groups > kDivGroups) groups = kDivGroups;
    hipLaunchKernelGGL(divergence_blocks, dim3((unsigned)groups), dim3(kDivBlock), lds, stream,
                       tex_id, sc, tex_to_dec, T, D, n_blocks, map, histogram, H, totals);
  }
  launch_reduce(map, n_blocks, histogram, H, totals, stream);
  return hip_status(hipGetLastError());
}

int launch_divergence(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                      int64_t len, int32_t wave, uint32_t *per_wave, uint64_t *totals,
                      hipStream_t stream) {
  const uint64_t n_windows = ((uint64_t)len + wave - 1) / wave;
  const uint64_t per_group = (uint64_t)kDivWaves * kWinBatch;  // one batch per wave
  uint64_t blocks = (n_windows + per_group - 1) / per_group;
  if (blocks > kDivGroups) blocks = kDivGroups;
  if (blocks < 1) blocks = 1;  // workgroup 0 clears the totals
  hipLaunchKernelGGL(divergence_windows, dim3((unsigned)blocks), dim3(kDivBlock), 0, stream,
                     tex_id, (uint32_t)n, tex_to_dec, (uint32_t)n_textures, (uint32_t)n_decoders,
                     order, (uint64_t)len, (uint32_t)wave, n_windows, per_wave, totals);
  launch_reduce(per_wave, n_windows, nullptr, 0, totals, stream);
  return hip_status(hipGetLastError());
}

}  // namespace ntc
