// ntc_bins.hip -- stable counting sort of texel queries by decoder id.
//
// Groups the query stream so that every 64-slot tile of `perm` belongs to one
// decoder; a wave then evaluates a single decoder, the situation the paper's
// shared decoder creates (Sec. 1; Sec. 4.4 "Performance analysis").  The
// binning itself is not in the paper.
//
// Three kernels:
//   hist    : workgroup b resolves the decoder id of every query of its chunk
//             (tex_to_dec[tex_id[q]]), stores it as a 16-bit id for the scatter,
//             and counts the ids into an LDS histogram written as column b of
//             hist[d][b]; row D counts the chunk's invalid queries.
//   scan    : workgroup d turns row d into an exclusive prefix over chunks and
//             writes bin_count[d]; the last workgroup to finish (found with a
//             device-scope counter) scans the counts into the padded
//             bin_offset and fills the padding slots with NTC_PAD.
//   scatter : workgroup b walks its chunk again in order, reading the 16-bit
//             ids, and writes each query to bin_offset[d] + hist[d][b] + (rank
//             of the query inside the chunk among queries of decoder d).
// Ranks inside a wave come from ballots over the distinct ids present (a peel
// loop whose trip count is the number of distinct decoders in the wave), so the
// order inside a bin is ascending query index: the permutation is unique.
// Each thread issues a whole batch of loads before it consumes any of them.
#include "ntc_internal.h"

namespace ntc {
namespace {

constexpr int kBatch = 16;                         // ids per thread per histogram batch
constexpr int kRows = 8;                           // 64-query rows per wave per scatter tile
constexpr int kTile = kBlock * kRows;              // queries per scatter step of a workgroup
constexpr int64_t kChunkQuantum = kBlock * kBatch; // chunks are multiples of this (and of kTile)
constexpr int64_t kMinChunk = 2 * kChunkQuantum;   // queries per workgroup, at least
constexpr int64_t kTargetBlocks = 1024;
constexpr uint16_t kInvalid16 = 0xFFFF;            // 16-bit id of an invalid query
constexpr int kScanPerThread = 8;                  // chunks per thread in the row scan

// The workspace starts with kStatusWords status words -- [0] scan completion
// counter, [1] invalid query count -- followed by the chunk histograms and then
// the 16-bit decoder id of every query.
constexpr int kStatusWords = 4;

__global__ void __launch_bounds__(kBlock)
bins_hist(const uint32_t *__restrict__ tex_id, uint32_t n,
          const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures, uint32_t n_decoders,
          uint32_t chunk, uint32_t nblocks, uint32_t *__restrict__ hist,
          uint32_t *__restrict__ status, uint16_t *__restrict__ dec16) {
  extern __shared__ uint32_t lds_hist[];  // n_decoders + 1 counters
  const uint32_t b = blockIdx.x;
  for (uint32_t d = threadIdx.x; d <= n_decoders; d += kBlock) lds_hist[d] = 0;
  if (b == 0 && threadIdx.x == 0) status[0] = 0;  // scan completion counter
  __syncthreads();
  const uint64_t begin = (uint64_t)b * chunk;
  const uint64_t end = begin + chunk < n ? begin + chunk : n;
  for (uint64_t base = begin; base < end; base += kChunkQuantum) {
    // row j of the batch: queries base + j * kBlock + thread
    uint32_t t[kBatch], d[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const uint64_t i = base + (uint64_t)j * kBlock + threadIdx.x;
      t[j] = i < end ? tex_id[i] : 0xFFFFFFFFu;
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const uint32_t dd = t[j] < n_textures ? tex_to_dec[t[j]] : n_decoders;
      d[j] = dd < n_decoders ? dd : n_decoders;  // n_decoders marks an invalid query
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const uint64_t i = base + (uint64_t)j * kBlock + threadIdx.x;
      const bool inside = i < end;
      if (inside) dec16[i] = d[j] < n_decoders ? (uint16_t)d[j] : kInvalid16;
      uint64_t todo = ballot(inside);
      while (todo) {
        const uint32_t leader = (uint32_t)__builtin_ctzll(todo);
        const uint32_t dl = read_lane(d[j], leader);
        const uint64_t same = ballot(d[j] == dl) & todo;
        if (lane_id() == leader) atomicAdd(&lds_hist[dl], (uint32_t)__builtin_popcountll(same));
        todo &= ~same;
      }
    }
  }
  __syncthreads();
  for (uint32_t d = threadIdx.x; d <= n_decoders; d += kBlock)
    hist[(size_t)d * nblocks + b] = lds_hist[d];
}

// Exclusive scan of the kBlock values held one per thread; returns the total.
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t &excl, uint32_t *lds_tmp) {
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  uint32_t incl = v;
#pragma unroll
  for (int s = 1; s < kWave; s <<= 1) {
    uint32_t o = __shfl_up(incl, s, kWave);
    if (lane >= (uint32_t)s) incl += o;
  }
  if (lane == kWave - 1) lds_tmp[w] = incl;
  __syncthreads();
  uint32_t base = 0, total = 0;
  for (int k = 0; k < kWavesPerBlock; ++k) {
    uint32_t t = lds_tmp[k];
    if (k < (int)w) base += t;
    total += t;
  }
  __syncthreads();
  excl = base + incl - v;
  return total;
}

__global__ void __launch_bounds__(kBlock)
bins_scan(uint32_t *__restrict__ hist, uint32_t nblocks, uint32_t n_decoders, uint32_t align,
          uint32_t *__restrict__ bin_count, uint32_t *__restrict__ bin_offset,
          uint32_t *__restrict__ perm, uint32_t *__restrict__ status) {
  __shared__ uint32_t lds_tmp[kWavesPerBlock];
  __shared__ uint32_t lds_last;
  const uint32_t d = blockIdx.x;  // row; row n_decoders counts invalid queries
  uint32_t *row = hist + (size_t)d * nblocks;
  // each thread owns kScanPerThread consecutive chunks of the row (nblocks is
  // at most kBlock * kScanPerThread); all of them are loaded at once
  const uint32_t lo = threadIdx.x * kScanPerThread;
  uint32_t v[kScanPerThread];
  uint32_t sum = 0;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    v[k] = lo + k < nblocks ? row[lo + k] : 0u;
    sum += v[k];
  }
  uint32_t excl;
  const uint32_t total = block_exclusive_scan(sum, excl, lds_tmp);
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (lo + k < nblocks) row[lo + k] = excl;
    excl += v[k];
  }
  if (threadIdx.x == 0) {
    if (d < n_decoders) bin_count[d] = total;
    else status[1] = total;
  }
  // The last row to finish turns the counts into padded offsets.
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) lds_last = atomicAdd(&status[0], 1u) == n_decoders;
  __syncthreads();
  if (!lds_last) return;
  __threadfence();
  const uint32_t dper = (n_decoders + kBlock - 1) / kBlock;
  const uint32_t dlo = threadIdx.x * dper;
  const uint32_t dhi = dlo + dper < n_decoders ? dlo + dper : n_decoders;
  uint32_t psum = 0;
  for (uint32_t k = dlo; k < dhi; ++k) {
    uint32_t c = __hip_atomic_load(&bin_count[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    psum += (c + align - 1) & ~(align - 1);
  }
  uint32_t pexcl;
  const uint32_t ptotal = block_exclusive_scan(psum, pexcl, lds_tmp);
  for (uint32_t k = dlo; k < dhi; ++k) {
    uint32_t c = __hip_atomic_load(&bin_count[k], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bin_offset[k] = pexcl;
    const uint32_t padded = (c + align - 1) & ~(align - 1);
    for (uint32_t s = pexcl + c; s < pexcl + padded; ++s) perm[s] = NTC_PAD;
    pexcl += padded;
  }
  if (threadIdx.x == kBlock - 1) bin_offset[n_decoders] = ptotal;
}

__global__ void __launch_bounds__(kBlock)
bins_scatter(const uint16_t *__restrict__ dec16, uint32_t n, uint32_t n_decoders,
             uint32_t chunk, uint32_t nblocks, const uint32_t *__restrict__ hist,
             const uint32_t *__restrict__ bin_offset, uint32_t *__restrict__ perm) {
  // cursor[d]: next free slot of bin d for this chunk;
  // wave_cnt[w][d]: queries of decoder d in wave w's part of the current tile.
  extern __shared__ uint32_t lds[];
  uint32_t *cursor = lds;
  uint32_t *wave_cnt = lds + n_decoders;
  const uint32_t b = blockIdx.x;
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  for (uint32_t d = threadIdx.x; d < n_decoders; d += kBlock) {
    cursor[d] = bin_offset[d] + hist[(size_t)d * nblocks + b];
#pragma unroll
    for (int k = 0; k < kWavesPerBlock; ++k) wave_cnt[k * n_decoders + d] = 0;
  }
  __syncthreads();
  uint32_t *my_cnt = wave_cnt + w * n_decoders;
  const uint64_t begin = (uint64_t)b * chunk;
  const uint64_t end = begin + chunk < n ? begin + chunk : n;
  // wave w owns queries [tile + w*64*kRows, +64*kRows) of a tile; row r lane l
  // holds query tile + w*64*kRows + r*64 + l.  The next tile's ids are fetched
  // while the current one is ranked and scattered.
  auto fetch = [&](uint64_t tile, uint32_t (&dec)[kRows]) {
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const uint64_t q = tile + (uint64_t)w * kWave * kRows + r * kWave + lane;
      const uint16_t v = q < end ? dec16[q] : kInvalid16;
      dec[r] = v == kInvalid16 ? n_decoders : (uint32_t)v;
    }
  };
  uint32_t nxt[kRows];
  if (begin < end) fetch(begin, nxt);
  for (uint64_t tile = begin; tile < end; tile += kTile) {
    uint32_t dec[kRows], rank[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) dec[r] = nxt[r];
    if (tile + kTile < end) fetch(tile + kTile, nxt);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      uint64_t todo = ballot(dec[r] < n_decoders);
      rank[r] = 0;
      while (todo) {
        const uint32_t leader = (uint32_t)__builtin_ctzll(todo);
        const uint32_t dl = read_lane(dec[r], leader);
        const uint64_t same = ballot(dec[r] == dl) & todo;
        const uint32_t before = my_cnt[dl];  // same address in every lane
        if (dec[r] == dl) rank[r] = before + lanes_below(same);
        if (lane == leader) my_cnt[dl] = before + (uint32_t)__builtin_popcountll(same);
        todo &= ~same;
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const uint32_t d = dec[r];
      if (d < n_decoders) {
        uint32_t pos = cursor[d] + rank[r];
        for (uint32_t k = 0; k < w; ++k) pos += wave_cnt[k * n_decoders + d];
        perm[pos] = (uint32_t)(tile + (uint64_t)w * kWave * kRows + r * kWave + lane);
      }
    }
    __syncthreads();
    // The last query of each decoder in this wave's part hands the count on to
    // the cursor and clears the wave's counter (all lanes read before any write).
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const uint32_t d = dec[r];
      const uint32_t cnt = d < n_decoders ? my_cnt[d] : 0u;
      const bool last = d < n_decoders && rank[r] + 1 == cnt;
      if (last) {
        atomicAdd(&cursor[d], cnt);
        my_cnt[d] = 0;
      }
    }
  }
}

}  // namespace

BinsLayout bins_layout(int64_t n, int32_t n_decoders) {
  BinsLayout L;
  int64_t chunk = (n + kTargetBlocks - 1) / kTargetBlocks;
  chunk = (chunk + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum;
  if (chunk < kMinChunk) chunk = kMinChunk;
  L.chunk = chunk;
  L.blocks = n > 0 ? (n + chunk - 1) / chunk : 1;
  L.hist_words = (size_t)(n_decoders + 1) * (size_t)L.blocks;
  const size_t dec_words = ((size_t)n + 1) / 2;  // 16-bit ids, two per word
  L.bytes = (kStatusWords + L.hist_words + dec_words) * sizeof(uint32_t);
  return L;
}

static_assert(kChunkQuantum % kTile == 0, "scatter tiles must divide the chunks");
static_assert(kTargetBlocks + 1 <= (int64_t)kBlock * kScanPerThread,
              "the row scan covers every chunk");

int launch_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, int32_t align,
                      uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                      void *workspace, hipStream_t stream) {
  const BinsLayout L = bins_layout(n, n_decoders);
  uint32_t *status = (uint32_t *)workspace;
  uint32_t *hist = status + kStatusWords;
  uint16_t *dec16 = (uint16_t *)(hist + L.hist_words);
  const uint32_t D = (uint32_t)n_decoders;
  const size_t lds_hist = (size_t)(D + 1) * sizeof(uint32_t);
  const size_t lds_scatter = (size_t)D * (1 + kWavesPerBlock) * sizeof(uint32_t);
  if (lds_scatter > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void *)bins_scatter,
                                       hipFuncAttributeMaxDynamicSharedMemorySize,
                                       (int)lds_scatter);
    if (e != hipSuccess) return NTC_ERR_HIP;
  }
  hipLaunchKernelGGL(bins_hist, dim3((unsigned)L.blocks), dim3(kBlock), lds_hist, stream, tex_id,
                     (uint32_t)n, tex_to_dec, (uint32_t)n_textures, D, (uint32_t)L.chunk,
                     (uint32_t)L.blocks, hist, status, dec16);
  hipLaunchKernelGGL(bins_scan, dim3(D + 1), dim3(kBlock), 0, stream, hist, (uint32_t)L.blocks, D,
                     (uint32_t)align, bin_count, bin_offset, perm, status);
  if (n > 0)
    hipLaunchKernelGGL(bins_scatter, dim3((unsigned)L.blocks), dim3(kBlock), lds_scatter, stream,
                       dec16, (uint32_t)n, D, (uint32_t)L.chunk, (uint32_t)L.blocks, hist,
                       bin_offset, perm);
  return hip_status(hipGetLastError());
}

size_t bins_status_bytes() { return kStatusWords * sizeof(uint32_t); }

int read_invalid_count(const void *workspace, uint64_t *n_invalid, hipStream_t stream) {
  const uint32_t *status = (const uint32_t *)workspace;
  uint32_t v = 0;
  hipError_t e = hipMemcpyAsync(&v, status + 1, sizeof(v), hipMemcpyDeviceToHost, stream);
  if (e == hipSuccess) e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return NTC_ERR_HIP;
  if (n_invalid) *n_invalid = v;
  return v ? NTC_ERR_INDEX : NTC_OK;
}

}  // namespace ntc
