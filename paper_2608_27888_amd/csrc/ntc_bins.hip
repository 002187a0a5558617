// ntc_bins.hip -- stable counting sort of texel queries by decoder id.
//
// Groups the query stream so that every 64-slot tile of `perm` belongs to one
// decoder; a wave then evaluates a single decoder, the situation the paper's
// shared decoder creates (Sec. 1; Sec. 4.4 "Performance analysis").  The
// binning itself is not in the paper.
//
// The unit of the sort is one wave's contiguous slice of the query stream
// (slice g = workgroup * 4 + wave).  Three kernels:
//   hist    : every wave resolves the decoder id of each query of its slice
//             (tex_to_dec[tex_id[q]]), stores it as a 16-bit id for the
//             scatter, and counts the ids in a wave-private LDS histogram that
//             becomes column g of hist[d][g]; row D counts invalid queries.
//   scan    : workgroup d turns row d into an exclusive prefix over slices and
//             writes bin_count[d] (row D: the invalid count).
//   scatter : every workgroup first scans bin_count into the padded bin
//             offsets (workgroup 0 writes bin_offset, the padding slots are
//             shared out among the workgroups); then each wave walks its slice
//             in order with wave-private cursors bin_offset[d] + hist[d][g] and
//             writes every query to the next slot of its bin.
// Inside a 64-query row the lanes that share a decoder id are ranked with a
// ballot and a lane count, so the order inside a bin is ascending query index
// and the permutation is unique.  A row whose queries all share the decoder of
// the previous such row (the common case for screen-coherent material maps)
// touches no LDS: the wave keeps that decoder's count or cursor in a register.
// Each lane issues a whole batch of loads (and the batch's map lookups) before
// it consumes any of them, and fetches the next batch while it counts this one.
#include "ntc_internal.h"

namespace ntc {
namespace {

constexpr int kRowsPerBatch = 8;                                  // rows a wave loads at once
constexpr int64_t kWaveQuantum = (int64_t)kWave * kRowsPerBatch;  // queries per wave batch
constexpr int64_t kChunkQuantum = kWaveQuantum * kWavesPerBlock;  // chunks are multiples of this
constexpr int64_t kMinChunk = 2 * kChunkQuantum;                  // queries per workgroup, at least
constexpr int64_t kTargetBlocks = 1024;
constexpr uint16_t kInvalid16 = 0xFFFF;                           // 16-bit id of an invalid query
constexpr uint32_t kOutside = 0xFFFFFFFFu;                        // marks a lane past the slice
constexpr int kScanPerThread = 16;                                // slices per thread in the row scan

// The workspace starts with kStatusWords status words -- [1] is the invalid
// query count -- followed by the slice histograms and, from a 16-byte aligned
// offset, the 16-bit decoder id of every query.
constexpr int kStatusWords = 4;

// Decoder id of texture t: n_decoders marks an invalid query.
__device__ __forceinline__ uint32_t decoder_of(uint32_t t, const uint32_t *tex_to_dec,
                                               uint32_t n_textures, uint32_t n_decoders) {
  const uint32_t d = t < n_textures ? tex_to_dec[t] : n_decoders;
  return d < n_decoders ? d : n_decoders;
}

// Query range [beg, end) of wave w of workgroup b.
struct Slice {
  uint64_t beg, end;
};

__device__ __forceinline__ Slice slice_of(uint32_t b, uint32_t w, uint64_t chunk, uint64_t n) {
  const uint64_t cbeg = (uint64_t)b * chunk;
  const uint64_t cend = cbeg + chunk < n ? cbeg + chunk : n;
  const uint64_t wchunk = chunk / kWavesPerBlock;
  const uint64_t beg = cbeg + w * wchunk < cend ? cbeg + w * wchunk : cend;
  return Slice{beg, beg + wchunk < cend ? beg + wchunk : cend};
}

__global__ void __launch_bounds__(kBlock)
bins_hist(const uint32_t *__restrict__ tex_id, uint32_t n,
          const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures, uint32_t n_decoders,
          uint32_t chunk, uint32_t n_slices, uint32_t *__restrict__ hist,
          uint16_t *__restrict__ dec16) {
  extern __shared__ uint32_t lds[];  // kWavesPerBlock x (n_decoders + 1) counters
  const uint32_t b = blockIdx.x, w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t rows = n_decoders + 1;
  const Slice sl = slice_of(b, w, chunk, n);
  // A run of whole rows with one decoder is counted in (run_d, run_n) and
  // added to the histogram when it ends.
  uint32_t run_d = kOutside, run_n = 0;
  // Lanes past the slice load its first id (an unconditional load keeps the
  // compiler's wait counts exact); the row loop masks them out.
  auto fetch = [&](uint64_t base, uint32_t (&v)[kRowsPerBatch]) {
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) {
      const uint64_t q = base + (uint64_t)j * kWave + lane;
      v[j] = tex_id[q < sl.end ? q : sl.beg];
    }
  };
  // the first batch is in flight while the histogram is cleared
  uint32_t nxt[kRowsPerBatch];
  if (sl.beg < sl.end) fetch(sl.beg, nxt);
  for (uint32_t i = threadIdx.x; i < kWavesPerBlock * rows; i += kBlock) lds[i] = 0;
  __syncthreads();
  uint32_t *h = lds + w * rows;
  for (uint64_t base = sl.beg; base < sl.end; base += kWaveQuantum) {
    uint32_t t[kRowsPerBatch];
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) t[j] = nxt[j];
    // Every row's map lookup is issued before any of them is used: the loads
    // are unconditional (texture 0 stands in for an out-of-range id or a lane
    // past the slice), so they are not serialised behind per-row branches.
    // They go out before the next batch's ids, so that waiting for them does
    // not wait for that prefetch (loads complete in issue order for the
    // wait counter).
    uint32_t m[kRowsPerBatch];
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) m[j] = tex_to_dec[t[j] < n_textures ? t[j] : 0u];
    __builtin_amdgcn_sched_barrier(0);
    if (base + kWaveQuantum < sl.end) fetch(base + kWaveQuantum, nxt);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) {
      const uint64_t q = base + (uint64_t)j * kWave + lane;
      const bool inside = q < sl.end;
      const uint32_t d = !inside ? kOutside
                         : (t[j] < n_textures && m[j] < n_decoders) ? m[j] : n_decoders;
      if (inside) dec16[q] = d < n_decoders ? (uint16_t)d : kInvalid16;
      const uint32_t v0 = __builtin_amdgcn_readfirstlane(d);
      if (ballot(d == v0) == ~0ull) {
        if (v0 != kOutside) {
          if (v0 != run_d) {
            if (run_n && lane == 0) atomicAdd(&h[run_d], run_n);
            run_d = v0;
            run_n = 0;
          }
          run_n += kWave;
        }
      } else {
        uint64_t todo = ballot(inside);
        while (todo) {
          const uint32_t leader = (uint32_t)__builtin_ctzll(todo);
          const uint32_t dl = read_lane(d, leader);
          const uint64_t same = ballot(d == dl) & todo;
          if (lane == leader) atomicAdd(&h[dl], (uint32_t)__builtin_popcountll(same));
          todo &= ~same;
        }
      }
    }
  }
  if (run_n && lane == 0) atomicAdd(&h[run_d], run_n);
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < kWavesPerBlock * rows; i += kBlock) {
    const uint32_t ww = i / rows, d = i % rows;
    hist[(size_t)d * n_slices + b * kWavesPerBlock + ww] = lds[i];
  }
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
bins_scan(uint32_t *__restrict__ hist, uint32_t n_slices, uint32_t n_decoders,
          uint32_t *__restrict__ bin_count, uint32_t *__restrict__ status,
          uint32_t *__restrict__ invalid_out) {
  __shared__ uint32_t lds_tmp[kWavesPerBlock];
  const uint32_t d = blockIdx.x;  // row; row n_decoders counts invalid queries
  uint32_t *row = hist + (size_t)d * n_slices;
  // each thread owns kScanPerThread consecutive slices of the row (n_slices is
  // at most kBlock * kScanPerThread); all of them are loaded at once
  const uint32_t lo = threadIdx.x * kScanPerThread;
  uint32_t v[kScanPerThread];
  uint32_t sum = 0;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    v[k] = lo + k < n_slices ? row[lo + k] : 0u;
    sum += v[k];
  }
  uint32_t excl;
  const uint32_t total = block_exclusive_scan(sum, excl, lds_tmp);
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (lo + k < n_slices) row[lo + k] = excl;
    excl += v[k];
  }
  if (threadIdx.x == 0) {
    if (d < n_decoders) {
      bin_count[d] = total;
    } else {
      status[1] = total;
      if (invalid_out) *invalid_out = total;
    }
  }
}

__global__ void __launch_bounds__(kBlock)
bins_scatter(const uint16_t *__restrict__ dec16, uint32_t n, uint32_t n_decoders,
             uint32_t align, uint32_t chunk, uint32_t n_slices,
             const uint32_t *__restrict__ hist, const uint32_t *__restrict__ bin_count,
             uint32_t *__restrict__ bin_offset, uint32_t *__restrict__ perm) {
  extern __shared__ uint32_t lds[];  // kWavesPerBlock x n_decoders cursors
  __shared__ uint32_t lds_tmp[kWavesPerBlock];
  const uint32_t b = blockIdx.x, w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t nblocks = gridDim.x;
  const Slice sl = slice_of(b, w, chunk, n);
  // Lanes past the slice read as invalid.  The first batch is in flight
  // during the offset scan below.
  auto fetch = [&](uint64_t base, uint32_t (&v)[kRowsPerBatch]) {
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) {
      const uint64_t q = base + (uint64_t)j * kWave + lane;
      v[j] = q < sl.end ? dec16[q] : kInvalid16;
    }
  };
  uint32_t nxt[kRowsPerBatch];
  if (sl.beg < sl.end) fetch(sl.beg, nxt);
  // Padded bin offsets: thread i owns decoders [dlo, dhi).
  const uint32_t dper = (n_decoders + kBlock - 1) / kBlock;
  const uint32_t dlo = min(threadIdx.x * dper, n_decoders);
  const uint32_t dhi = min(dlo + dper, n_decoders);
  uint32_t psum = 0;
  for (uint32_t k = dlo; k < dhi; ++k) psum += (bin_count[k] + align - 1) & ~(align - 1);
  uint32_t off;
  const uint32_t total = block_exclusive_scan(psum, off, lds_tmp);
  for (uint32_t k = dlo; k < dhi; ++k) {
    const uint32_t c = bin_count[k];
    const uint32_t padded = (c + align - 1) & ~(align - 1);
#pragma unroll
    for (int i = 0; i < kWavesPerBlock; ++i)
      lds[i * n_decoders + k] = off + hist[(size_t)k * n_slices + b * kWavesPerBlock + i];
    if (b == 0) bin_offset[k] = off;
    if (k % nblocks == b)  // the padding slots of bin k
      for (uint32_t s = off + c; s < off + padded; ++s) perm[s] = NTC_PAD;
    off += padded;
  }
  if (b == 0 && threadIdx.x == 0) bin_offset[n_decoders] = total;
  __syncthreads();
  uint32_t *cur = lds + w * n_decoders;
  // (cd, cc): a decoder whose cursor lives in a register while whole rows of
  // it follow one another; cur[cd] is stale meanwhile.
  uint32_t cd = kOutside, cc = 0;
  for (uint64_t base = sl.beg; base < sl.end; base += kWaveQuantum) {
    uint32_t v[kRowsPerBatch];
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) v[j] = nxt[j];
    if (base + kWaveQuantum < sl.end) fetch(base + kWaveQuantum, nxt);
#pragma unroll
    for (int j = 0; j < kRowsPerBatch; ++j) {
      const uint32_t q = (uint32_t)(base + (uint64_t)j * kWave + lane);
      const uint32_t d = v[j] == kInvalid16 ? n_decoders : v[j];  // lanes past the end: invalid
      const uint32_t v0 = __builtin_amdgcn_readfirstlane(d);
      if (ballot(d == v0) == ~0ull && v0 < n_decoders) {
        if (v0 != cd) {
          if (cd != kOutside && lane == 0) cur[cd] = cc;
          cd = v0;
          cc = cur[v0];
        }
        perm[cc + lane] = q;
        cc += kWave;
      } else {
        if (cd != kOutside) {
          if (lane == 0) cur[cd] = cc;
          cd = kOutside;
        }
        uint64_t todo = ballot(d < n_decoders);
        while (todo) {
          const uint32_t leader = (uint32_t)__builtin_ctzll(todo);
          const uint32_t dl = read_lane(d, leader);
          const uint64_t same = ballot(d == dl) & todo;
          const uint32_t at = cur[dl];  // same address in every lane
          if (d == dl) perm[at + lanes_below(same)] = q;
          if (lane == leader) cur[dl] = at + (uint32_t)__builtin_popcountll(same);
          todo &= ~same;
        }
      }
    }
  }
}

// Lets a kernel use more than the default 64 KB of dynamic LDS.
int allow_lds(const void *kernel, size_t bytes) {
  if (bytes + 64 <= 64 * 1024) return NTC_OK;
  return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) ==
                 hipSuccess
             ? NTC_OK
             : NTC_ERR_HIP;
}

}  // namespace

BinsLayout bins_layout(int64_t n, int32_t n_decoders) {
  BinsLayout L;
  int64_t chunk = (n + kTargetBlocks - 1) / kTargetBlocks;
  chunk = (chunk + kChunkQuantum - 1) / kChunkQuantum * kChunkQuantum;
  if (chunk < kMinChunk) chunk = kMinChunk;
  L.chunk = chunk;
  L.blocks = n > 0 ? (n + chunk - 1) / chunk : 1;
  L.hist_words = (size_t)(n_decoders + 1) * (size_t)L.blocks * kWavesPerBlock;
  L.dec_offset = ((kStatusWords + L.hist_words) * sizeof(uint32_t) + 15) & ~(size_t)15;
  L.bytes = L.dec_offset + (((size_t)n * sizeof(uint16_t) + 15) & ~(size_t)15);
  return L;
}

static_assert(kTargetBlocks * kWavesPerBlock <= (int64_t)kBlock * kScanPerThread,
              "the row scan covers every slice");

int launch_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, int32_t align,
                      uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                      void *workspace, uint32_t *invalid_out, hipStream_t stream) {
  const BinsLayout L = bins_layout(n, n_decoders);
  uint32_t *status = (uint32_t *)workspace;
  uint32_t *hist = status + kStatusWords;
  uint16_t *dec16 = (uint16_t *)((char *)workspace + L.dec_offset);
  const uint32_t D = (uint32_t)n_decoders;
  const uint32_t n_slices = (uint32_t)L.blocks * kWavesPerBlock;
  const size_t lds_hist = (size_t)kWavesPerBlock * (D + 1) * sizeof(uint32_t);
  const size_t lds_scatter = (size_t)kWavesPerBlock * D * sizeof(uint32_t);
  int st = allow_lds((const void *)bins_hist, lds_hist);
  if (st == NTC_OK) st = allow_lds((const void *)bins_scatter, lds_scatter);
  if (st != NTC_OK) return st;
  hipLaunchKernelGGL(bins_hist, dim3((unsigned)L.blocks), dim3(kBlock), lds_hist, stream, tex_id,
                     (uint32_t)n, tex_to_dec, (uint32_t)n_textures, D, (uint32_t)L.chunk, n_slices,
                     hist, dec16);
  hipLaunchKernelGGL(bins_scan, dim3(D + 1), dim3(kBlock), 0, stream, hist, n_slices, D,
                     bin_count, status, invalid_out);
  hipLaunchKernelGGL(bins_scatter, dim3((unsigned)L.blocks), dim3(kBlock), lds_scatter, stream,
                     dec16, (uint32_t)n, D, (uint32_t)align, (uint32_t)L.chunk, n_slices, hist,
                     bin_count, bin_offset, perm);
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
