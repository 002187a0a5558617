// ntc_bins.hip -- stable counting sort of texel queries by decoder id.
//
// Groups the query stream so that every 64-slot tile of `perm` belongs to one
// decoder; a wave then evaluates a single decoder, the situation the paper's
// shared decoder creates (Sec. 1; Sec. 4.4 "Performance analysis").  The
// binning itself is not in the paper.
//
// The unit of the sort is one wave's contiguous slice of the query stream
// (slice g = workgroup * waves + wave), processed in batches of kBatchRows rows
// of 64 queries.
//
// Up to 64 decoders (while every workgroup can sum the rows of tot in two
// rounds of loads), two kernels on workgroups of 4 to 16 waves:
//   count : every wave resolves the decoder id of each query of its slice
//           (tex_to_dec[tex_id[q]]) and counts the ids; the workgroup writes its
//           sums over its waves, column b of tot[d][b] (row D: invalid
//           queries), and for slice g its waves' exclusive prefix, hist[d][g].
//   place : every workgroup sums the rows of tot (at most 512 words each): the
//           totals give the padded bin offsets (workgroup 0 writes bin_count
//           and bin_offset, the padding slots are shared out among the
//           workgroups), the columns before its own its offset inside every
//           bin, and hist[d][g] each wave's offset after that.  Each wave then
//           resolves the ids of its slice again and writes every query to the
//           next slot of its bin.
// Otherwise three kernels on workgroups of 4 waves: count writes hist only;
// scan (workgroup d) turns row d of hist into its exclusive prefix over slices
// and writes bin_count[d]; place scans bin_count into the padded offsets and
// starts its cursors at bin_offset[d] + hist[d][g].
// Inside a 64-query row the lanes that share a decoder id are ranked with a
// ballot and a lane count, one pass per distinct id of the row, so the order
// inside a bin is ascending query index and the permutation is unique.  With at
// most 64 decoders the wave's counters (count) and cursors (place) live in one
// register, lane k holding decoder k's, and a row costs no LDS access; with more
// they live in a wave-private LDS table.  A wave issues the id loads of a whole
// batch, then all of its map lookups, before it uses any of them.  The decoder
// ids are not stored between the passes: reading tex_id twice moves as many
// bytes as writing and reading back 16-bit ids, and leaves the count pass
// without stores.  Workgroups are numbered XCD by XCD, so the histogram
// entries of neighbouring slices are written from one L2.
#include "ntc_internal.h"

namespace ntc {
namespace {

constexpr int kBatchRows = 16;                                   // rows of 64 per wave batch
constexpr int64_t kWaveQuantum = (int64_t)kWave * kBatchRows;    // queries per wave batch
constexpr int64_t kTargetBlocks = 2048;                          // workgroups, at most
// The two-kernel path: workgroups of 4, 8 or 16 waves, at most kSumBlocks of
// them, so that every place workgroup can sum the tot rows.  The widest
// workgroups that still give every CU one (kCus) keep many waves in flight on a
// large frame; a smaller frame takes narrower ones, since the per-row ranking
// runs on the CU's one scalar unit and a CU without a workgroup sits idle.
constexpr int64_t kSumBlocks = 512;
constexpr int64_t kCus = 256;
constexpr int kSumLanes = 32;  // place: lanes per row of tot
constexpr int kSumPer = 16;    // place: words of a row per lane
constexpr int kSumRounds = 2;  // place: at most this many rounds of those loads
constexpr int64_t kMaxHistWords = (int64_t)1 << 20;              // slice histograms, at most
constexpr uint32_t kOutside = 0xFFFFFFFFu;                       // a lane past the slice
constexpr int kScanThreads = 1024;                               // scan: threads per column
constexpr int kScanPerThread = 8;                                // scan: slices per thread
constexpr uint32_t kRegDecoders = kWave;                         // register tables up to here

static_assert(kTargetBlocks * kWavesPerBlock <= (int64_t)kScanThreads * kScanPerThread,
              "one scan pass covers every slice");

// The workspace starts with kStatusWords status words -- [1] is the invalid
// query count -- followed by hist[n_decoders + 1][slices] and, on the
// two-kernel path, tot[n_decoders + 1][workgroups].
constexpr int kStatusWords = 4;

// Query range [beg, end) of wave w of a workgroup b of WAVES waves.
struct Slice {
  uint64_t beg, end;
};

template <int WAVES>
__device__ __forceinline__ Slice slice_of(uint32_t b, uint32_t w, uint64_t chunk, uint64_t n) {
  const uint64_t cbeg = (uint64_t)b * chunk;
  const uint64_t cend = cbeg + chunk < n ? cbeg + chunk : n;
  const uint64_t wchunk = chunk / WAVES;
  const uint64_t beg = cbeg + w * wchunk < cend ? cbeg + w * wchunk : cend;
  return Slice{beg, beg + wchunk < cend ? beg + wchunk : cend};
}

// Decoder ids of the batch of kBatchRows rows starting at query `base` (wave
// uniform, base < end): lanes at or past `end` get kOutside, invalid queries
// `invalid`.  Every id load is issued, then every map lookup, before any result
// is used; the loads are unconditional (clamped into the slice), addressed from
// one wave-uniform pointer with 32-bit lane offsets.
__device__ __forceinline__ void load_batch(const uint32_t *__restrict__ tex_id,
                                           const uint32_t *__restrict__ tex_to_dec,
                                           uint32_t n_textures, uint32_t n_decoders,
                                           uint32_t invalid, uint64_t base, uint64_t end,
                                           uint32_t lane, uint32_t (&d)[kBatchRows]) {
  const uint32_t *row = tex_id + base;
  const uint64_t left = end - base;
  const uint32_t lim = left < (uint64_t)kWaveQuantum ? (uint32_t)left : (uint32_t)kWaveQuantum;
#pragma unroll
  for (int j = 0; j < kBatchRows; ++j) {
    const uint32_t o = (uint32_t)j * kWave + lane;
    d[j] = row[o < lim - 1 ? o : lim - 1];
  }
  uint32_t m[kBatchRows];
#pragma unroll
  for (int j = 0; j < kBatchRows; ++j) m[j] = tex_to_dec[d[j] < n_textures ? d[j] : 0u];
#pragma unroll
  for (int j = 0; j < kBatchRows; ++j) {
    const uint32_t o = (uint32_t)j * kWave + lane;
    d[j] = o >= lim ? kOutside : d[j] < n_textures && m[j] < n_decoders ? m[j] : invalid;
  }
}

// Table of one value per decoder: lane k of a register (REG) or word k of a
// wave-private LDS array.
template <bool REG>
struct WaveTable {
  uint32_t reg;
  uint32_t *lds;
  // value of decoder dl (wave uniform)
  __device__ __forceinline__ uint32_t get(uint32_t dl) const {
    if constexpr (REG) return __builtin_amdgcn_readlane(reg, dl);
    else return lds[dl];
  }
  // adds c to decoder dl's value (called by every lane; `leader` is one lane):
  // a no-return LDS atomic does not wait for the old value
  __device__ __forceinline__ void add(uint32_t dl, uint32_t c, uint32_t lane, bool leader) {
    if constexpr (REG) reg += lane == dl ? c : 0u;
    else if (leader) atomicAdd(&lds[dl], c);
  }
};

// Ranks the valid lanes of one row (d != kOutside) by decoder: each lane gets
// the table value of its decoder plus the number of lanes below it with the same
// decoder, and the table advances by the row's count of each decoder.
template <bool REG, bool RANK>
__device__ __forceinline__ uint32_t rank_row(uint32_t d, WaveTable<REG> &t, uint32_t lane) {
  uint64_t todo = ballot(d != kOutside);
  uint32_t pos = 0;
  while (todo) {
    const uint32_t leader = (uint32_t)__builtin_ctzll(todo);
    const uint32_t dl = read_lane(d, leader);
    const uint64_t same = ballot(d == dl) & todo;
    const uint32_t c = (uint32_t)__builtin_popcountll(same);
    if constexpr (RANK && !REG) {
      // LDS table: the leader's returning atomic reads and advances the cursor
      uint32_t old = 0;
      if (lane == leader) old = atomicAdd(&t.lds[dl], c);
      pos = d == dl ? read_lane(old, leader) + lanes_below(same) : pos;
    } else {
      if constexpr (RANK) {
        const uint32_t at = t.get(dl);
        pos = d == dl ? at + lanes_below(same) : pos;
      }
      t.add(dl, c, lane, lane == leader);
    }
    todo &= ~same;
  }
  return pos;
}

// REG: register tables (n_decoders <= 64).  tot (REG only): the workgroup's
// sums over its waves, column b of tot[n_decoders + 1][gridDim.x], with hist
// holding each wave's exclusive prefix over the workgroup's waves; NULL: hist
// holds each wave's own counts.
template <bool REG, int WAVES>
__global__ void __launch_bounds__(WAVES * kWave)
bins_count(const uint32_t *__restrict__ tex_id, uint32_t n,
           const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures, uint32_t n_decoders,
           uint32_t chunk, uint32_t *__restrict__ hist, uint32_t *__restrict__ tot) {
  extern __shared__ uint32_t lds[];  // !REG: WAVES x (n_decoders + 1) counters
  __shared__ uint32_t part[REG ? WAVES : 1][kWave + 1];
  const uint32_t b = xcd_local_block(blockIdx.x, gridDim.x), lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint32_t cols = n_decoders + 1, n_slices = gridDim.x * WAVES;
  const Slice sl = slice_of<WAVES>(b, w, chunk, n);
  WaveTable<REG> h{0u, lds + w * cols};
  if constexpr (!REG)
    for (uint32_t i = lane; i < cols; i += kWave) h.lds[i] = 0;
  // With the register table the invalid queries are counted apart, in a
  // wave-uniform counter, so that all 64 lanes can hold decoders.
  uint32_t invalid = 0;
  for (uint64_t base = sl.beg; base < sl.end; base += kWaveQuantum) {
    uint32_t d[kBatchRows];
    load_batch(tex_id, tex_to_dec, n_textures, n_decoders, n_decoders, base, sl.end, lane, d);
#pragma unroll
    for (int j = 0; j < kBatchRows; ++j) {
      if constexpr (REG) {
        const uint64_t bad = ballot(d[j] == n_decoders);
        invalid += (uint32_t)__builtin_popcountll(bad);
        rank_row<REG, false>(d[j] == n_decoders ? kOutside : d[j], h, lane);
      } else {
        rank_row<REG, false>(d[j], h, lane);
      }
    }
  }
  if constexpr (REG) {
    const size_t col = b * WAVES + w;
    if (!tot) {
      if (lane < n_decoders) hist[(size_t)lane * n_slices + col] = h.reg;
      if (lane == 0) hist[(size_t)n_decoders * n_slices + col] = invalid;
    } else {
      part[w][lane] = h.reg;
      if (lane == 0) part[w][kWave] = invalid;
      __syncthreads();
      if (lane < n_decoders) {
        uint32_t excl = 0;
        for (uint32_t k = 0; k < w; ++k) excl += part[k][lane];
        hist[(size_t)lane * n_slices + col] = excl;
      }
      if (threadIdx.x < cols) {
        const uint32_t r = threadIdx.x < n_decoders ? threadIdx.x : kWave;
        uint32_t sum = 0;
#pragma unroll
        for (int k = 0; k < WAVES; ++k) sum += part[k][r];
        tot[(size_t)threadIdx.x * gridDim.x + b] = sum;
      }
    }
  } else {
    // the workgroup's WAVES slices are neighbours in every row of hist: thread
    // t writes row t / WAVES, slice t % WAVES, so a wave covers 64 / WAVES rows
    // with pieces of 4 WAVES bytes
    __syncthreads();
    for (uint32_t i = threadIdx.x; i < cols * WAVES; i += WAVES * kWave) {
      const uint32_t r = i / WAVES, ww = i % WAVES;
      hist[(size_t)r * n_slices + b * WAVES + ww] = lds[ww * cols + r];
    }
  }
}

// Exclusive scan over the workgroup of one value per thread; returns the total.
// tmp: one LDS word per wave.
template <int WAVES>
__device__ uint32_t block_exclusive_scan(uint32_t v, uint32_t &excl, uint32_t *tmp) {
  const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
  uint32_t incl = v;
#pragma unroll
  for (int s = 1; s < kWave; s <<= 1) {
    const uint32_t o = __shfl_up(incl, s, kWave);
    if (lane >= (uint32_t)s) incl += o;
  }
  if (lane == kWave - 1) tmp[w] = incl;
  __syncthreads();
  uint32_t base = 0, total = 0;
#pragma unroll
  for (int k = 0; k < WAVES; ++k) {
    const uint32_t t = tmp[k];
    base += k < (int)w ? t : 0u;
    total += t;
  }
  __syncthreads();
  excl = base + incl - v;
  return total;
}

// Workgroup d scans row d of hist[cols][n_slices]; thread i owns slices
// [i * kScanPerThread, ...) and loads all of them at once.
__global__ void __launch_bounds__(kScanThreads)
bins_scan(uint32_t *__restrict__ hist, uint32_t n_slices, uint32_t n_decoders,
          uint32_t *__restrict__ bin_count, uint32_t *__restrict__ status,
          uint32_t *__restrict__ invalid_out) {
  __shared__ uint32_t tmp[kScanThreads / kWave];
  const uint32_t d = blockIdx.x;
  const uint32_t s0 = threadIdx.x * kScanPerThread;
  uint32_t *row = hist + (size_t)d * n_slices;
  uint32_t v[kScanPerThread];
  uint32_t sum = 0;
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    v[k] = s0 + k < n_slices ? row[s0 + k] : 0u;
    sum += v[k];
  }
  uint32_t excl;
  const uint32_t total = block_exclusive_scan<kScanThreads / kWave>(sum, excl, tmp);
#pragma unroll
  for (int k = 0; k < kScanPerThread; ++k) {
    if (s0 + k < n_slices) row[s0 + k] = excl;
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

// Place of the three-kernel path.
template <bool REG>
__global__ void __launch_bounds__(kBlock)
bins_place(const uint32_t *__restrict__ tex_id, uint32_t n,
           const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures, uint32_t n_decoders,
           uint32_t align, uint32_t chunk, const uint32_t *__restrict__ hist,
           const uint32_t *__restrict__ bin_count, uint32_t *__restrict__ bin_offset,
           uint32_t *__restrict__ perm) {
  extern __shared__ uint32_t lds[];  // kWavesPerBlock x n_decoders cursors
  __shared__ uint32_t scan_tmp[kWavesPerBlock];
  const uint32_t D = n_decoders;
  const uint32_t b = xcd_local_block(blockIdx.x, gridDim.x), lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint32_t nblocks = gridDim.x, n_slices = nblocks * kWavesPerBlock;
  const Slice sl = slice_of<kWavesPerBlock>(b, w, chunk, n);
  // The first batch's ids are in flight during the offset scan below; invalid
  // queries are marked as outside: they go nowhere.
  uint32_t d[kBatchRows];
  if (sl.beg < sl.end)
    load_batch(tex_id, tex_to_dec, n_textures, D, kOutside, sl.beg, sl.end, lane, d);
  // Padded bin offsets: thread i owns decoders [dlo, dhi).
  const uint32_t dper = (D + kBlock - 1) / kBlock;
  const uint32_t dlo = min(threadIdx.x * dper, D);
  const uint32_t dhi = min(dlo + dper, D);
  uint32_t psum = 0;
  for (uint32_t k = dlo; k < dhi; ++k) psum += (bin_count[k] + align - 1) & ~(align - 1);
  uint32_t off;
  const uint32_t total = block_exclusive_scan<kWavesPerBlock>(psum, off, scan_tmp);
  // the slices' prefixes of decoder k: one 16-byte piece (n_slices is a
  // multiple of 4 and hist 16-byte aligned)
  static_assert(kWavesPerBlock == 4, "one 16-byte piece per decoder");
  const uint32_t *prefix = hist + b * kWavesPerBlock;
  for (uint32_t k = dlo; k < dhi; ++k) {
    const uint32_t cnt = bin_count[k];
    const uint32_t padded = (cnt + align - 1) & ~(align - 1);
    const uint4 p = *(const uint4 *)(prefix + (size_t)k * n_slices);
    lds[0 * D + k] = off + p.x;
    lds[1 * D + k] = off + p.y;
    lds[2 * D + k] = off + p.z;
    lds[3 * D + k] = off + p.w;
    if (b == 0) bin_offset[k] = off;
    if (k % nblocks == b)  // the padding slots of bin k
      for (uint32_t s = off + cnt; s < off + padded; ++s) perm[s] = NTC_PAD;
    off += padded;
  }
  if (b == 0 && threadIdx.x == 0) bin_offset[D] = total;
  __syncthreads();
  WaveTable<REG> cur{0u, lds + w * D};
  if constexpr (REG) cur.reg = lane < D ? cur.lds[lane] : 0u;
  for (uint64_t base = sl.beg; base < sl.end; base += kWaveQuantum) {
    if (base != sl.beg)
      load_batch(tex_id, tex_to_dec, n_textures, D, kOutside, base, sl.end, lane, d);
#pragma unroll
    for (int j = 0; j < kBatchRows; ++j) {
      const uint32_t pos = rank_row<REG, true>(d[j], cur, lane);
      if (d[j] != kOutside) perm[pos] = (uint32_t)(base + (uint64_t)j * kWave + lane);
    }
  }
}

// Place of the two-kernel path (register tables, n_decoders <= 64): the offsets
// come from tot and from this workgroup's columns of hist.
// Eight waves per SIMD (with 16-wave workgroups two per CU), so every
// workgroup of a 4K frame is resident at once (the scalar registers decide).
template <int WAVES>
__global__ void __launch_bounds__(WAVES * kWave) __attribute__((amdgpu_waves_per_eu(8)))
bins_place_sum(const uint32_t *__restrict__ tex_id, uint32_t n,
               const uint32_t *__restrict__ tex_to_dec, uint32_t n_textures,
               uint32_t n_decoders, uint32_t align, uint32_t chunk,
               const uint32_t *__restrict__ hist, const uint32_t *__restrict__ tot,
               uint32_t *__restrict__ bin_count, uint32_t *__restrict__ bin_offset,
               uint32_t *__restrict__ perm, uint32_t *__restrict__ status,
               uint32_t *__restrict__ invalid_out) {
  __shared__ uint32_t total[kWave + 1], before[kWave + 1], start[kWave];
  const uint32_t D = n_decoders;
  const uint32_t b = xcd_local_block(blockIdx.x, gridDim.x), lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
  const uint32_t nblocks = gridDim.x, n_slices = nblocks * WAVES;
  const Slice sl = slice_of<WAVES>(b, w, chunk, n);
  // The first batch's ids are in flight while the offsets are summed; invalid
  // queries are marked as outside: they go nowhere.
  uint32_t d[kBatchRows];
  if (sl.beg < sl.end)
    load_batch(tex_id, tex_to_dec, n_textures, D, kOutside, sl.beg, sl.end, lane, d);
  // Row r of tot (r = D: invalid queries): its total and its sum over the
  // workgroups before this one.  kSumLanes lanes take a row, kSumPer words
  // each, all loaded at once.
  static_assert(kSumLanes * kSumPer >= kSumBlocks, "a row fits its lanes");
  for (uint32_t t = threadIdx.x; t < kSumLanes * (D + 1); t += WAVES * kWave) {
    const uint32_t r = t / kSumLanes, i0 = (t % kSumLanes) * kSumPer;
    const uint32_t *row = tot + (size_t)r * nblocks;
    uint32_t v[kSumPer];
#pragma unroll
    for (int k = 0; k < kSumPer; ++k) v[k] = i0 + k < nblocks ? row[i0 + k] : 0u;
    uint32_t all = 0, prior = 0;
#pragma unroll
    for (int k = 0; k < kSumPer; ++k) {
      all += v[k];
      prior += i0 + k < b ? v[k] : 0u;
    }
    // the kSumLanes lanes of a row are one aligned group, all active
#pragma unroll
    for (int sh = kSumLanes / 2; sh > 0; sh >>= 1) {
      all += __shfl_xor(all, sh, kWave);
      prior += __shfl_xor(prior, sh, kWave);
    }
    const uint32_t k = r < D ? r : kWave;
    if (t % kSumLanes == 0) {
      total[k] = all;
      before[k] = prior;
    }
  }
  __syncthreads();
  if (w == 0) {
    // padded bin offsets: lane k holds decoder k
    const uint32_t cnt = lane < D ? total[lane] : 0u;
    const uint32_t padded = (cnt + align - 1) & ~(align - 1);
    uint32_t incl = padded;
#pragma unroll
    for (int s = 1; s < kWave; s <<= 1) {
      const uint32_t o = __shfl_up(incl, s, kWave);
      if (lane >= (uint32_t)s) incl += o;
    }
    const uint32_t off = incl - padded;
    start[lane] = off;
    if (b == 0) {
      if (lane < D) {
        bin_count[lane] = cnt;
        bin_offset[lane] = off;
      }
      if (lane == kWave - 1) {
        bin_offset[D] = incl;
        status[1] = total[kWave];
        if (invalid_out) *invalid_out = total[kWave];
      }
    }
    if (lane < D && lane % nblocks == b)  // the padding slots of bin `lane`
      for (uint32_t s = off + cnt; s < off + padded; ++s) perm[s] = NTC_PAD;
  }
  __syncthreads();
  // this wave's cursor of decoder k (lane k): the bin's offset, the queries of
  // the workgroups before this one, then those of this workgroup's earlier waves
  WaveTable<true> cur{0u, nullptr};
  if (lane < D) cur.reg = start[lane] + before[lane] + hist[(size_t)lane * n_slices + b * WAVES + w];
  for (uint64_t base = sl.beg; base < sl.end; base += kWaveQuantum) {
    if (base != sl.beg)
      load_batch(tex_id, tex_to_dec, n_textures, D, kOutside, base, sl.end, lane, d);
#pragma unroll
    for (int j = 0; j < kBatchRows; ++j) {
      const uint32_t pos = rank_row<true, true>(d[j], cur, lane);
      if (d[j] != kOutside) perm[pos] = (uint32_t)(base + (uint64_t)j * kWave + lane);
    }
  }
}

// The two kernels of the register-table path, on workgroups of WAVES waves.
template <int WAVES>
void launch_sum(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                int32_t n_textures, uint32_t D, int32_t align, const BinsLayout &L,
                uint32_t *hist, uint32_t *tot, uint32_t *bin_count, uint32_t *bin_offset,
                uint32_t *perm, uint32_t *status, uint32_t *invalid_out, hipStream_t stream) {
  const dim3 grid((unsigned)L.blocks), block(WAVES * kWave);
  hipLaunchKernelGGL((bins_count<true, WAVES>), grid, block, 0, stream, tex_id, (uint32_t)n,
                     tex_to_dec, (uint32_t)n_textures, D, (uint32_t)L.chunk, hist, tot);
  hipLaunchKernelGGL(bins_place_sum<WAVES>, grid, block, 0, stream, tex_id, (uint32_t)n,
                     tex_to_dec, (uint32_t)n_textures, D, (uint32_t)align, (uint32_t)L.chunk,
                     hist, tot, bin_count, bin_offset, perm, status, invalid_out);
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

// Workgroups and queries per workgroup for chunks of multiples of
// kWaveQuantum * waves, at most max_blocks workgroups.
static void split(BinsLayout &L, int64_t n, int64_t max_blocks) {
  const int64_t quantum = kWaveQuantum * L.waves;
  int64_t chunk = (n + max_blocks - 1) / max_blocks;
  chunk = (chunk + quantum - 1) / quantum * quantum;
  if (chunk < quantum) chunk = quantum;
  L.chunk = chunk;
  L.blocks = n > 0 ? (n + chunk - 1) / chunk : 1;
}

BinsLayout bins_layout(int64_t n, int32_t n_decoders) {
  BinsLayout L;
  L.reg = (uint32_t)n_decoders <= kRegDecoders;
  L.sum = false;
  if (L.reg) {
    // the two-kernel path while a place workgroup sums the tot rows in at most
    // kSumRounds rounds of loads (kSumLanes threads per row)
    L.waves = n >= kCus * 16 * kWaveQuantum ? 16 : n >= kCus * 8 * kWaveQuantum ? 8 : 4;
    split(L, n, kSumBlocks);
    L.sum = (int64_t)kSumLanes * (n_decoders + 1) <= (int64_t)kSumRounds * L.waves * kWave;
  }
  if (!L.sum) {
    // fewer, longer slices for many decoders: the histograms stay within 4 MiB
    L.waves = kWavesPerBlock;
    int64_t max_blocks = kMaxHistWords / ((int64_t)kWavesPerBlock * (n_decoders + 1));
    max_blocks = max_blocks < 1 ? 1 : max_blocks > kTargetBlocks ? kTargetBlocks : max_blocks;
    split(L, n, max_blocks);
  }
  L.hist_words = (size_t)(n_decoders + 1) * (size_t)L.blocks * L.waves;
  L.tot_words = L.sum ? (size_t)(n_decoders + 1) * (size_t)L.blocks : 0;
  L.bytes = (kStatusWords + L.hist_words + L.tot_words) * sizeof(uint32_t);
  return L;
}

int launch_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, int32_t align,
                      uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                      void *workspace, uint32_t *invalid_out, hipStream_t stream) {
  const BinsLayout L = bins_layout(n, n_decoders);
  uint32_t *status = (uint32_t *)workspace;
  uint32_t *hist = status + kStatusWords;
  const uint32_t D = (uint32_t)n_decoders;
  if (L.sum) {
    uint32_t *tot = hist + L.hist_words;
    if (L.waves == 16)
      launch_sum<16>(tex_id, n, tex_to_dec, n_textures, D, align, L, hist, tot, bin_count,
                     bin_offset, perm, status, invalid_out, stream);
    else if (L.waves == 8)
      launch_sum<8>(tex_id, n, tex_to_dec, n_textures, D, align, L, hist, tot, bin_count,
                    bin_offset, perm, status, invalid_out, stream);
    else
      launch_sum<4>(tex_id, n, tex_to_dec, n_textures, D, align, L, hist, tot, bin_count,
                    bin_offset, perm, status, invalid_out, stream);
    return hip_status(hipGetLastError());
  }
  const uint32_t n_slices = (uint32_t)L.blocks * kWavesPerBlock;
  const size_t lds_count = L.reg ? 0 : (size_t)kWavesPerBlock * (D + 1) * sizeof(uint32_t);
  const size_t lds_place = (size_t)kWavesPerBlock * D * sizeof(uint32_t);
  const void *count_fn = L.reg ? (const void *)bins_count<true, kWavesPerBlock>
                               : (const void *)bins_count<false, kWavesPerBlock>;
  const void *place_fn = L.reg ? (const void *)bins_place<true> : (const void *)bins_place<false>;
  int st = allow_lds(count_fn, lds_count);
  if (st == NTC_OK) st = allow_lds(place_fn, lds_place);
  if (st != NTC_OK) return st;
  const dim3 grid((unsigned)L.blocks), block(kBlock);
  if (L.reg)
    hipLaunchKernelGGL((bins_count<true, kWavesPerBlock>), grid, block, lds_count, stream, tex_id,
                       (uint32_t)n, tex_to_dec, (uint32_t)n_textures, D, (uint32_t)L.chunk, hist,
                       nullptr);
  else
    hipLaunchKernelGGL((bins_count<false, kWavesPerBlock>), grid, block, lds_count, stream, tex_id,
                       (uint32_t)n, tex_to_dec, (uint32_t)n_textures, D, (uint32_t)L.chunk, hist,
                       nullptr);
  hipLaunchKernelGGL(bins_scan, dim3(D + 1), dim3(kScanThreads), 0, stream, hist, n_slices, D,
                     bin_count, status, invalid_out);
  if (L.reg)
    hipLaunchKernelGGL(bins_place<true>, grid, block, lds_place, stream, tex_id, (uint32_t)n,
                       tex_to_dec, (uint32_t)n_textures, D, (uint32_t)align, (uint32_t)L.chunk,
                       hist, bin_count, bin_offset, perm);
  else
    hipLaunchKernelGGL(bins_place<false>, grid, block, lds_place, stream, tex_id, (uint32_t)n,
                       tex_to_dec, (uint32_t)n_textures, D, (uint32_t)align, (uint32_t)L.chunk,
                       hist, bin_count, bin_offset, perm);
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
