// ntc_internal.h -- shared declarations of the HIP library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ntc.h"

namespace ntc {

constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kBlock = 256;        // threads per workgroup in every kernel
constexpr int kWavesPerBlock = kBlock / kWave;

// ----------------------------------------------------------------- wave ops

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Number of set bits of `mask` below this lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t read_lane(uint32_t v, uint32_t lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

// Workgroup index remapped so that consecutive logical indices stay on one XCD:
// the hardware deals workgroups round-robin over the 8 XCDs, each with its own
// L2, so logical neighbours (which read neighbouring data) share an L2.
__device__ __forceinline__ uint32_t xcd_local_block(uint32_t b, uint32_t nblocks) {
  constexpr uint32_t kXcd = 8;
  uint32_t per = nblocks / kXcd, rem = nblocks % kXcd;
  uint32_t xcd = b % kXcd, idx = b / kXcd;
  // XCDs below `rem` own one extra block
  return (xcd < rem ? xcd * (per + 1) : rem * (per + 1) + (xcd - rem) * per) + idx;
}

// ------------------------------------------------------------ host helpers

// Largest output of one decode call: byte offsets into it are 32-bit.
constexpr int64_t kMaxOutBytes = 0xFFFFFE00LL;

struct BinsLayout {
  bool reg;           // register tables (n_decoders <= 64), else LDS tables
  bool sum;           // two kernels (register tables, tot rows small enough), else three
  int waves;          // waves per workgroup
  int64_t chunk;      // queries per workgroup
  int64_t blocks;     // workgroups of the histogram / scatter kernels
  size_t hist_words;  // (n_decoders + 1) * blocks * waves
  size_t tot_words;   // two kernels: (n_decoders + 1) * blocks
  size_t bytes;       // total workspace bytes
};

BinsLayout bins_layout(int64_t n, int32_t n_decoders);

// workspace: bins_layout(n, n_decoders).bytes, 16-byte aligned; invalid_out
// (device, may be NULL) also receives the invalid-query count.
int launch_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, int32_t align,
                      uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                      void *workspace, uint32_t *invalid_out, hipStream_t stream);

size_t bins_status_bytes();
int read_invalid_count(const void *workspace, uint64_t *n_invalid, hipStream_t stream);

int launch_divergence(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                      int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                      int64_t len, int32_t wave, uint32_t *per_wave, uint64_t *totals,
                      hipStream_t stream);
int launch_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                          const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                          int32_t block_w, int32_t block_h, uint32_t *map, uint32_t *histogram,
                          int32_t hist_len, uint64_t *totals, hipStream_t stream);

struct DecodeArgs {
  const uint16_t *latents;
  int64_t tex_stride;                 // fp16 values per texture
  uint32_t level_off[NTC_MAX_LEVELS]; // fp16 offset of each level in a texture
  int32_t res[NTC_MAX_LEVELS];
  float resf[NTC_MAX_LEVELS];
  int32_t n_textures;
  const uint16_t *params;
  int64_t dec_stride;                 // fp16 values per decoder
  int32_t n_decoders;
  int32_t n_hidden;                   // hidden -> hidden layers
  int32_t out_dim;
  const uint32_t *tex_to_dec;
  const uint32_t *tex_id;
  const float *uv;
  const float *mip;
  uint32_t n;
  const uint32_t *bin_offset;         // NULL: stream mode
  const uint32_t *perm;
  uint64_t perm_capacity;             // entries of perm (binned mode)
  uint32_t max_tiles;                 // upper bound of the tile count (grid sizing)
  void *out;
  uint32_t leaky;                     // hidden activation: 0 ReLU, 1 LeakyReLU
  uint32_t slope_h2;                  // LeakyReLU slope as an fp16 pair
  uint32_t out_f16;                   // output rows: 0 fp32, 1 fp16
  int32_t pe_octaves;                 // positional-encoding octaves (0: none)
  int32_t gather;                     // NTC_GATHER_DIRECT or NTC_GATHER_STAGED
  int32_t fma_cache;                  // FMA engine: weights through the LDS decoder cache
  uint32_t split;                     // binned: 2:1 tile ranges for a CU's two workgroups
};

// Returns NTC_ERR_UNSUPPORTED when no kernel is built for the shape.
int launch_decode(const DecodeArgs &a, int n_levels, int channels, int feat, int hidden,
                  hipStream_t stream);
// Feature rows of every query, fp32 or fp16 (ntc_gather_features); the same
// shapes as launch_decode.
int launch_gather(const DecodeArgs &a, int n_levels, int channels, bool f16, hipStream_t stream);
// Per-lane vector-FMA decode in stream order (NTC_ENGINE_FMA); same contract.
int launch_decode_fma(const DecodeArgs &a, int n_levels, int channels, int hidden,
                      hipStream_t stream);

// The kernels of one decoder shape family (levels, channels per level,
// positional-encoding features, hidden width), defined in ntc_decode_kernels.h
// and instantiated once per family in ntc_decode_<family>.hip.
template <int NL, int CH, int PE, int HID>
int launch_decode_shape(const DecodeArgs &a, hipStream_t stream);
template <int NL, int CH, int PE, int HID>
int launch_decode_fma_shape(const DecodeArgs &a, hipStream_t stream);

// k-means of per-texture features (ntc_cluster.hip).  Workspace: m seed
// indices, then one u32 flag per iteration.
size_t kmeans_workspace_bytes(int32_t m, int32_t max_iter);
int launch_kmeans(const float *features, int32_t n, int32_t dim, int32_t m, const uint32_t *init,
                  int32_t max_iter, uint32_t *assign, double *centroids, uint32_t *counts,
                  void *workspace, hipStream_t stream);
int read_kmeans_state(const void *workspace, int32_t m, int32_t max_iter, int32_t *iterations,
                      int32_t *converged, hipStream_t stream);

inline int hip_status(hipError_t e) { return e == hipSuccess ? NTC_OK : NTC_ERR_HIP; }

}  // namespace ntc
