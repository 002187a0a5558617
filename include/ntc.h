/*
 * ntc.h -- C ABI of libntc: neural texture decode with per-wave decoder binning
 * on AMD Instinct MI355X (gfx950).
 *
 * What is computed (paper: "Thread-Efficient Decoding for Neural Texture
 * Compression"):
 *   - each texture i owns a multi-resolution latent grid (its "encoder" output,
 *     Sec. 1) and uses decoder c(i) (Alg. "Overall texture processing
 *     pipeline", Stage 2, the texture -> group map);
 *   - a texel query (texture, uv, mip) samples the latent grid, concatenates
 *     the per-level samples and runs the texture's MLP decoder (Sec. 1 and the
 *     setup paragraph of Sec. 4);
 *   - a wave that decodes queries of k distinct decoders runs k serial tensor
 *     passes (Sec. 1 and Sec. 4.4); ntc_build_bins groups queries by decoder id
 *     so that every 64-lane wave of ntc_decode runs exactly one decoder;
 *   - ntc_divergence_stats counts distinct decoders per wave-sized block, the
 *     divergence map of Sec. 2, and the totals behind the metric of
 *     Eq. (normalized_ones_metric); ntc_divergence_map does the same over 2-D
 *     screen blocks and adds the histogram of the map.
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers unless marked (host).  The caller owns every
 *     buffer; the library never allocates device memory and keeps no state
 *     between calls.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).  All
 *     device work is enqueued on it and the call returns without waiting,
 *     except ntc_get_device_error and ntc_kmeans_result, which synchronise
 *     the stream, and ntc_kmeans, which waits for its copy of a host array.
 *   - Calls on different streams are independent; two calls that share an
 *     output or workspace buffer must be ordered by the caller.
 *   - Arguments are validated on the host before anything is enqueued; on an
 *     error nothing is enqueued and a negative ntc_status is returned.
 */
#ifndef NTC_H
#define NTC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  NTC_OK = 0,
  NTC_ERR_ARG = -1,         /* NULL pointer, negative or too large size, bad alignment */
  NTC_ERR_UNSUPPORTED = -2, /* a shape the kernels are not built for */
  NTC_ERR_CAPACITY = -3,    /* an output or workspace buffer is too small */
  NTC_ERR_HIP = -4,         /* a HIP runtime call failed */
  NTC_ERR_INDEX = -5        /* device-side: a query named a texture or decoder out of range */
} ntc_status;

#define NTC_PAD 0xFFFFFFFFu /* padding entry of a bin in `perm` */
#define NTC_MAX_LEVELS 4
#define NTC_MAX_LAYERS 8
#define NTC_MAX_DECODERS 4096 /* binning keeps one counter per decoder in LDS */
#define NTC_MAX_ALIGN 4096

/*
 * Latent grids, one block per texture, all textures alike.  Level l is a
 * res[l] x res[l] grid of channels[l] fp16 values per texel, stored [y][x][c]
 * (channel-last).  Texture t starts at latents + t * S, S = sum_l res[l]^2 *
 * channels[l]; inside it the levels follow one another, finest first.
 * Sampling (Sec. 1 "latent pyramids or grids"): bilinear, texel centres at
 * ((i + 1/2) / res, (j + 1/2) / res), clamp-to-edge addressing.
 */
typedef struct {
  int32_t n_textures;
  int32_t n_levels;                  /* 1 .. NTC_MAX_LEVELS */
  int32_t res[NTC_MAX_LEVELS];       /* (host values) */
  int32_t channels[NTC_MAX_LEVELS];  /* (host values) */
  const uint16_t *latents;           /* fp16 bit patterns */
} ntc_grids;

/*
 * MLP decoders (Sec. 4 setup: an MLP of a few fully connected layers).  Layer
 * i maps dims[i] -> dims[i+1]: z = W_i h + b_i, W_i row-major [dims[i+1]][dims[i]].
 * Hidden layers apply ReLU, the last layer the logistic sigmoid, so decoded
 * channels lie in [0, 1].  Decoder d occupies params + d * P with
 * P = sum_i dims[i+1] * (dims[i] + 1) fp16 values laid out W_0, b_0, W_1, b_1, ...
 */
typedef struct {
  int32_t n_decoders;
  int32_t n_layers;                  /* 1 .. NTC_MAX_LAYERS */
  int32_t dims[NTC_MAX_LAYERS + 1];  /* (host values); dims[0] = sum of grid channels */
  const uint16_t *params;            /* fp16 bit patterns */
} ntc_decoders;

/*
 * Query stream, one entry per texel request in issue order (row-major pixels,
 * samples innermost).  uv is [n][2] float; any finite uv is valid (taps clamp
 * to the edge).  mip may be NULL (all zero).  With a mip, slot l of the
 * feature vector samples the pyramid at level of detail max(l, mip), mip
 * clamped to [0, n_levels-1], blending the two levels around it linearly; all
 * levels must then have the same channel count.
 */
typedef struct {
  const uint32_t *tex_id;  /* [n] */
  const float *uv;         /* [n][2] */
  const float *mip;        /* [n] or NULL */
  int64_t n;               /* 0 .. 2^32 - 2 */
} ntc_queries;

/* (host) Bytes of device workspace ntc_build_bins needs for n queries and
 * n_decoders bins; 0 when the arguments are out of range. */
size_t ntc_bins_workspace_bytes(int64_t n, int32_t n_decoders);

/* (host) Entries `perm` must hold: n + n_decoders * (align - 1), the largest
 * padded total; -1 when the arguments are out of range. */
int64_t ntc_bins_capacity(int64_t n, int32_t n_decoders, int32_t align);

/*
 * Bin queries by decoder id: a stable counting sort.  With d(q) =
 * tex_to_dec[tex_id[q]]:
 *   bin_count[d]  = |{q : d(q) = d}|                          (u32 [n_decoders])
 *   bin_offset[0] = 0, bin_offset[d+1] = bin_offset[d] + roundup(bin_count[d], align)
 *                                                             (u32 [n_decoders + 1])
 *   perm[bin_offset[d] + r] = the r-th query of decoder d in ascending q order;
 *   slots [bin_offset[d] + bin_count[d], bin_offset[d+1]) hold NTC_PAD; entries
 *   at and past bin_offset[n_decoders] are left untouched.
 * The result is unique, so it is reproducible bit for bit.  Queries with
 * tex_id >= n_textures or d(q) >= n_decoders are left out of every bin and
 * counted; read the count with ntc_get_device_error.
 * align: power of two in [1, NTC_MAX_ALIGN]; 64 (one wave) for ntc_decode.
 * perm_capacity >= ntc_bins_capacity(n, n_decoders, align) (NTC_ERR_CAPACITY).
 * workspace: device buffer of >= ntc_bins_workspace_bytes(n, n_decoders) bytes,
 * 16-byte aligned (NTC_ERR_ARG otherwise), owned by the caller, contents need
 * not be initialised; it holds the invalid-query count until the next call
 * that uses it.
 * n = 0 is valid: bin_count and bin_offset become all zero.
 */
int ntc_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                   int32_t n_textures, int32_t n_decoders, int32_t align,
                   uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                   int64_t perm_capacity, void *workspace, size_t workspace_bytes,
                   void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * ntc_build_bins with the library's own device scratch in place of a caller
 * workspace.  Arguments, results and errors are those of ntc_build_bins,
 * except that:
 *   - the scratch is a static device array of NTC_NOALLOC_SCRATCH_BYTES bytes,
 *     one per GPU the library runs on, held until the process ends.  A call
 *     needs ntc_bins_workspace_bytes(n, n_decoders) bytes of it, which is at
 *     most 4 MiB + 16 bytes whatever n and n_decoders, so every valid call
 *     fits; a call that needed more would return NTC_ERR_CAPACITY before
 *     anything is enqueued;
 *   - n_invalid (device, may be NULL) receives the number of queries left out
 *     of every bin, the count ntc_get_device_error reads for ntc_build_bins;
 *   - every call on one GPU works in that GPU's one scratch array, which keeps
 *     the last call's contents (nothing in it needs to start at zero): calls
 *     that overlap on one GPU (different streams, or threads without ordering)
 *     race and give undefined results; calls ordered on one stream are safe.
 * It calls no hipMalloc, hipFree or other allocating routine.  Its first call
 * on a device looks up that device's scratch address (NTC_ERR_HIP on failure).
 */
#define NTC_NOALLOC_SCRATCH_BYTES (5u << 20)
int ntc_build_bins_noalloc(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                           int32_t n_textures, int32_t n_decoders, int32_t align,
                           uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                           int64_t perm_capacity, uint32_t *n_invalid, void *stream);

/*
 * (synchronises `stream`) Number of queries the last ntc_build_bins on this
 * workspace left out because of an out-of-range texture or decoder id; writes it
 * to *n_invalid (host, may be NULL).  Returns NTC_OK when it is zero,
 * NTC_ERR_INDEX otherwise.
 */
int ntc_get_device_error(const void *workspace, uint64_t *n_invalid, void *stream);

/*
 * The feature vector of every query, without the MLP (the gather step of
 * ntc_decode; Sec. 1 "latent pyramids or grids", sampled as described for
 * ntc_queries): out[q][c] for c < F = n_levels * channels, row-major [n][F],
 * slot l (level l, or the blend of the levels around max(l, mip)) at
 * [l * channels, (l + 1) * channels).  The values are those ntc_decode feeds
 * its MLP: bilinear weights rounded to fp16, every product and sum an fp16
 * operation; out_format NTC_OUT_F32 widens them to float32 exactly,
 * NTC_OUT_F16 stores them as fp16 bit patterns.  Rows of queries with
 * tex_id >= n_textures are left untouched.
 * Shapes as for ntc_decode: (n_levels, channels) in {(2, 8), (2, 16), (3, 16)},
 * level resolutions in 2 .. 16384, latents of one texture < 2^31 values
 * (NTC_ERR_UNSUPPORTED otherwise; malformed grids NTC_ERR_ARG).
 * Alignment (NTC_ERR_ARG otherwise, when n > 0): latents and out 16 bytes, uv
 * 8 bytes, tex_id and mip 4 bytes.
 */
int ntc_gather_features(const ntc_grids *grids, const ntc_queries *queries, void *out,
                        int32_t out_format, void *stream);

/*
 * Decode every query: out[q][c] = MLP_{d(q)}(features(q))[c], float32,
 * [n][dims[n_layers]] row-major, rows in original query order.
 *   Binned mode (bin_offset != NULL): queries are taken from `perm` in tiles of
 *   64 consecutive slots, each tile belonging to one bin (align must be a
 *   multiple of 64 and equal to the align given to ntc_build_bins); the tile's
 *   decoder is its bin's, and tex_to_dec is not read.  NTC_PAD slots and slots
 *   holding q >= n are skipped.  perm_capacity must be the capacity passed to
 *   ntc_build_bins.
 *   Stream mode (bin_offset == NULL): tiles are 64 consecutive queries; a wave
 *   whose tile holds k distinct decoders runs the MLP k times (the divergent
 *   execution of Sec. 1 and Sec. 4.4); perm is ignored.
 * Rows of queries with tex_id >= n_textures (or, in stream mode, a decoder id
 * >= n_decoders) are left untouched.  A query's result depends only on that
 * query, so both modes give identical bits.
 * Supported shapes (else NTC_ERR_UNSUPPORTED): (n_levels, channels per level)
 * in {(2, 8), (2, 16), (3, 16)}, the same channel count on every level and
 * dims[0] = their sum; 3 or 4 layers whose hidden widths are all equal, 64 or
 * 128; dims[n_layers] in 1 .. 16; level resolutions in 2 .. 16384;
 * latents of one texture < 2^31 values; output of one call at most
 * 4 GiB - 512 bytes (n * dims[n_layers] * 4 bytes).  Other malformed shapes give NTC_ERR_ARG.
 * Alignment (NTC_ERR_ARG otherwise, when n > 0): latents 16 bytes (taps are read
 * as 16-byte pieces), uv 8 bytes, tex_id, mip and out 4 bytes (2 for fp16 rows).
 */
int ntc_decode(const ntc_grids *grids, const ntc_decoders *decoders,
               const uint32_t *tex_to_dec, const ntc_queries *queries,
               const uint32_t *bin_offset, const uint32_t *perm, int64_t perm_capacity,
               int32_t align, float *out, void *stream);

#define NTC_ACT_RELU 0       /* hidden activation max(x, 0) */
#define NTC_ACT_LEAKY_RELU 1 /* hidden activation max(x, slope * x) */
#define NTC_OUT_F32 0        /* output rows of float */
#define NTC_OUT_F16 1        /* output rows of fp16 (IEEE binary16 bits, rounded to nearest even) */

/*
 * Decoder variants of ntc_decode_ex.  The Sec. 4 setup trains its decoders with
 * LeakyReLU hidden activations, the encoder output concatenated with a
 * positional encoding, and three output channels (RGB); fp16 output rows halve
 * the bytes the decode writes.
 *
 * Positional encoding (the paper names it without its form; this is the
 * library's reading): with K = pe_octaves, the decoder input is the latent
 * feature vector followed by 4K values, for k = 0 .. K-1 in order
 *   sin(2^k pi u), cos(2^k pi u), sin(2^k pi v), cos(2^k pi v)
 * of the query's (u, v), so dims[0] = sum of channels + 4K.  K is 0 (none), 4
 * or 8; K > 0 is supported for 2 levels of 8 or 16 channels, 3 layers of
 * hidden width 64 and queries without mip (else NTC_ERR_UNSUPPORTED).
 */
typedef struct {
  int32_t hidden_activation; /* NTC_ACT_RELU or NTC_ACT_LEAKY_RELU */
  float leaky_slope;         /* NTC_ACT_LEAKY_RELU only: 0 < slope < 1 (held as fp16) */
  int32_t output_format;     /* NTC_OUT_F32 or NTC_OUT_F16 */
  int32_t pe_octaves;        /* positional-encoding octaves K: 0, 4 or 8 */
  int32_t engine;            /* NTC_ENGINE_MFMA or NTC_ENGINE_FMA */
  int32_t gather;            /* NTC_GATHER_DIRECT or NTC_GATHER_STAGED */
} ntc_decode_options;

/*
 * Engines (Sec. 4.4 compares a shared decoder with two non-shared
 * implementations, one on tensor instructions and one on plain fused
 * multiply-adds):
 *   NTC_ENGINE_MFMA: the MLP runs on MFMA once per decoder present in a wave
 *     (ntc_decode's engine); binned or stream mode.
 *   NTC_ENGINE_FMA: every lane evaluates its own query's decoder with vector
 *     fp16 dot products (fp32 accumulation), reading that decoder's weights
 *     itself, so a wave's cost does not depend on how many decoders it holds
 *     (the paper's Non-Shared FMA).  With hidden width 64 the weights come from
 *     a per-CU LDS cache of whole decoders (a tile of 1024 queries stages the
 *     decoders it misses; a tile with more distinct decoders than the cache
 *     holds takes several passes); other widths read them as with
 *     NTC_ENGINE_FMA_DIRECT.
 *   NTC_ENGINE_FMA_DIRECT: the same per-lane evaluation with every lane
 *     loading its weight rows through the L1/L2 caches (16-byte loads).
 *   Both FMA engines: stream mode only (NTC_ERR_UNSUPPORTED with bin_offset);
 *     dims[n_layers] must be 8 or 16 (NTC_ERR_UNSUPPORTED) and decoders->params
 *     16-byte aligned (NTC_ERR_ARG).  Results agree with the MFMA engine within
 *     rounding, not bit for bit, and with each other bit for bit.
 */
#define NTC_ENGINE_MFMA 0
#define NTC_ENGINE_FMA 1
#define NTC_ENGINE_FMA_DIRECT 2

/*
 * Latent gathers (Sec. 1: each query samples its texture's latent grid):
 *   NTC_GATHER_DIRECT: every lane loads the four bilinear taps of its query
 *     from memory, level by level (the default, and the faster of the two on
 *     MI355X).
 *   NTC_GATHER_STAGED: the taps of a 64-query tile are staged in LDS first.
 *     A query whose bilinear quad differs from the previous query's in the
 *     tile leads; each leader's quad is loaded once, by several lanes, into a
 *     wave-private LDS region (prefetched one tile ahead), and every query
 *     reads its taps from there.  The MLP then runs on 16x16x32 MFMAs.
 *     Binned decode with the MFMA engine only, 2 levels, no mip and output
 *     widths up to 8 (NTC_ERR_UNSUPPORTED otherwise).  Results agree with the
 *     direct gather within rounding (the MFMA shape differs), not bit for bit.
 */
#define NTC_GATHER_DIRECT 0
#define NTC_GATHER_STAGED 1

/*
 * ntc_decode with options (NULL = ReLU, float rows and the MFMA engine, i.e.
 * ntc_decode).  `out`
 * holds n * dims[n_layers] elements of the chosen format, rows in original
 * query order; with NTC_OUT_F16 the bytes are n * dims[n_layers] * 2 (same
 * 4 GiB - 512 limit).  LeakyReLU is applied to the fp16-rounded pre-activation,
 * in fp16.  Invalid options give NTC_ERR_ARG; everything else as ntc_decode.
 */
int ntc_decode_ex(const ntc_grids *grids, const ntc_decoders *decoders,
                  const uint32_t *tex_to_dec, const ntc_queries *queries,
                  const uint32_t *bin_offset, const uint32_t *perm, int64_t perm_capacity,
                  int32_t align, const ntc_decode_options *options, void *out, void *stream);

/*
 * Divergence per wave-sized block (Sec. 2): for window w = entries
 * [w * wave, min(len, (w+1) * wave)) of an order, per_wave_distinct[w] = number
 * of distinct decoder ids d(q) over the window's entries q = order[i] (order ==
 * NULL: q = i).  Entries with q >= n (NTC_PAD included), tex_id[q] >= n_textures
 * or d(q) >= n_decoders are skipped.  totals (u64 [4]) = {windows with at least
 * one entry kept, sum of per_wave_distinct, windows with more than one decoder,
 * largest per_wave_distinct}.  The metric of Eq. (normalized_ones_metric) over
 * the kept windows is totals[1] / totals[0] - 1.  Pass an identity tex_to_dec
 * to count distinct textures instead.  wave: 1 .. 64.
 * per_wave_distinct: u32 [ceil(len / wave)].
 */
int ntc_divergence_stats(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                         int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                         int64_t len, int32_t wave, uint32_t *per_wave_distinct,
                         uint64_t *totals, void *stream);

/*
 * Divergence map of Sec. 2 over screen blocks.  The queries form a screen of
 * width x height pixels with spp samples per pixel in row-major order,
 * q = (y * width + x) * spp + s, n = width * height * spp.  Block (i, j) holds
 * every sample of the pixels x in [j * block_w, min(width, (j + 1) * block_w)),
 * y in [i * block_h, min(height, (i + 1) * block_h)), so edge blocks may be
 * partial.  map[i * Wb + j] = number of distinct decoder ids d(q) among the
 * block's queries, skipping queries with tex_id >= n_textures or
 * d(q) >= n_decoders; Wb = ceil(width / block_w), Hb = ceil(height / block_h);
 * map: u32 [Hb * Wb].  histogram (u32 [hist_len]): histogram[k] = number of
 * blocks whose count is k for k < hist_len - 1; the last entry counts every
 * block whose count is >= hist_len - 1.  totals (u64 [4]) = {blocks with at
 * least one query kept, sum of map, blocks with more than one decoder, largest
 * count}; the metric of Eq. (normalized_ones_metric) over the kept blocks is
 * totals[1] / totals[0] - 1.  Pass an identity tex_to_dec to count textures.
 * Limits: width, height, block_w, block_h >= 1; spp 1 .. 64;
 * width * height * spp <= 2^32 - 2; hist_len 1 .. 4096.
 */
int ntc_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                       const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                       int32_t block_w, int32_t block_h, uint32_t *map, uint32_t *histogram,
                       int32_t hist_len, uint64_t *totals, void *stream);

/*
 * Stage 2 of Alg. "Overall texture processing pipeline" (Sec. 3.3): k-means
 * clustering of one feature vector per texture (the paper clusters CLIP
 * embeddings of the textures, Stage 1) into m groups; assign[i] = c(i) is then the texture ->
 * decoder map of ntc_build_bins and ntc_decode, and counts[g] = k_g the size
 * of group g.  Lloyd's algorithm in float64:
 *   centroid g starts as the features of texture init[g];
 *   iteration t: every texture takes the nearest centroid (squared Euclidean
 *   distance, ties to the lower g); if no label changed (t > 0) the run stops;
 *   otherwise every centroid becomes the mean of its textures (members summed
 *   in ascending i, then divided by their count); an empty group keeps its
 *   centroid.
 * At most max_iter iterations; ntc_kmeans_result reports how many ran and
 * whether the labels converged.  A label decided by a near-exact distance tie
 * may differ from another implementation's.
 *   features:  f32 [n][dim] (device), row-major
 *   init:      u32 [m] (HOST), distinct texture indices < n (the seeding is the
 *              caller's choice; the paper does not state one); copied to the
 *              device before the call returns (the call waits for `stream`)
 *   assign:    u32 [n] (device, output)
 *   centroids: f64 [m][dim] (device, output)
 *   counts:    u32 [m] (device, output)
 *   workspace: >= ntc_kmeans_workspace_bytes(m, max_iter) bytes (device),
 *              4-byte aligned; holds the iteration state until its next use.
 * Limits: 1 <= m <= min(n, NTC_MAX_DECODERS); n <= NTC_KMEANS_MAX_POINTS;
 * dim <= NTC_KMEANS_MAX_DIM; 1 <= max_iter <= NTC_KMEANS_MAX_ITER (else
 * NTC_ERR_ARG).  Work per iteration is O(n * m * dim) for the assignment and
 * O(m * n * dim) for the update (one workgroup per group scans all labels).
 */
#define NTC_KMEANS_MAX_POINTS (1 << 20)
#define NTC_KMEANS_MAX_DIM 65536
#define NTC_KMEANS_MAX_ITER 4096
size_t ntc_kmeans_workspace_bytes(int32_t m, int32_t max_iter);
int ntc_kmeans(const float *features, int32_t n, int32_t dim, int32_t m, const uint32_t *init,
               int32_t max_iter, uint32_t *assign, double *centroids, uint32_t *counts,
               void *workspace, size_t workspace_bytes, void *stream);

/* (synchronises `stream`) Iterations the last ntc_kmeans on this workspace ran
 * (the last one found no label change when *converged is 1; otherwise the run
 * stopped at max_iter).  Either output may be NULL. */
int ntc_kmeans_result(const void *workspace, int32_t m, int32_t max_iter, int32_t *iterations,
                      int32_t *converged, void *stream);

/*
 * (host) Gradual decoder freezing (Sec. 3.2, Alg. SelfFreezeDecoderGradually):
 * the factor lambda(e) in [0, 1] that scales the shared decoder's updates at
 * epoch e, 1/2 (1 + cos(pi p)) with p = clamp((e - freeze_start) /
 * freeze_duration, 0, 1): 1 before the freezing window, a half-cosine down to
 * 0 across it, 0 after it.  freeze_start = NaN means no freezing (1 always); a
 * freeze_duration <= 0 freezes at freeze_start.
 */
double ntc_freeze_scale(double epoch, double freeze_start, double freeze_duration);

/* (host) Static description of a status code. */
const char *ntc_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* NTC_H */
