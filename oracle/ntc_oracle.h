/*
 * ntc_oracle.h -- plain CPU oracle for neural texture decode with decoder binning.
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists to check the GPU library
 * against a slow, obviously correct implementation of the same definitions.
 * Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it; the product path never does.  It shares no code, header, table or
 * helper with the GPU library.
 *
 * Floating point is evaluated in IEEE double.  Stored latents and decoder
 * parameters are fp16 (the paper's decode runs in FP16, Sec. 4.4 "Performance
 * analysis"); they are widened exactly to double before use.
 *
 * Definitions followed (paper sections / equations):
 *   - texture -> decoder map c(i): Alg. "Overall texture processing pipeline",
 *     Stage 2 and Sec. 3.3 "Clustering into m groups";
 *   - decode = latent-grid sampling, concatenation, MLP decoder: Sec. 1
 *     (encoder output is a latent pyramid or grid, decoder is an MLP) and
 *     Sec. 4 setup (grid, concatenation, MLP layers);
 *   - divergence map D(i,j) = number of distinct ids per block and the metric
 *     of Eq. (normalized_ones_metric): Sec. 2 "Thread Divergence in NTC".
 * The binning by decoder id is not in the paper; it is the counting sort
 * spelled out in ntc_oracle_build_bins below.
 *
 * Every function is pinned by a host test against something other than
 * itself (brute force, library routines, closed forms); see the test files
 * tests/test_oracle_*.py.
 */
#ifndef NTC_ORACLE_H
#define NTC_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define NTC_ORACLE_PAD 0xFFFFFFFFu

/* Return codes. */
#define NTC_ORACLE_OK 0
#define NTC_ORACLE_ERR_ARG (-1)
#define NTC_ORACLE_ERR_CAPACITY (-3)

/*
 * Stable counting sort of query indices by decoder id.
 *   d(q) = tex_to_dec[tex_id[q]]; a query is invalid (dropped, counted in
 *   *n_invalid) when tex_id[q] >= n_textures or d(q) >= n_decoders.
 *   bin_count[d]  = number of valid queries with decoder d;
 *   bin_offset[0] = 0, bin_offset[d+1] = bin_offset[d] + roundup(bin_count[d], align);
 *   perm[bin_offset[d] + r] = the r-th (in ascending q) valid query of decoder d;
 *   every other slot of [0, bin_offset[n_decoders]) holds NTC_ORACLE_PAD.
 * align must be a power of two >= 1; perm_capacity >= bin_offset[n_decoders].
 */
int ntc_oracle_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                          int32_t n_textures, int32_t n_decoders, int32_t align,
                          uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                          int64_t perm_capacity, int64_t *n_invalid);

/*
 * Per-window distinct decoder count (Sec. 2, divergence map with one block per
 * window of `wave` consecutive entries of an order).
 *   entry i of the order is q = order ? order[i] : i; it is skipped when
 *   q >= n (this covers NTC_ORACLE_PAD), tex_id[q] >= n_textures or its decoder
 *   >= n_decoders.
 *   per_wave[w] = number of distinct decoders among the kept entries of window
 *   w = [w*wave, min(len, (w+1)*wave)).
 *   totals[0] = windows with at least one kept entry,
 *   totals[1] = sum of per_wave, totals[2] = windows with per_wave > 1,
 *   totals[3] = max of per_wave.
 */
int ntc_oracle_divergence(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                          int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                          int64_t len, int32_t wave, uint32_t *per_wave, uint64_t *totals);

/*
 * Divergence map over screen blocks (Sec. 2: D(i,j) = number of distinct ids
 * in block (i,j); Eq. (normalized_ones_metric) from the totals).
 *   The queries form a width x height screen with spp samples per pixel,
 *   q = (y * width + x) * spp + s.  Block (i, j) = pixels x in
 *   [j*block_w, min(width, (j+1)*block_w)), y in [i*block_h, min(height,
 *   (i+1)*block_h)), all their samples.  map[i * Wb + j] = distinct decoder ids
 *   among the block's queries (skipping tex_id >= n_textures and decoder ids
 *   >= n_decoders), Wb = ceil(width / block_w).
 *   histogram[k] = blocks with count k (k < hist_len - 1); histogram[hist_len-1]
 *   = blocks with count >= hist_len - 1.
 *   totals as for ntc_oracle_divergence, over blocks.
 */
int ntc_oracle_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                              const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                              int32_t block_w, int32_t block_h, uint32_t *map,
                              uint32_t *histogram, int32_t hist_len, uint64_t *totals);

/*
 * Feature vector of each query: per slot l = 0..n_levels-1 the latent sampled
 * at uv (bilinear, texel centres at (i + 1/2)/res, clamp-to-edge), blended
 * between adjacent pyramid levels by the query's mip; slots concatenated
 * finest first, channels in storage order.  out: [n_sel][sum(ch)].
 * subset: query indices to evaluate (NULL -> all n, n_sel = n).
 * pe_octaves K >= 0 appends the positional encoding of (u, v) (Sec. 4 setup;
 * its form is a reading): for k = 0 .. K-1, sin(2^k pi u), cos(2^k pi u),
 * sin(2^k pi v), cos(2^k pi v).  Rows are [sum(ch) + 4K] wide.
 * Invalid queries (tex_id >= n_textures) leave their row untouched.
 */
int ntc_oracle_features(const uint16_t *latents, int32_t n_textures, int32_t n_levels,
                        const int32_t *res, const int32_t *ch, const uint32_t *tex_id,
                        const float *uv, const float *mip, int64_t n, const int64_t *subset,
                        int64_t n_sel, int32_t n_threads, int32_t pe_octaves, double *out);

/*
 * Full decode: features as above, then the MLP of decoder tex_to_dec[tex_id[q]]:
 *   z = b_i + W_i h (W_i row-major [d_{i+1}][d_i]); hidden layers
 *   h = z > 0 ? z : leaky_slope * z (ReLU for slope 0, the Sec. 4 setup's
 *   LeakyReLU for 0 < slope < 1); last layer logistic sigmoid.
 *   params: per decoder contiguous
 *   W0, b0, W1, b1, ... (fp16 bits).  out: [n_sel][dims[n_layers]].
 *   The decoder input is the feature row with pe_octaves positional-encoding
 *   octaves appended (dims[0] = sum(ch) + 4 * pe_octaves).
 * Invalid queries (bad tex_id or decoder id) leave their row untouched.
 */
int ntc_oracle_decode(const uint16_t *latents, int32_t n_textures, int32_t n_levels,
                      const int32_t *res, const int32_t *ch, const uint16_t *params,
                      int32_t n_decoders, int32_t n_layers, const int32_t *dims,
                      const uint32_t *tex_to_dec, const uint32_t *tex_id, const float *uv,
                      const float *mip, int64_t n, const int64_t *subset, int64_t n_sel,
                      int32_t n_threads, double leaky_slope, int32_t pe_octaves, double *out);

/* fp16 bit pattern -> double (exact). */
double ntc_oracle_half_to_double(uint16_t h);

#ifdef __cplusplus
}
#endif
#endif
