/*
 * ntc_oracle.c -- plain CPU oracle for neural texture decode with decoder binning.
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the
 * benchmark's CPU-baseline leg, never by the product path.  No code is shared
 * with the GPU library.  All arithmetic is IEEE double; nothing is blocked,
 * fused or reordered beyond what the definitions state.  The only parallelism
 * is an OpenMP loop over independent queries.
 *
 * Paper passages followed:
 *   - Sec. 1: the encoder output is a latent grid/pyramid, the decoder an MLP;
 *   - Sec. 4 (setup): the latent grid is sampled, the samples are concatenated
 *     and fed to a multi-layer MLP;
 *   - Alg. "Overall texture processing pipeline", Stage 2: texture i uses
 *     decoder c(i);
 *   - Sec. 2: divergence map = number of distinct ids per block, and the metric
 *     of Eq. (normalized_ones_metric).
 * Where the paper is silent (sampling convention, activations, level blending,
 * binning order), the reading taken is stated next to the code that takes it.
 */
#include "ntc_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

double ntc_oracle_half_to_double(uint16_t h) {
  int sign = (h >> 15) & 1;
  int expo = (h >> 10) & 0x1f;
  int mant = h & 0x3ff;
  double v;
  if (expo == 0) {
    v = ldexp((double)mant, -24); /* subnormal: mant * 2^-14 * 2^-10 */
  } else if (expo == 31) {
    v = mant ? NAN : INFINITY;
  } else {
    v = ldexp((double)(mant | 0x400), expo - 25); /* (1.mant) * 2^(expo-15) */
  }
  return sign ? -v : v;
}

/* ------------------------------------------------------------------ binning */

int ntc_oracle_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                          int32_t n_textures, int32_t n_decoders, int32_t align,
                          uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                          int64_t perm_capacity, int64_t *n_invalid) {
  if (n < 0 || n_textures < 0 || n_decoders < 1 || align < 1 || (align & (align - 1)) != 0)
    return NTC_ORACLE_ERR_ARG;
  if (!bin_count || !bin_offset || (n > 0 && (!tex_id || !perm)) ||
      (n_textures > 0 && !tex_to_dec))
    return NTC_ORACLE_ERR_ARG;

  int64_t bad = 0;
  /* 1. histogram of decoder ids */
  for (int32_t d = 0; d < n_decoders; ++d) bin_count[d] = 0;
  for (int64_t q = 0; q < n; ++q) {
    uint32_t t = tex_id[q];
    if (t >= (uint32_t)n_textures) { ++bad; continue; }
    uint32_t d = tex_to_dec[t];
    if (d >= (uint32_t)n_decoders) { ++bad; continue; }
    bin_count[d] += 1;
  }
  /* 2. exclusive scan of the counts, each rounded up to a multiple of align */
  uint64_t acc = 0;
  for (int32_t d = 0; d < n_decoders; ++d) {
    bin_offset[d] = (uint32_t)acc;
    uint64_t c = bin_count[d];
    acc += (c + (uint64_t)align - 1) / (uint64_t)align * (uint64_t)align;
  }
  bin_offset[n_decoders] = (uint32_t)acc;
  if ((int64_t)acc > perm_capacity || acc > 0xFFFFFFFFull) return NTC_ORACLE_ERR_CAPACITY;
  /* 3. padding everywhere, then each query in ascending order to its bin's cursor */
  for (uint64_t i = 0; i < acc; ++i) perm[i] = NTC_ORACLE_PAD;
  uint32_t *cursor = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n_decoders);
  if (!cursor) return NTC_ORACLE_ERR_ARG;
  for (int32_t d = 0; d < n_decoders; ++d) cursor[d] = bin_offset[d];
  for (int64_t q = 0; q < n; ++q) {
    uint32_t t = tex_id[q];
    if (t >= (uint32_t)n_textures) continue;
    uint32_t d = tex_to_dec[t];
    if (d >= (uint32_t)n_decoders) continue;
    perm[cursor[d]] = (uint32_t)q;
    cursor[d] += 1;
  }
  free(cursor);
  if (n_invalid) *n_invalid = bad;
  return NTC_ORACLE_OK;
}

/* --------------------------------------------------------------- divergence */

int ntc_oracle_divergence(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                          int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                          int64_t len, int32_t wave, uint32_t *per_wave, uint64_t *totals) {
  if (n < 0 || len < 0 || wave < 1 || n_decoders < 1 || !totals) return NTC_ORACLE_ERR_ARG;
  if (len > 0 && (!per_wave || !tex_id)) return NTC_ORACLE_ERR_ARG;
  totals[0] = totals[1] = totals[2] = totals[3] = 0;
  uint32_t *seen = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)wave);
  if (!seen) return NTC_ORACLE_ERR_ARG;
  int64_t n_windows = (len + wave - 1) / wave;
  for (int64_t w = 0; w < n_windows; ++w) {
    /* the set of distinct ids of this window, kept as a plain list */
    int n_seen = 0;
    for (int64_t i = w * wave; i < len && i < (w + 1) * wave; ++i) {
      uint64_t q = order ? order[i] : (uint64_t)i;
      if (q >= (uint64_t)n) continue;
      uint32_t t = tex_id[q];
      if (t >= (uint32_t)n_textures) continue;
      uint32_t d = tex_to_dec[t];
      if (d >= (uint32_t)n_decoders) continue;
      int found = 0;
      for (int k = 0; k < n_seen; ++k)
        if (seen[k] == d) { found = 1; break; }
      if (!found) seen[n_seen++] = d;
    }
    per_wave[w] = (uint32_t)n_seen;
    if (n_seen > 0) {
      totals[0] += 1;
      totals[1] += (uint64_t)n_seen;
      if (n_seen > 1) totals[2] += 1;
      if ((uint64_t)n_seen > totals[3]) totals[3] = (uint64_t)n_seen;
    }
  }
  free(seen);
  return NTC_ORACLE_OK;
}

int ntc_oracle_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                              const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                              int32_t block_w, int32_t block_h, uint32_t *map,
                              uint32_t *histogram, int32_t hist_len, uint64_t *totals) {
  if (!tex_id || !tex_to_dec || !map || !histogram || !totals || width < 1 || height < 1 ||
      spp < 1 || block_w < 1 || block_h < 1 || n_textures < 1 || n_decoders < 1 || hist_len < 1)
    return NTC_ORACLE_ERR_ARG;
  const int64_t bx = (width + block_w - 1) / block_w, by = (height + block_h - 1) / block_h;
  totals[0] = totals[1] = totals[2] = totals[3] = 0;
  for (int k = 0; k < hist_len; ++k) histogram[k] = 0;
  const int64_t cap = (int64_t)block_w * block_h * spp;
  uint32_t *seen = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)cap);
  if (!seen) return NTC_ORACLE_ERR_ARG;
  for (int64_t i = 0; i < by; ++i) {
    for (int64_t j = 0; j < bx; ++j) {
      /* the distinct decoder ids of block (i, j), kept as a plain list */
      int64_t n_seen = 0;
      for (int64_t y = i * block_h; y < height && y < (i + 1) * block_h; ++y) {
        for (int64_t x = j * block_w; x < width && x < (j + 1) * block_w; ++x) {
          for (int64_t s = 0; s < spp; ++s) {
            uint32_t t = tex_id[(y * width + x) * spp + s];
            if (t >= (uint32_t)n_textures) continue;
            uint32_t d = tex_to_dec[t];
            if (d >= (uint32_t)n_decoders) continue;
            int found = 0;
            for (int64_t k = 0; k < n_seen; ++k)
              if (seen[k] == d) { found = 1; break; }
            if (!found) seen[n_seen++] = d;
          }
        }
      }
      map[i * bx + j] = (uint32_t)n_seen;
      histogram[n_seen < hist_len - 1 ? n_seen : hist_len - 1] += 1;
      if (n_seen > 0) {
        totals[0] += 1;
        totals[1] += (uint64_t)n_seen;
        if (n_seen > 1) totals[2] += 1;
        if ((uint64_t)n_seen > totals[3]) totals[3] = (uint64_t)n_seen;
      }
    }
  }
  free(seen);
  return NTC_ORACLE_OK;
}

/* ----------------------------------------------------------------- sampling */

static double lerp(double a, double b, double t) { return a + t * (b - a); }

static int clampi(int64_t v, int lo, int hi) {
  return (int)(v < lo ? lo : (v > hi ? hi : v));
}

/*
 * Bilinear sample of one level at (u, v): texel centres sit at (i + 1/2)/res,
 * taps outside the grid are clamped to the edge, and the two horizontal lerps
 * are followed by one vertical lerp.  Writes ch values to f.
 */
static void sample_level(const uint16_t *level, int res, int ch, double u, double v, double *f) {
  double x = u * res - 0.5, y = v * res - 0.5;
  double x0f = floor(x), y0f = floor(y);
  double fx = x - x0f, fy = y - y0f;
  /* far outside the grid both taps clamp to the same edge texel; bound the
     integer conversion so it stays defined for any finite uv */
  if (x0f < -1.0) x0f = -1.0;
  if (x0f > res) x0f = res;
  if (y0f < -1.0) y0f = -1.0;
  if (y0f > res) y0f = res;
  int x0 = clampi((int64_t)x0f, 0, res - 1), x1 = clampi((int64_t)x0f + 1, 0, res - 1);
  int y0 = clampi((int64_t)y0f, 0, res - 1), y1 = clampi((int64_t)y0f + 1, 0, res - 1);
  const uint16_t *t00 = level + ((size_t)y0 * res + x0) * ch;
  const uint16_t *t10 = level + ((size_t)y0 * res + x1) * ch;
  const uint16_t *t01 = level + ((size_t)y1 * res + x0) * ch;
  const uint16_t *t11 = level + ((size_t)y1 * res + x1) * ch;
  for (int c = 0; c < ch; ++c) {
    double top = lerp(ntc_oracle_half_to_double(t00[c]), ntc_oracle_half_to_double(t10[c]), fx);
    double bot = lerp(ntc_oracle_half_to_double(t01[c]), ntc_oracle_half_to_double(t11[c]), fx);
    f[c] = lerp(top, bot, fy);
  }
}

static int grids_valid(int32_t n_levels, const int32_t *res, const int32_t *ch, int has_mip) {
  if (n_levels < 1 || n_levels > 8 || !res || !ch) return 0;
  for (int l = 0; l < n_levels; ++l) {
    if (res[l] < 1 || ch[l] < 1 || ch[l] > 256) return 0;
    if (has_mip && ch[l] != ch[0]) return 0;
  }
  return 1;
}

/*
 * Feature vector of one query.  Slot l samples the pyramid at level of detail
 * lod = max(l, m), m = mip clamped to [0, L-1]: the two levels around lod are
 * sampled and blended linearly (trilinear filtering); lod integral means a
 * single bilinear sample.  With mip == 0, slot l is exactly level l.
 */
static void query_features(const uint16_t *tex_base, int32_t n_levels, const int32_t *res,
                           const int32_t *ch, const size_t *level_off, double u, double v,
                           double mipv, double *x, double *scratch) {
  double m = mipv;
  if (!(m > 0.0)) m = 0.0; /* also maps NaN to 0 */
  if (m > n_levels - 1) m = n_levels - 1;
  int pos = 0;
  for (int l = 0; l < n_levels; ++l) {
    double lod = (double)l > m ? (double)l : m;
    int k0 = (int)floor(lod);
    int k1 = k0 + 1 < n_levels ? k0 + 1 : n_levels - 1;
    double t = lod - k0;
    sample_level(tex_base + level_off[k0], res[k0], ch[k0], u, v, x + pos);
    if (t != 0.0) {
      sample_level(tex_base + level_off[k1], res[k1], ch[k1], u, v, scratch);
      for (int c = 0; c < ch[l]; ++c) x[pos + c] = lerp(x[pos + c], scratch[c], t);
    }
    pos += ch[l];
  }
}

/*
 * Positional encoding of (u, v) with K octaves, appended to the decoder input
 * (Sec. 4 setup: the encoder output is concatenated with a positional
 * encoding; the paper does not give its form, this is the library's reading):
 * for k = 0 .. K-1, sin(2^k pi u), cos(2^k pi u), sin(2^k pi v), cos(2^k pi v).
 */
static void pos_encoding(double u, double v, int K, double *x) {
  for (int k = 0; k < K; ++k) {
    const double a = ldexp(3.14159265358979323846, k); /* 2^k pi */
    x[4 * k + 0] = sin(a * u);
    x[4 * k + 1] = cos(a * u);
    x[4 * k + 2] = sin(a * v);
    x[4 * k + 3] = cos(a * v);
  }
}

static void level_layout(int32_t n_levels, const int32_t *res, const int32_t *ch, size_t *off,
                         size_t *stride) {
  size_t acc = 0;
  for (int l = 0; l < n_levels; ++l) {
    off[l] = acc;
    acc += (size_t)res[l] * (size_t)res[l] * (size_t)ch[l];
  }
  *stride = acc;
}

int ntc_oracle_features(const uint16_t *latents, int32_t n_textures, int32_t n_levels,
                        const int32_t *res, const int32_t *ch, const uint32_t *tex_id,
                        const float *uv, const float *mip, int64_t n, const int64_t *subset,
                        int64_t n_sel, int32_t n_threads, int32_t pe_octaves, double *out) {
  if (!grids_valid(n_levels, res, ch, mip != NULL) || n < 0 || pe_octaves < 0 ||
      pe_octaves > 16)
    return NTC_ORACLE_ERR_ARG;
  if (!subset) n_sel = n;
  if (n_sel < 0 || (n_sel > 0 && (!latents || !tex_id || !uv || !out))) return NTC_ORACLE_ERR_ARG;
  size_t off[8], stride;
  level_layout(n_levels, res, ch, off, &stride);
  int FL = 0;
  for (int l = 0; l < n_levels; ++l) FL += ch[l];
  const int F = FL + 4 * pe_octaves;
  int bad = 0;
#pragma omp parallel for schedule(static) num_threads(n_threads > 0 ? n_threads : 1)
  for (int64_t i = 0; i < n_sel; ++i) {
    int64_t q = subset ? subset[i] : i;
    if (q < 0 || q >= n) { bad = 1; continue; }
    uint32_t t = tex_id[q];
    if (t >= (uint32_t)n_textures) continue;
    double scratch[256];
    query_features(latents + (size_t)t * stride, n_levels, res, ch, off, uv[2 * q],
                   uv[2 * q + 1], mip ? (double)mip[q] : 0.0, out + (size_t)i * F, scratch);
    pos_encoding(uv[2 * q], uv[2 * q + 1], pe_octaves, out + (size_t)i * F + FL);
  }
  return bad ? NTC_ORACLE_ERR_ARG : NTC_ORACLE_OK;
}

/* ---------------------------------------------------------------------- MLP */

static int dims_valid(int32_t n_layers, const int32_t *dims) {
  if (n_layers < 1 || n_layers > 8 || !dims) return 0;
  for (int i = 0; i <= n_layers; ++i)
    if (dims[i] < 1 || dims[i] > 256) return 0;
  return 1;
}

/*
 * One decoder on one feature vector: for each layer z_j = b_j + sum_k W_jk h_k
 * (ascending k); between layers h = z for z > 0 and slope * z otherwise (ReLU for
 * slope 0, the LeakyReLU of the Sec. 4 setup for slope > 0); logistic sigmoid on
 * the last layer.
 */
static void mlp(const uint16_t *p, int32_t n_layers, const int32_t *dims, const double *x,
                double slope, double *y) {
  double h[256], z[256];
  for (int k = 0; k < dims[0]; ++k) h[k] = x[k];
  for (int i = 0; i < n_layers; ++i) {
    int din = dims[i], dout = dims[i + 1];
    const uint16_t *W = p;
    const uint16_t *b = p + (size_t)din * dout;
    for (int j = 0; j < dout; ++j) {
      double s = ntc_oracle_half_to_double(b[j]);
      for (int k = 0; k < din; ++k) s += ntc_oracle_half_to_double(W[(size_t)j * din + k]) * h[k];
      z[j] = s;
    }
    p = b + dout;
    if (i + 1 < n_layers) {
      for (int j = 0; j < dout; ++j) h[j] = z[j] > 0.0 ? z[j] : slope * z[j];
    } else {
      for (int j = 0; j < dout; ++j) y[j] = 1.0 / (1.0 + exp(-z[j]));
    }
  }
}

int ntc_oracle_decode(const uint16_t *latents, int32_t n_textures, int32_t n_levels,
                      const int32_t *res, const int32_t *ch, const uint16_t *params,
                      int32_t n_decoders, int32_t n_layers, const int32_t *dims,
                      const uint32_t *tex_to_dec, const uint32_t *tex_id, const float *uv,
                      const float *mip, int64_t n, const int64_t *subset, int64_t n_sel,
                      int32_t n_threads, double leaky_slope, int32_t pe_octaves, double *out) {
  if (!grids_valid(n_levels, res, ch, mip != NULL) || !dims_valid(n_layers, dims) || n < 0 ||
      n_decoders < 1 || !(leaky_slope >= 0.0 && leaky_slope < 1.0) || pe_octaves < 0 ||
      pe_octaves > 16)
    return NTC_ORACLE_ERR_ARG;
  int FL = 0;
  for (int l = 0; l < n_levels; ++l) FL += ch[l];
  if (dims[0] != FL + 4 * pe_octaves) return NTC_ORACLE_ERR_ARG;
  if (!subset) n_sel = n;
  if (n_sel < 0 || (n_sel > 0 && (!latents || !params || !tex_to_dec || !tex_id || !uv || !out)))
    return NTC_ORACLE_ERR_ARG;
  size_t off[8], stride;
  level_layout(n_levels, res, ch, off, &stride);
  size_t dec_stride = 0;
  for (int i = 0; i < n_layers; ++i) dec_stride += (size_t)dims[i + 1] * (dims[i] + 1);
  int out_dim = dims[n_layers];
  int bad = 0;
#pragma omp parallel for schedule(static) num_threads(n_threads > 0 ? n_threads : 1)
  for (int64_t i = 0; i < n_sel; ++i) {
    int64_t q = subset ? subset[i] : i;
    if (q < 0 || q >= n) { bad = 1; continue; }
    uint32_t t = tex_id[q];
    if (t >= (uint32_t)n_textures) continue;
    uint32_t d = tex_to_dec[t];
    if (d >= (uint32_t)n_decoders) continue;
    double x[256], scratch[256];
    query_features(latents + (size_t)t * stride, n_levels, res, ch, off, uv[2 * q],
                   uv[2 * q + 1], mip ? (double)mip[q] : 0.0, x, scratch);
    pos_encoding(uv[2 * q], uv[2 * q + 1], pe_octaves, x + FL);
    mlp(params + (size_t)d * dec_stride, n_layers, dims, x, leaky_slope,
        out + (size_t)i * out_dim);
  }
  return bad ? NTC_ORACLE_ERR_ARG : NTC_ORACLE_OK;
}
