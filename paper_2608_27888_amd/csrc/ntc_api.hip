// ntc_api.hip -- the extern "C" entry points of libntc: host-side validation,
// then the kernel launches of ntc_bins.hip, ntc_decode.hip, ntc_divergence.hip.
#include <algorithm>
#include <cmath>
#include <mutex>
#include <vector>

#include "ntc_internal.h"

using namespace ntc;

// Device scratch of ntc_build_bins_noalloc, in place of a caller workspace:
// one copy per GPU the library runs on, held until the process ends.  In host
// code `scratch` only names the variable; its device address on the current
// GPU comes from hipGetSymbolAddress, looked up once per device.
static __device__ __align__(256) unsigned char scratch[NTC_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int64_t kMaxQueries = 0xFFFFFFFELL;  // ids and slots are 32-bit; NTC_PAD reserved

bool pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void *scratch_ptr[kMaxDevices] = {};

// Device address of this GPU's scratch (the current device), or NULL.
void *device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void *p = nullptr;
    size_t bytes = 0;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    if (hipGetSymbolSize(&bytes, HIP_SYMBOL(scratch)) != hipSuccess ||
        bytes != (size_t)NTC_NOALLOC_SCRATCH_BYTES)
      return nullptr;
    scratch_ptr[dev] = p;
  }
  return scratch_ptr[dev];
}

// Host checks shared by ntc_build_bins and ntc_build_bins_noalloc.
int check_bins_args(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                    int32_t n_textures, int32_t n_decoders, int32_t align,
                    const uint32_t *bin_count, const uint32_t *bin_offset, const uint32_t *perm,
                    int64_t perm_capacity) {
  if (n < 0 || n > kMaxQueries || n_textures < 1 || n_decoders < 1 ||
      n_decoders > NTC_MAX_DECODERS || !pow2(align) || align > NTC_MAX_ALIGN)
    return NTC_ERR_ARG;
  if (!tex_to_dec || !bin_count || !bin_offset || (n > 0 && (!tex_id || !perm)))
    return NTC_ERR_ARG;
  const int64_t cap = ntc_bins_capacity(n, n_decoders, align);
  if (perm_capacity < cap || cap > kMaxQueries + 1) return NTC_ERR_CAPACITY;
  return NTC_OK;
}

}  // namespace

extern "C" {

const char *ntc_status_string(int status) {
  switch (status) {
    case NTC_OK: return "ok";
    case NTC_ERR_ARG: return "invalid argument";
    case NTC_ERR_UNSUPPORTED: return "unsupported shape";
    case NTC_ERR_CAPACITY: return "buffer too small";
    case NTC_ERR_HIP: return "HIP runtime error";
    case NTC_ERR_INDEX: return "texture or decoder id out of range";
    default: return "unknown status";
  }
}

size_t ntc_bins_workspace_bytes(int64_t n, int32_t n_decoders) {
  if (n < 0 || n > kMaxQueries || n_decoders < 1 || n_decoders > NTC_MAX_DECODERS) return 0;
  return bins_layout(n, n_decoders).bytes;
}

int64_t ntc_bins_capacity(int64_t n, int32_t n_decoders, int32_t align) {
  if (n < 0 || n > kMaxQueries || n_decoders < 1 || n_decoders > NTC_MAX_DECODERS ||
      !pow2(align) || align > NTC_MAX_ALIGN)
    return -1;
  return n + (int64_t)n_decoders * (align - 1);
}

int ntc_build_bins(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                   int32_t n_textures, int32_t n_decoders, int32_t align,
                   uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                   int64_t perm_capacity, void *workspace, size_t workspace_bytes,
                   void *stream) {
  const int st = check_bins_args(tex_id, n, tex_to_dec, n_textures, n_decoders, align, bin_count,
                                 bin_offset, perm, perm_capacity);
  if (st != NTC_OK) return st;
  if (!workspace || ((uintptr_t)workspace & 15)) return NTC_ERR_ARG;
  if (workspace_bytes < ntc_bins_workspace_bytes(n, n_decoders)) return NTC_ERR_CAPACITY;
  return launch_build_bins(tex_id, n, tex_to_dec, n_textures, n_decoders, align, bin_count,
                           bin_offset, perm, workspace, nullptr, (hipStream_t)stream);
}

int ntc_build_bins_noalloc(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                           int32_t n_textures, int32_t n_decoders, int32_t align,
                           uint32_t *bin_count, uint32_t *bin_offset, uint32_t *perm,
                           int64_t perm_capacity, uint32_t *n_invalid, void *stream) {
  const int st = check_bins_args(tex_id, n, tex_to_dec, n_textures, n_decoders, align, bin_count,
                                 bin_offset, perm, perm_capacity);
  if (st != NTC_OK) return st;
  if (ntc_bins_workspace_bytes(n, n_decoders) > (size_t)NTC_NOALLOC_SCRATCH_BYTES)
    return NTC_ERR_CAPACITY;
  void *ws = device_scratch();
  if (!ws) return NTC_ERR_HIP;
  return launch_build_bins(tex_id, n, tex_to_dec, n_textures, n_decoders, align, bin_count,
                           bin_offset, perm, ws, n_invalid, (hipStream_t)stream);
}

int ntc_get_device_error(const void *workspace, uint64_t *n_invalid, void *stream) {
  if (!workspace) return NTC_ERR_ARG;
  return read_invalid_count(workspace, n_invalid, (hipStream_t)stream);
}

// Level layout of the grids into a: offsets, resolutions, values per texture,
// latents and texture count (the level count is checked by the caller).
static int set_grids(const ntc_grids *g, DecodeArgs &a) {
  const int ch = g->channels[0];
  int64_t tex_stride = 0;
  for (int l = 0; l < g->n_levels; ++l) {
    const int r = g->res[l];
    if (r < 1 || r > 16384 || g->channels[l] < 1) return NTC_ERR_ARG;
    if (r < 2) return NTC_ERR_UNSUPPORTED;  // the gather addresses a 2x2 quad
    if (g->channels[l] != ch) return NTC_ERR_UNSUPPORTED;
    a.level_off[l] = (uint32_t)tex_stride;
    a.res[l] = r;
    a.resf[l] = (float)r;
    tex_stride += (int64_t)r * r * ch;
    if (tex_stride >= ((int64_t)1 << 31)) return NTC_ERR_UNSUPPORTED;
  }
  a.latents = g->latents;
  a.tex_stride = tex_stride;
  a.n_textures = g->n_textures;
  return NTC_OK;
}

int ntc_gather_features(const ntc_grids *g, const ntc_queries *q, void *out, int32_t out_format,
                        void *stream) {
  if (!g || !q) return NTC_ERR_ARG;
  if (out_format != NTC_OUT_F32 && out_format != NTC_OUT_F16) return NTC_ERR_ARG;
  if (q->n < 0 || q->n > kMaxQueries) return NTC_ERR_ARG;
  if (g->n_textures < 1 || g->n_levels < 1 || g->n_levels > NTC_MAX_LEVELS) return NTC_ERR_ARG;
  if (q->n > 0 && (!g->latents || !q->tex_id || !q->uv || !out)) return NTC_ERR_ARG;
  // taps as 16-byte pieces, (u, v) as one 8-byte pair, rows as 16-byte pieces
  if (q->n > 0 && (((uintptr_t)g->latents & 15) || ((uintptr_t)q->uv & 7) ||
                   ((uintptr_t)q->tex_id & 3) || ((uintptr_t)q->mip & 3) ||
                   ((uintptr_t)out & 15)))
    return NTC_ERR_ARG;
  DecodeArgs a = {};
  const int gs = set_grids(g, a);
  if (gs != NTC_OK) return gs;
  a.tex_id = q->tex_id;
  a.uv = q->uv;
  a.mip = q->mip;
  a.n = (uint32_t)q->n;
  a.out = out;
  if (q->n == 0) {
    const int L = g->n_levels, ch = g->channels[0];
    const bool known = (L == 2 && (ch == 8 || ch == 16)) || (L == 3 && ch == 16);
    return known ? NTC_OK : NTC_ERR_UNSUPPORTED;
  }
  return launch_gather(a, g->n_levels, g->channels[0], out_format == NTC_OUT_F16,
                       (hipStream_t)stream);
}

int ntc_decode(const ntc_grids *g, const ntc_decoders *m, const uint32_t *tex_to_dec,
               const ntc_queries *q, const uint32_t *bin_offset, const uint32_t *perm,
               int64_t perm_capacity, int32_t align, float *out, void *stream) {
  return ntc_decode_ex(g, m, tex_to_dec, q, bin_offset, perm, perm_capacity, align, nullptr,
                       out, stream);
}

int ntc_decode_ex(const ntc_grids *g, const ntc_decoders *m, const uint32_t *tex_to_dec,
                  const ntc_queries *q, const uint32_t *bin_offset, const uint32_t *perm,
                  int64_t perm_capacity, int32_t align, const ntc_decode_options *opt,
                  void *out, void *stream) {
  if (!g || !m || !q) return NTC_ERR_ARG;
  ntc_decode_options o = {NTC_ACT_RELU, 0.f, NTC_OUT_F32, 0, NTC_ENGINE_MFMA, NTC_GATHER_DIRECT};
  if (opt) o = *opt;
  if (o.hidden_activation != NTC_ACT_RELU && o.hidden_activation != NTC_ACT_LEAKY_RELU)
    return NTC_ERR_ARG;
  if (o.hidden_activation == NTC_ACT_LEAKY_RELU && !(o.leaky_slope > 0.f && o.leaky_slope < 1.f))
    return NTC_ERR_ARG;
  if (o.output_format != NTC_OUT_F32 && o.output_format != NTC_OUT_F16) return NTC_ERR_ARG;
  if (o.pe_octaves != 0 && o.pe_octaves != 4 && o.pe_octaves != 8) return NTC_ERR_ARG;
  if (o.engine != NTC_ENGINE_MFMA && o.engine != NTC_ENGINE_FMA &&
      o.engine != NTC_ENGINE_FMA_DIRECT)
    return NTC_ERR_ARG;
  if (o.gather != NTC_GATHER_DIRECT && o.gather != NTC_GATHER_STAGED) return NTC_ERR_ARG;
  const bool fma = o.engine != NTC_ENGINE_MFMA;
  const int64_t elem = o.output_format == NTC_OUT_F16 ? 2 : 4;
  if (q->n < 0 || q->n > kMaxQueries) return NTC_ERR_ARG;
  if (g->n_textures < 1 || g->n_levels < 1 || g->n_levels > NTC_MAX_LEVELS) return NTC_ERR_ARG;
  if (m->n_decoders < 1 || m->n_decoders > NTC_MAX_DECODERS || m->n_layers < 1 ||
      m->n_layers > NTC_MAX_LAYERS)
    return NTC_ERR_ARG;
  const bool binned = bin_offset != nullptr;
  if (q->n > 0 && (!g->latents || !m->params || !q->tex_id || !q->uv || !out))
    return NTC_ERR_ARG;
  // taps are loaded as 16-byte pieces of a texel row, (u, v) as one 8-byte pair
  if (q->n > 0 && (((uintptr_t)g->latents & 15) || ((uintptr_t)q->uv & 7) ||
                   ((uintptr_t)q->tex_id & 3) || ((uintptr_t)q->mip & 3) ||
                   ((uintptr_t)out & (elem - 1))))
    return NTC_ERR_ARG;
  // the FMA engine reads 16-byte weight vectors straight from the parameter block
  if (fma && ((uintptr_t)m->params & 15)) return NTC_ERR_ARG;
  if (binned) {
    if (!perm || align < 64 || !pow2(align) || align > NTC_MAX_ALIGN) return NTC_ERR_ARG;
    if (perm_capacity < ntc_bins_capacity(q->n, m->n_decoders, align)) return NTC_ERR_CAPACITY;
  } else if (!tex_to_dec && q->n > 0) {
    return NTC_ERR_ARG;
  }
  // grid shape
  const int L = g->n_levels;
  const int ch = g->channels[0];
  DecodeArgs a = {};
  const int gs = set_grids(g, a);
  if (gs != NTC_OK) return gs;
  // decoder shape: dims[0] = features, equal hidden widths, small output
  const int F = L * ch + 4 * o.pe_octaves;
  const int nl = m->n_layers;
  if (m->dims[0] != F) return NTC_ERR_ARG;
  for (int i = 0; i <= nl; ++i)
    if (m->dims[i] < 1) return NTC_ERR_ARG;
  if (nl < 2) return NTC_ERR_UNSUPPORTED;
  const int hid = m->dims[1];
  for (int i = 1; i < nl; ++i)
    if (m->dims[i] != hid) return NTC_ERR_UNSUPPORTED;
  const int out_dim = m->dims[nl];
  if (out_dim > 16) return NTC_ERR_UNSUPPORTED;
  // one buffer resource with 32-bit byte offsets covers the output
  if (q->n * (int64_t)out_dim * elem > kMaxOutBytes) return NTC_ERR_UNSUPPORTED;
  int64_t dec_stride = 0;
  for (int i = 0; i < nl; ++i) dec_stride += (int64_t)m->dims[i + 1] * (m->dims[i] + 1);

  a.params = m->params;
  a.dec_stride = dec_stride;
  a.n_decoders = m->n_decoders;
  a.n_hidden = nl - 2;
  a.out_dim = out_dim;
  a.tex_to_dec = tex_to_dec;
  a.tex_id = q->tex_id;
  a.uv = q->uv;
  a.mip = q->mip;
  a.n = (uint32_t)q->n;
  a.bin_offset = bin_offset;
  a.perm = perm;
  a.perm_capacity = binned ? (uint64_t)perm_capacity : 0;
  a.max_tiles = binned ? (uint32_t)((ntc_bins_capacity(q->n, m->n_decoders, align) + 63) / 64)
                       : (uint32_t)((q->n + 63) / 64);
  a.out = out;
  a.leaky = o.hidden_activation == NTC_ACT_LEAKY_RELU;
  const _Float16 slope = (_Float16)o.leaky_slope;
  a.slope_h2 = (uint32_t)__builtin_bit_cast(uint16_t, slope) * 0x00010001u;
  a.out_f16 = o.output_format == NTC_OUT_F16;
  a.pe_octaves = o.pe_octaves;
  a.gather = o.gather;
  a.fma_cache = o.engine == NTC_ENGINE_FMA;
  if (o.gather == NTC_GATHER_STAGED &&
      (fma || !binned || q->mip || L != 2 || out_dim > 8))
    return NTC_ERR_UNSUPPORTED;
  if (fma) {
    if (binned) return NTC_ERR_UNSUPPORTED;  // per-lane decoders: stream order only
    if (out_dim % 8 != 0) return NTC_ERR_UNSUPPORTED;
    if (q->n == 0) return NTC_OK;
    return launch_decode_fma(a, L, ch, hid, (hipStream_t)stream);
  }
  if (q->n == 0) return NTC_OK;
  return launch_decode(a, L, ch, F, hid, (hipStream_t)stream);
}

int ntc_divergence_stats(const uint32_t *tex_id, int64_t n, const uint32_t *tex_to_dec,
                         int32_t n_textures, int32_t n_decoders, const uint32_t *order,
                         int64_t len, int32_t wave, uint32_t *per_wave_distinct,
                         uint64_t *totals, void *stream) {
  if (n < 0 || n > kMaxQueries || len < 0 || n_textures < 1 || n_decoders < 1 || wave < 1 ||
      wave > 64 || !totals || !tex_to_dec)
    return NTC_ERR_ARG;
  if (!order && len > n) return NTC_ERR_ARG;
  if (order && len > kMaxQueries + 1) return NTC_ERR_ARG;
  if (len > 0 && (!per_wave_distinct || (n > 0 && !tex_id))) return NTC_ERR_ARG;
  return launch_divergence(tex_id, n, tex_to_dec, n_textures, n_decoders, order, len, wave,
                           per_wave_distinct, totals, (hipStream_t)stream);
}

int ntc_divergence_map(const uint32_t *tex_id, int32_t width, int32_t height, int32_t spp,
                       const uint32_t *tex_to_dec, int32_t n_textures, int32_t n_decoders,
                       int32_t block_w, int32_t block_h, uint32_t *map, uint32_t *histogram,
                       int32_t hist_len, uint64_t *totals, void *stream) {
  if (!tex_id || !tex_to_dec || !map || !histogram || !totals) return NTC_ERR_ARG;
  if (width < 1 || height < 1 || spp < 1 || spp > 64 || block_w < 1 || block_h < 1 ||
      n_textures < 1 || n_decoders < 1 || n_decoders > NTC_MAX_DECODERS || hist_len < 1 ||
      hist_len > 4096)
    return NTC_ERR_ARG;
  if ((int64_t)width * height * spp > kMaxQueries) return NTC_ERR_ARG;
  return launch_divergence_map(tex_id, width, height, spp, tex_to_dec, n_textures, n_decoders,
                               block_w, block_h, map, histogram, hist_len, totals,
                               (hipStream_t)stream);
}

size_t ntc_kmeans_workspace_bytes(int32_t m, int32_t max_iter) {
  if (m < 1 || m > NTC_MAX_DECODERS || max_iter < 1 || max_iter > NTC_KMEANS_MAX_ITER) return 0;
  return kmeans_workspace_bytes(m, max_iter);
}

int ntc_kmeans(const float *features, int32_t n, int32_t dim, int32_t m, const uint32_t *init,
               int32_t max_iter, uint32_t *assign, double *centroids, uint32_t *counts,
               void *workspace, size_t workspace_bytes, void *stream) {
  if (!features || !init || !assign || !centroids || !counts || !workspace) return NTC_ERR_ARG;
  if (n < 1 || n > NTC_KMEANS_MAX_POINTS || dim < 1 || dim > NTC_KMEANS_MAX_DIM || m < 1 ||
      m > n || m > NTC_MAX_DECODERS || max_iter < 1 || max_iter > NTC_KMEANS_MAX_ITER)
    return NTC_ERR_ARG;
  if ((uintptr_t)workspace & 3) return NTC_ERR_ARG;
  if (workspace_bytes < kmeans_workspace_bytes(m, max_iter)) return NTC_ERR_CAPACITY;
  std::vector<uint32_t> seeds(init, init + m);  // distinct textures, each < n
  std::sort(seeds.begin(), seeds.end());
  if (seeds.back() >= (uint32_t)n || std::adjacent_find(seeds.begin(), seeds.end()) != seeds.end())
    return NTC_ERR_ARG;
  return launch_kmeans(features, n, dim, m, init, max_iter, assign, centroids, counts, workspace,
                       (hipStream_t)stream);
}

int ntc_kmeans_result(const void *workspace, int32_t m, int32_t max_iter, int32_t *iterations,
                      int32_t *converged, void *stream) {
  if (!workspace || m < 1 || m > NTC_MAX_DECODERS || max_iter < 1 ||
      max_iter > NTC_KMEANS_MAX_ITER)
    return NTC_ERR_ARG;
  return read_kmeans_state(workspace, m, max_iter, iterations, converged, (hipStream_t)stream);
}

double ntc_freeze_scale(double epoch, double freeze_start, double freeze_duration) {
  if (std::isnan(freeze_start)) return 1.0;  // no freezing scheduled
  // progress p through the freezing window, clamped to [0, 1]; a window of
  // zero length freezes at its start
  double p;
  if (freeze_duration > 0.0) {
    p = (epoch - freeze_start) / freeze_duration;
    p = p < 0.0 ? 0.0 : (p > 1.0 ? 1.0 : p);
  } else {
    p = epoch >= freeze_start ? 1.0 : 0.0;
  }
  return 0.5 * (1.0 + std::cos(M_PI * p));
}

}  // extern "C"
