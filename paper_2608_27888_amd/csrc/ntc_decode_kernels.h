#pragma once
// ntc_decode_kernels.h -- fused latent gather + MLP decoder on MFMA (gfx950).
//
// A query samples its texture's latent grid level by level (bilinear, texel
// centres at (i + 1/2)/res, clamp-to-edge; blended between levels by mip),
// concatenates the samples and runs an MLP decoder: ReLU hidden layers and a
// sigmoid output (Sec. 1 and Sec. 4 setup of the paper).  Tensor instructions
// run once per wave, so a wave whose queries use k decoders pays k MLP passes
// (Sec. 1, Sec. 4.4); binned mode feeds each wave one decoder.
//
// Work unit: one wave, one tile of 64 queries (lane l owns query slot l).
//
// Layer math: the layer output H^T = W X^T is computed with
// v_mfma_f32_32x32x16_f16, weights as the A operand (rows = output units) and
// the activations of 32 queries as the B operand (columns = queries); a tile is
// two such 32-query column blocks.  Each lane holds, for its column, 8 K-values
// of A and of B per instruction (half h = lane / 32 holds K-values 8h .. 8h+7 of
// a 16-wide K-slice) and 16 fp32 results: rows 8g + 4h + r (register 4g + r).
// Those 16 results, converted to fp16, are directly the B operand of the next
// layer once the next layer's weight columns are permuted: inside every
// 16-wide K-slice, logical K-position kappa reads hidden unit sigma(kappa), sigma
// swapping bits 2 and 3.  The permutation is applied when the weights are
// staged into LDS, so no activation ever leaves registers.  Biases enter as the
// accumulator input of the first MFMA of each layer.
//
// Decoder weights live in LDS, pre-arranged so that each lane reads its 8
// fp16 A-values of a fragment with one 16-byte load.  Binned mode: a workgroup
// walks a contiguous range of 64-slot tiles of the permutation, four tiles at a
// time (one per wave) inside one bin, restaging weights only when the bin
// changes.  Stream mode: a workgroup takes 4 consecutive tiles, computes the
// features once, then loops over the distinct decoders present; every wave
// that holds queries of that decoder runs its full MLP and keeps the results
// of those lanes only.
//
// A second engine (decode_fma, end of the file) evaluates the MLP per lane with
// vector dot products instead: the paper's Non-Shared FMA comparison.
#include "ntc_internal.h"

namespace ntc {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x3 __attribute__((ext_vector_type(3)));
typedef short short2v __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// Two floats -> packed fp16 pair, round to nearest even (one v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pack_half2(float a, float b) {
  const float2v f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, half2v));
}

__device__ __forceinline__ half8 as_half8(u32x4 v) { return __builtin_bit_cast(half8, v); }

__device__ __forceinline__ floatx16 mfma(half8 a, half8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Logical K-position inside a 16-wide slice -> hidden unit that the previous
// layer's accumulator layout places there.
__device__ __forceinline__ int sigma16(int k) {
  return (k & ~0xC) | ((k & 4) << 1) | ((k & 8) >> 1);
}

template <int NL, int CH, int PE, int HID>
struct Shape {
  static constexpr int FL = NL * CH;         // latent features per query
  static constexpr int F = FL + PE;          // + positional-encoding features
  static constexpr int KS0 = F / 16;         // K-slices of layer 0
  static constexpr int MB = HID / 32;        // 32-row output blocks of a hidden layer
  static constexpr int KSH = HID / 16;       // K-slices of a layer fed by a hidden layer
  static_assert(F % 16 == 0, "feature count must be a multiple of 16");
  static_assert(HID % 32 == 0, "hidden width must be a multiple of 32");
  static_assert(CH == 8 || CH == 16, "8 or 16 channels per level");
  static_assert(PE % 16 == 0, "positional features come in whole K-slices");
};

// LDS image of one decoder: A fragments (64 lanes x 16 B each), then fp32
// biases (rows padded to 32 per block).
struct Image {
  int n_frags;    // fragments
  int bias_off;   // float offset of the biases inside the image (after fragments)
  int n_bias;     // floats
  int bytes;
};

template <int NL, int CH, int PE, int HID>
__host__ __device__ inline Image image_of(int n_hidden) {
  using S = Shape<NL, CH, PE, HID>;
  Image im;
  im.n_frags = S::MB * S::KS0 + n_hidden * S::MB * S::KSH + S::KSH;
  im.bias_off = im.n_frags * 256;  // 1024 B = 256 floats per fragment
  im.n_bias = HID * (1 + n_hidden) + 32;
  im.bytes = (im.bias_off + im.n_bias) * 4;
  return im;
}

// Source of lane-slice lf of the image: the layer's weight block and the row,
// K-slice, half and shape that select its 8 weights.
template <int NL, int CH, int PE, int HID>
struct SliceSource {
  size_t woff;  // offset of W_layer inside the decoder's parameter block
  int layer, row, s, h, din, dout;
};

template <int NL, int CH, int PE, int HID>
__device__ __forceinline__ SliceSource<NL, CH, PE, HID> slice_source(const DecodeArgs &a, int lf) {
  using S = Shape<NL, CH, PE, HID>;
  SliceSource<NL, CH, PE, HID> r;
  const int f = lf / kWave, lane = lf % kWave;
  int mb;
  if (f < S::MB * S::KS0) {
    r.layer = 0; mb = f / S::KS0; r.s = f % S::KS0; r.din = S::F; r.dout = HID;
  } else if (f < S::MB * S::KS0 + a.n_hidden * S::MB * S::KSH) {
    const int g = f - S::MB * S::KS0;
    r.layer = 1 + g / (S::MB * S::KSH);
    const int q = g % (S::MB * S::KSH);
    mb = q / S::KSH; r.s = q % S::KSH; r.din = HID; r.dout = HID;
  } else {
    r.layer = a.n_hidden + 1; mb = 0; r.s = f - S::MB * S::KS0 - a.n_hidden * S::MB * S::KSH;
    r.din = HID; r.dout = a.out_dim;
  }
  r.woff = r.layer == 0 ? 0 : (size_t)HID * (S::F + 1) + (size_t)(r.layer - 1) * HID * (HID + 1);
  r.row = mb * 32 + (lane & 31);
  r.h = lane >> 5;
  return r;
}

// Weight unit that element e of a lane-slice holds (layer 0 reads the
// features in order; later layers read the previous layer's accumulator
// order, see sigma16).
template <int NL, int CH, int PE, int HID>
__device__ __forceinline__ int slice_unit(const SliceSource<NL, CH, PE, HID> &r, int e) {
  const int kap = 8 * r.h + e;
  return 16 * r.s + (r.layer == 0 ? kap : sigma16(kap));
}

// Copies decoder `dec` into the LDS image, re-arranged into A fragments; all
// threads of the workgroup take part; the caller brackets it with barriers.
// The decoder block is read through a raw buffer resource: 32-bit offsets, and
// a weight outside its layer (padding rows and columns) gets an offset past
// the block, which the hardware returns as zero.  A thread issues the loads of
// kStageSlices lane-slices (8 weights each) back to back, so staging costs one
// memory round trip per kStageSlices * THREADS lane-slices.
constexpr int kStageSlices = 2;
constexpr uint32_t kPastBlock = 0xFFFFFF00u;  // byte offset past any decoder block

template <int NL, int CH, int PE, int HID, int THREADS>
__device__ void stage_decoder(const DecodeArgs &a, uint32_t dec, uint32_t *lds) {
  const Image im = image_of<NL, CH, PE, HID>(a.n_hidden);
  const uint16_t *p = a.params + (size_t)dec * (size_t)a.dec_stride;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)p, 0, (int)(a.dec_stride * 2), 0x00020000);
  const int n_layers = a.n_hidden + 2;
  const int n_slices = im.n_frags * kWave;
  for (int base = threadIdx.x; base < n_slices; base += kStageSlices * THREADS) {
    uint32_t v[kStageSlices][8];
#pragma unroll
    for (int i = 0; i < kStageSlices; ++i) {
      const int lf = base + i * THREADS;
      const SliceSource<NL, CH, PE, HID> r = slice_source<NL, CH, PE, HID>(a, lf < n_slices ? lf : 0);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int unit = slice_unit(r, e);
        const bool in = r.row < r.dout && unit < r.din;
        const uint32_t off = in ? (uint32_t)(r.woff + (size_t)r.row * r.din + unit) * 2u : kPastBlock;
        v[i][e] = __builtin_amdgcn_raw_buffer_load_b16(rsrc, off, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < kStageSlices; ++i) {
      const int lf = base + i * THREADS;
      if (lf < n_slices) {
        const u32x4 packed = {v[i][0] | v[i][1] << 16, v[i][2] | v[i][3] << 16,
                              v[i][4] | v[i][5] << 16, v[i][6] | v[i][7] << 16};
        *(u32x4 *)(lds + (size_t)(lf / kWave) * 256 + (lf % kWave) * 4) = packed;
      }
    }
  }
  // biases, converted to fp32; rows past the layer width read zero, as above
  using S = Shape<NL, CH, PE, HID>;
  float *bias = (float *)(lds + im.bias_off);
  for (int i = threadIdx.x; i < im.n_bias; i += THREADS) {
    int layer, row, dout;
    if (i < HID * (1 + a.n_hidden)) {
      layer = i / HID; row = i % HID; dout = HID;
    } else {
      layer = n_layers - 1; row = i - HID * (1 + a.n_hidden); dout = a.out_dim;
    }
    const size_t off =
        layer == 0 ? 0 : (size_t)HID * (S::F + 1) + (size_t)(layer - 1) * HID * (HID + 1);
    const int din = layer == 0 ? S::F : HID;
    const uint32_t boff = row < dout ? (uint32_t)(off + (size_t)dout * din + row) * 2u : kPastBlock;
    const uint16_t hb = __builtin_amdgcn_raw_buffer_load_b16(rsrc, boff, 0, 0);
    const float v = (float)__builtin_bit_cast(_Float16, hb);
    bias[i] = layer == n_layers - 1 ? v * -kLog2e : v;
  }
}

// 16 bias values of output block `mb` of a layer, in accumulator order.
__device__ __forceinline__ floatx16 bias_frag(const float *bias_layer, int mb) {
  const int h = lane_id() >> 5;
  floatx16 c;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const floatx4 v = *(const floatx4 *)(bias_layer + mb * 32 + 8 * g + 4 * h);
    c[4 * g + 0] = v[0];
    c[4 * g + 1] = v[1];
    c[4 * g + 2] = v[2];
    c[4 * g + 3] = v[3];
  }
  return c;
}

__device__ __forceinline__ half8 a_frag(const uint32_t *lds, int f) {
  return as_half8(*(const u32x4 *)(lds + (size_t)f * 256 + lane_id() * 4));
}

// Positional encoding of the query's texture coordinate, PE / 4 octaves k:
// sin(2^k pi u), cos(2^k pi u), sin(2^k pi v), cos(2^k pi v), appended after
// the latent features as fp16 pairs (sin, cos).  v_sin_f32 / v_cos_f32 take
// the angle in turns: 2^k pi u is 2^(k-1) u turns, reduced to [0, 1) first
// (exact in fp32) so any finite coordinate stays inside the instructions'
// input range.
template <int PE>
__device__ __forceinline__ void pos_encoding(float u, float v, uint32_t *xo) {
#pragma unroll
  for (int k = 0; k < PE / 4; ++k) {
    const float scale = k == 0 ? 0.5f : (float)(1 << (k - 1));
    const float tu = __builtin_amdgcn_fractf(u * scale), tv = __builtin_amdgcn_fractf(v * scale);
    xo[2 * k] = pack_half2(__builtin_amdgcn_sinf(tu), __builtin_amdgcn_cosf(tu));
    xo[2 * k + 1] = pack_half2(__builtin_amdgcn_sinf(tv), __builtin_amdgcn_cosf(tv));
  }
}

// -------------------------------------------------------------------- gather

struct Query {
  uint32_t q;      // query index (only meaningful when valid)
  bool valid;
  uint32_t tex;
  float u, v, mip;
};

// The 2x2 texels of one level around a query and its position between them.
// fetch_level clamps the lower tap to [0, res - 2] and the weight to [0, 1]:
// for res >= 2 this is exactly bilinear filtering with both taps clamped to
// the edge, and it puts the right-hand tap 2*CH bytes after the left one (an
// immediate offset) and the lower row res*CH values further on.  Any finite
// or NaN coordinate keeps every tap inside the level.
template <int CH>
struct LevelTaps {
  static constexpr int NV = CH / 8;  // 16-byte vectors per texel
  u32x4 t00[NV], t10[NV], t01[NV], t11[NV];
  float fx, fy;
};

template <int CH>
__device__ __forceinline__ void fetch_level(const uint16_t *tex, uint32_t level_off, int res,
                                            float resf, float u, float v, LevelTaps<CH> &L) {
  const float x = __builtin_fmaf(u, resf, -0.5f), y = __builtin_fmaf(v, resf, -0.5f);
  const float hi = resf - 2.f;
  // med3 clamps (a NaN coordinate converts to index 0 below)
  const float x0 = __builtin_amdgcn_fmed3f(__builtin_floorf(x), 0.f, hi);
  const float y0 = __builtin_amdgcn_fmed3f(__builtin_floorf(y), 0.f, hi);
  L.fx = __builtin_amdgcn_fmed3f(x - x0, 0.f, 1.f);
  L.fy = __builtin_amdgcn_fmed3f(y - y0, 0.f, 1.f);
  const uint32_t idx = level_off + ((uint32_t)y0 * (uint32_t)res + (uint32_t)x0) * CH;
  const u32x4 *r0 = (const u32x4 *)(tex + idx);
  const u32x4 *r1 = (const u32x4 *)(tex + idx + (uint32_t)res * CH);
#pragma unroll
  for (int i = 0; i < LevelTaps<CH>::NV; ++i) {
    L.t00[i] = r0[i];
    L.t10[i] = r0[LevelTaps<CH>::NV + i];
    L.t01[i] = r1[i];
    L.t11[i] = r1[LevelTaps<CH>::NV + i];
  }
}

// Bilinear weights applied in packed fp16: each operation handles a channel
// pair, the four weights are rounded to fp16 and every product and sum is an
// fp16 operation (one v_pk_mul_f16 and three v_pk_fma_f16 per pair), half the
// instructions of an fp32 interpolation; its rounding stays well inside the
// decode tolerance.  Writes CH / 2 packed pairs, channel order.
__device__ __forceinline__ half2v as_h2(uint32_t v) { return __builtin_bit_cast(half2v, v); }

template <int CH>
__device__ __forceinline__ void interp_level_h2(const LevelTaps<CH> &L, uint32_t *xo) {
  const float gx = 1.f - L.fx, gy = 1.f - L.fy;
  const float2v w0 = {gx * gy, L.fx * gy}, w1 = {gx * L.fy, L.fx * L.fy};
  const half2v h0 = __builtin_convertvector(w0, half2v), h1 = __builtin_convertvector(w1, half2v);
  const half2v w00 = {h0[0], h0[0]}, w10 = {h0[1], h0[1]};
  const half2v w01 = {h1[0], h1[0]}, w11 = {h1[1], h1[1]};
#pragma unroll
  for (int i = 0; i < LevelTaps<CH>::NV; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      half2v r = as_h2(L.t00[i][e]) * w00;
      r = __builtin_elementwise_fma(as_h2(L.t10[i][e]), w10, r);
      r = __builtin_elementwise_fma(as_h2(L.t01[i][e]), w01, r);
      r = __builtin_elementwise_fma(as_h2(L.t11[i][e]), w11, r);
      xo[4 * i + e] = __builtin_bit_cast(uint32_t, r);
    }
  }
}

// v[k] for a per-lane level index k < NL, as a chain of selects (no scratch).
template <int NL, typename T>
__device__ __forceinline__ T pick(const T (&v)[NTC_MAX_LEVELS], int k) {
  T r = v[0];
#pragma unroll
  for (int i = 1; i < NL; ++i) r = k == i ? v[i] : r;
  return r;
}

// Feature vector of the lane's query, packed as fp16 pairs: x[c/2] holds
// features c and c+1; slot l occupies features [l*CH, (l+1)*CH).
template <int NL, int CH, int PE, bool MIP>
__device__ __forceinline__ void gather(const DecodeArgs &a, const Query &qq,
                                       uint32_t (&x)[(NL * CH + PE) / 2]) {
  if constexpr (PE > 0) pos_encoding<PE>(qq.u, qq.v, x + NL * CH / 2);
  const uint16_t *tex = a.latents + (size_t)qq.tex * (size_t)a.tex_stride;
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    if (!MIP) {
      LevelTaps<CH> L;
      fetch_level<CH>(tex, a.level_off[l], a.res[l], a.resf[l], qq.u, qq.v, L);
      interp_level_h2<CH>(L, x + l * CH / 2);
    } else {
      // Each level is interpolated in packed fp16 like the plain path, and the
      // blend f0 + t (f1 - f0) is one packed subtract and one packed fma per
      // pair (max-abs error of the decoded channels 9.7e-4 against 7.1e-4 for
      // an fp32 interpolation, 4 % less decode time on Wide + trilinear).  The
      // second level is fetched only when some lane of the wave blends: the
      // coarsest slot never does (its level of detail is always NL - 1).
      const float m = __builtin_fminf(__builtin_fmaxf(qq.mip, 0.f), (float)(NL - 1));
      const float lod = __builtin_fmaxf((float)l, m);
      const int k0 = (int)__builtin_floorf(lod);
      const int k1 = min(k0 + 1, NL - 1);
      const float t = lod - (float)k0;
      LevelTaps<CH> L0;
      fetch_level<CH>(tex, pick<NL>(a.level_off, k0), pick<NL>(a.res, k0), pick<NL>(a.resf, k0),
                      qq.u, qq.v, L0);
      interp_level_h2<CH>(L0, x + l * CH / 2);
      if (__builtin_amdgcn_ballot_w64(t != 0.f)) {
        LevelTaps<CH> L1;
        fetch_level<CH>(tex, pick<NL>(a.level_off, k1), pick<NL>(a.res, k1), pick<NL>(a.resf, k1),
                        qq.u, qq.v, L1);
        uint32_t f1[CH / 2];
        interp_level_h2<CH>(L1, f1);
        const _Float16 th = (_Float16)t;
        const half2v t2 = {th, th};
#pragma unroll
        for (int c = 0; c < CH / 2; ++c) {
          const half2v a0 = as_h2(x[l * CH / 2 + c]);
          x[l * CH / 2 + c] =
              __builtin_bit_cast(uint32_t, __builtin_elementwise_fma(t2, as_h2(f1[c]) - a0, a0));
        }
      }
    }
  }
}

// Taps of all levels of one query, for the pipelined path without mip.
template <int NL, int CH>
struct TileTaps {
  LevelTaps<CH> lv[NL];
};

template <int NL, int CH>
__device__ __forceinline__ void fetch_taps(const DecodeArgs &a, const Query &qq,
                                           TileTaps<NL, CH> &T) {
  const uint16_t *tex = a.latents + (size_t)qq.tex * (size_t)a.tex_stride;
#pragma unroll
  for (int l = 0; l < NL; ++l)
    fetch_level<CH>(tex, a.level_off[l], a.res[l], a.resf[l], qq.u, qq.v, T.lv[l]);
}

template <int NL, int CH, int PE>
__device__ __forceinline__ void interp_taps(const TileTaps<NL, CH> &T,
                                            uint32_t (&x)[(NL * CH + PE) / 2]) {
#pragma unroll
  for (int l = 0; l < NL; ++l) interp_level_h2<CH>(T.lv[l], x + l * CH / 2);
}

// Exchange halves between lane l and lane l ^ 32 so that, per 16-wide K-slice,
// b0 holds the slice for column block 0 (queries of lanes 0..31) and b1 for
// column block 1 (queries of lanes 32..63), each lane holding K-values 8h..8h+7.
// v_permlane32_swap(lo, hi) moves lanes 0..31 of hi into lanes 32..63 of lo and
// lanes 32..63 of lo into lanes 0..31 of hi: afterwards lo is the column-block-0
// operand and hi the column-block-1 operand in every lane.
template <int KS>
__device__ __forceinline__ void to_b_operands(const uint32_t (&x)[KS * 8], half8 (&b0)[KS],
                                              half8 (&b1)[KS]) {
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    u32x4 v0, v1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto r = __builtin_amdgcn_permlane32_swap(x[8 * s + i], x[8 * s + 4 + i], false,
                                                      false);
      v0[i] = r[0];
      v1[i] = r[1];
    }
    b0[s] = as_half8(v0);
    b1[s] = as_half8(v1);
  }
}

// fp16 pair (round to nearest even) with ReLU applied on the packed halves: a
// negative half has its sign bit set, so a signed 16-bit max with 0 zeroes it.
// Rounding commutes with ReLU, so this equals rounding ReLU(x).
__device__ __forceinline__ uint32_t relu_pack2(float a, float b) {
  const short2v h = __builtin_bit_cast(short2v, pack_half2(a, b));
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(h, short2v{0, 0}));
}

// fp16 pair with LeakyReLU max(x, slope * x) (0 < slope < 1) applied on the
// packed halves, after rounding.
__device__ __forceinline__ uint32_t leaky_pack2(float a, float b, uint32_t slope_h2) {
  const half2v h = __builtin_bit_cast(half2v, pack_half2(a, b));
  const half2v s = __builtin_bit_cast(half2v, slope_h2);
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(h, h * s));
}

// Hidden activation + fp16 of one 32-row output block -> two K-slices of the
// next layer.  LEAKY selects LeakyReLU; it is a template parameter so that the
// layer's MFMAs and conversions stay in one basic block.
template <bool LEAKY>
__device__ __forceinline__ void relu_pack(const floatx16 &acc, half8 &s0, half8 &s1,
                                          uint32_t slope_h2) {
  u32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (LEAKY) {
      a[i] = leaky_pack2(acc[2 * i], acc[2 * i + 1], slope_h2);
      b[i] = leaky_pack2(acc[8 + 2 * i], acc[8 + 2 * i + 1], slope_h2);
    } else {
      a[i] = relu_pack2(acc[2 * i], acc[2 * i + 1]);
      b[i] = relu_pack2(acc[8 + 2 * i], acc[8 + 2 * i + 1]);
    }
  }
  s0 = as_half8(a);
  s1 = as_half8(b);
}

// 1 / (1 + exp(-(z + b))) with nb = -b * log2(e).
__device__ __forceinline__ float sigmoid(float z, float nb) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(__builtin_fmaf(z, -kLog2e, nb)));
}

// Runs the staged decoder on the tile's features; returns the output layer's
// accumulators (sigmoid applied) for the two column blocks.
template <int NL, int CH, int PE, int HID, int NH, bool LEAKY>
__device__ __forceinline__ void run_mlp(const uint32_t *lds,
                                        const half8 (&xb0)[(NL * CH + PE) / 16],
                                        const half8 (&xb1)[(NL * CH + PE) / 16], floatx16 &y0,
                                        floatx16 &y1, uint32_t slope_h2) {
  using S = Shape<NL, CH, PE, HID>;
  const float *bias = (const float *)(lds) + image_of<NL, CH, PE, HID>(NH).bias_off;
  half8 h0[S::KSH], h1[S::KSH];
  // layer 0: F -> HID
#pragma unroll
  for (int mb = 0; mb < S::MB; ++mb) {
    floatx16 c0 = bias_frag(bias, mb), c1 = c0;
#pragma unroll
    for (int s = 0; s < S::KS0; ++s) {
      const half8 w = a_frag(lds, mb * S::KS0 + s);
      c0 = mfma(w, xb0[s], c0);
      c1 = mfma(w, xb1[s], c1);
    }
    relu_pack<LEAKY>(c0, h0[2 * mb], h0[2 * mb + 1], slope_h2);
    relu_pack<LEAKY>(c1, h1[2 * mb], h1[2 * mb + 1], slope_h2);
  }
  int frag = S::MB * S::KS0;
  const float *bl = bias + HID;
  // hidden -> hidden
#pragma unroll
  for (int layer = 0; layer < NH; ++layer) {
    half8 n0[S::KSH], n1[S::KSH];
#pragma unroll
    for (int mb = 0; mb < S::MB; ++mb) {
      floatx16 c0 = bias_frag(bl, mb), c1 = c0;
#pragma unroll
      for (int s = 0; s < S::KSH; ++s) {
        const half8 w = a_frag(lds, frag + mb * S::KSH + s);
        c0 = mfma(w, h0[s], c0);
        c1 = mfma(w, h1[s], c1);
      }
      relu_pack<LEAKY>(c0, n0[2 * mb], n0[2 * mb + 1], slope_h2);
      relu_pack<LEAKY>(c1, n1[2 * mb], n1[2 * mb + 1], slope_h2);
    }
#pragma unroll
    for (int s = 0; s < S::KSH; ++s) {
      h0[s] = n0[s];
      h1[s] = n1[s];
    }
    frag += S::MB * S::KSH;
    bl += HID;
  }
  // output layer: HID -> out (rows padded to 32 with zero weights).  Its
  // accumulators start at zero (an inline constant); the bias is added by the
  // sigmoid, which needs one multiply-add per value anyway.
  floatx16 c0 = {}, c1 = {};
#pragma unroll
  for (int s = 0; s < S::KSH; ++s) {
    const half8 w = a_frag(lds, frag + s);
    c0 = mfma(w, h0[s], c0);
    c1 = mfma(w, h1[s], c1);
  }
  y0 = c0;
  y1 = c1;
}

// Output-layer biases of this lane's rows 4h..4h+3, pre-scaled by -log2(e)
// when the decoder is staged (the sigmoid's exponent is then one fma).
template <int NL, int CH, int PE, int HID, int NH>
__device__ __forceinline__ floatx4 out_bias(const uint32_t *lds, int first_row) {
  const float *b = (const float *)(lds) + image_of<NL, CH, PE, HID>(NH).bias_off + HID * (1 + NH);
  return *(const floatx4 *)(b + first_row + 4 * (lane_id() >> 5));
}

// Raw buffer resource over the output rows: a store whose byte offset lies past
// the range is dropped by the hardware, so masked lanes need no branch and
// every path issues the same number of stores.  The output is at most
// kMaxOutBytes, so the drop offset (and the few 16-byte steps added to it) is
// past the range and offset + 16 never wraps around 32 bits.
constexpr uint32_t kDropOffset = 0xFFFFFF00u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t out_resource(const DecodeArgs &a) {
  const uint32_t bytes = a.n * (uint32_t)a.out_dim * (a.out_f16 ? 2u : 4u);  // <= kMaxOutBytes
  return __builtin_amdgcn_make_buffer_rsrc(a.out, 0, (int)bytes, 0x00020000);
}

// How a column block's rows reach memory: for an output width of 4 or 8, one
// fp32 (or fp16) run of the 4 rows each lane holds; for a width of 3 (RGB rows,
// the Sec. 4 setup) the lanes holding rows 0..3 store rows 0..2 (fp32: one
// 12-byte store; fp16: a 4-byte and a 2-byte store); for any other width up to
// 16, one store per row.
enum StoreMode { kStoreF32x4 = 0, kStoreF16x4 = 1, kStoreEach = 2, kStoreF32x3 = 3,
                 kStoreF16x3 = 4 };

// Store instructions per 32-query column block; fixed for a mode, so the wait
// counts of the software pipeline do not depend on the data.
template <int STORE>
constexpr int kStoresPerBlock = STORE == kStoreEach ? 8 : STORE == kStoreF16x3 ? 2 : 1;

// Decoded values this lane stores for one 32-query column block: rows 4h..4h+3
// (lo) and 8+4h..8+4h+3 (hi) of the query in its column, after the sigmoid, as
// fp32 bits.  hi exists only in the per-row mode and is computed only when the
// width reaches it (otherwise its stores are dropped and its value is unused).
struct OutRows {
  u32x4 lo, hi;
};

// Scaled output biases (see out_bias) of the lane's lo and hi rows.
struct OutBias {
  floatx4 lo, hi;
};

template <int NL, int CH, int PE, int HID, int NH, int STORE>
__device__ __forceinline__ OutBias load_out_bias(const uint32_t *lds, int out_dim) {
  OutBias b;
  b.lo = out_bias<NL, CH, PE, HID, NH>(lds, 0);
  b.hi = STORE == kStoreEach && out_dim > 8 ? out_bias<NL, CH, PE, HID, NH>(lds, 8) : b.lo;
  return b;
}

template <int STORE>
__device__ __forceinline__ OutRows finish_rows(const floatx16 &z, const OutBias &b, int out_dim) {
  OutRows r;
  r.hi = __builtin_nondeterministic_value(r.hi);
#pragma unroll
  for (int i = 0; i < 4; ++i) r.lo[i] = __builtin_bit_cast(uint32_t, sigmoid(z[i], b.lo[i]));
  if (STORE == kStoreEach && out_dim > 8) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      r.hi[i] = __builtin_bit_cast(uint32_t, sigmoid(z[4 + i], b.hi[i]));
  }
  return r;
}

// Cache policy of the output stores: non-temporal.  The decoded rows are
// written once and not read again by the kernel; streaming them past the L2
// keeps the L2 for the latent texels that neighbouring queries share (about
// 13 % less decode time on the 4K clustered frame than default stores).
constexpr int kOutPolicy = 2;  // nt

// Every store of the mode is always issued (rows past the width, and masked
// lanes, get the drop offset), so the number of stores never depends on the
// data or the width.
template <int STORE>
__device__ __forceinline__ void store_rows(__amdgpu_buffer_rsrc_t out, int out_dim, uint32_t q,
                                           bool ok, const OutRows &r, uint32_t out_f16) {
  const int h = lane_id() >> 5;
  const int r0 = 4 * h;
  if constexpr (STORE == kStoreF32x4) {
    const uint32_t off = ok && r0 < out_dim ? (q * (uint32_t)out_dim + (uint32_t)r0) * 4u
                                            : kDropOffset;
    __builtin_amdgcn_raw_buffer_store_b128(r.lo, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF16x4) {
    const uint32_t off = ok && r0 < out_dim ? (q * (uint32_t)out_dim + (uint32_t)r0) * 2u
                                            : kDropOffset;
    const float4 lo = __builtin_bit_cast(float4, r.lo);
    const u32x2 lo16 = {pack_half2(lo.x, lo.y), pack_half2(lo.z, lo.w)};
    __builtin_amdgcn_raw_buffer_store_b64(lo16, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF32x3) {
    const uint32_t off = ok && h == 0 ? q * 12u : kDropOffset;
    const u32x3 v = {r.lo[0], r.lo[1], r.lo[2]};
    __builtin_amdgcn_raw_buffer_store_b96(v, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF16x3) {
    // the row's 6 bytes start at 6q: for even q the pair (0, 1) is 4-byte
    // aligned and row 2 follows; for odd q row 0 comes first, then the
    // aligned pair (1, 2)
    const float4 lo = __builtin_bit_cast(float4, r.lo);
    const bool even = (q & 1u) == 0;
    const uint32_t base = q * 6u;
    const bool st = ok && h == 0;
    const uint32_t off32 = st ? (even ? base : base + 2u) : kDropOffset;
    const uint32_t off16 = st ? (even ? base + 4u : base) : kDropOffset;
    const uint32_t pair = even ? pack_half2(lo.x, lo.y) : pack_half2(lo.y, lo.z);
    const _Float16 single = (_Float16)(even ? lo.z : lo.x);
    __builtin_amdgcn_raw_buffer_store_b32(pair, out, off32, 0, kOutPolicy);
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, single), out, off16, 0,
                                           kOutPolicy);
  } else {
    const uint32_t row = q * (uint32_t)out_dim;
    const uint32_t es = out_f16 ? 2u : 4u;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rr = 8 * g + 4 * h + i;
        const uint32_t off = ok && rr < out_dim ? (row + (uint32_t)rr) * es : kDropOffset;
        const uint32_t v = g ? r.hi[i] : r.lo[i];
        if (out_f16) {
          const _Float16 f = (_Float16)__builtin_bit_cast(float, v);
          __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, f), out, off, 0,
                                                 kOutPolicy);
        } else {
          __builtin_amdgcn_raw_buffer_store_b32(v, out, off, 0, kOutPolicy);
        }
      }
    }
  }
}

// Column block 0 holds the queries of lanes 0..31, block 1 those of lanes
// 32..63; a lane of half h stores, for each block, the query of lane
// (block * 32 + lane % 32): its own in block h, its partner's in the other.
// One v_permlane32_swap of (q, q) gives both: its first result holds the
// lower half's values in both halves, its second the upper half's.
template <int STORE>
__device__ __forceinline__ void store_tile(__amdgpu_buffer_rsrc_t out, int out_dim, uint32_t q,
                                           bool ok, const OutRows &b0, const OutRows &b1,
                                           uint32_t out_f16) {
  const uint32_t okw = ok ? 1u : 0u;
  const auto qs = __builtin_amdgcn_permlane32_swap(q, q, false, false);
  const auto oks = __builtin_amdgcn_permlane32_swap(okw, okw, false, false);
  store_rows<STORE>(out, out_dim, qs[0], oks[0] != 0, b0, out_f16);
  store_rows<STORE>(out, out_dim, qs[1], oks[1] != 0, b1, out_f16);
}

// Query data of a slot.  The loads are unconditional (a slot without a valid
// query reads query 0), so every wave issues the same loads on every path and
// the compiler's waits stay exact.  The texture id is checked by validate(),
// once the tile that owns the query is about to use it.
template <int NL, bool MIP>
__device__ __forceinline__ Query load_query(const DecodeArgs &a, uint32_t q, bool in_range) {
  Query r;
  r.q = q;
  r.valid = in_range && q < a.n;
  const uint32_t qs = r.valid ? q : 0u;
  r.tex = a.tex_id[qs];
  const float2 uv = ((const float2 *)a.uv)[qs];
  r.u = uv.x;
  r.v = uv.y;
  r.mip = MIP ? a.mip[qs] : 0.f;
  return r;
}

// Marks a query with an out-of-range texture invalid and points it at texture
// 0, so its (discarded) gather stays inside the latents.
__device__ __forceinline__ Query validate(const DecodeArgs &a, Query r) {
  r.valid = r.valid && r.tex < (uint32_t)a.n_textures;
  if (!r.valid) r.tex = 0;
  return r;
}

// ------------------------------------------------------------------- kernels

typedef const __attribute__((address_space(4))) uint32_t *const_u32p;

// Wave-uniform read of the bin offsets through the constant address space, so
// it becomes a scalar load that does not enter the vector-memory counter.
__device__ __forceinline__ uint32_t bin_off(const DecodeArgs &a, uint32_t i) {
  return ((const_u32p)a.bin_offset)[i];
}

// A group of up to WAVES consecutive tiles of one bin: tiles [t, t + n) of bin
// d, whose tiles end at be; r counts the groups of a weighted sequence.  n == 0
// marks the end of a workgroup's range.
struct Group {
  uint32_t t, n, d, be;
  uint32_t r = 0;
};

template <int WAVES>
__device__ __forceinline__ Group group_at(const DecodeArgs &a, uint32_t t, uint32_t d,
                                          uint32_t be, uint32_t D, uint32_t t_end) {
  while (t >= be && d + 1 < D) {  // next non-empty bin
    ++d;
    be = bin_off(a, d + 1) / kWave;
  }
  const uint32_t n =
      (t >= be || t >= t_end) ? 0u : min(min((uint32_t)WAVES, be - t), t_end - t);
  return Group{t, n, d, be};
}

template <int WAVES>
__device__ __forceinline__ Group next_group(const DecodeArgs &a, const Group &g, uint32_t D,
                                            uint32_t t_end) {
  return g.n ? group_at<WAVES>(a, g.t + g.n, g.d, g.be, D, t_end) : g;
}

// Weighted groups: after every kRounds groups of up to WAVES tiles, one of up
// to WAVES / 2 tiles, for the first half of the waves only, so that the first
// half takes kRounds + 1 tiles for every kRounds of the second.  Waves w and
// w + WAVES / 2 of a workgroup share a SIMD, which issues the older wave, w,
// first.  Used by the binned decode of 128-wide decoders (2.64 -> 2.58 ms on
// the 4-sample trilinear 4K frame); with 64-wide ones it gained nothing on the
// 4K clustered frame and cost 2-4 % with positional encoding.
constexpr uint32_t kRounds = 6;

template <int WAVES>
__device__ __forceinline__ Group wgroup_at(const DecodeArgs &a, uint32_t t, uint32_t d,
                                           uint32_t be, uint32_t D, uint32_t t_end, uint32_t r) {
  Group g = group_at<WAVES>(a, t, d, be, D, t_end);
  if (r == kRounds) g.n = min(g.n, (uint32_t)WAVES / 2);
  g.r = r;
  return g;
}

template <int WAVES>
__device__ __forceinline__ Group next_wgroup(const DecodeArgs &a, const Group &g, uint32_t D,
                                             uint32_t t_end) {
  return g.n ? wgroup_at<WAVES>(a, g.t + g.n, g.d, g.be, D, t_end, g.r == kRounds ? 0u : g.r + 1)
             : g;
}

// Waves per workgroup.  The staged decoder is shared by a workgroup's waves.
// Binned kernels use 8 waves: one LDS image then serves twice as many tiles
// (about 3 % less decode time than 4-wave workgroups on the 4K clustered frame
// with 64-wide decoders), and a 128-wide decoder's image (about 86 KB for
// 48-128-128-128-8) allows only one workgroup per CU anyway.  Stream kernels
// with 64-wide decoders keep 4 waves: a workgroup restages every decoder
// present in its group of tiles, and a group of 8 tiles holds more of them
// (7 % more time with one decoder per texture).
template <int HID, bool BINNED>
constexpr int kWaves = BINNED || HID > 64 ? 8 : 4;
template <int HID, bool BINNED>
constexpr int kThreads = kWaves<HID, BINNED> * kWave;
// Minimum waves per SIMD the register allocation must allow (the second
// argument of __launch_bounds__): 4 for the 64-wide stream kernels (<= 128
// VGPRs), 2 for the 64-wide binned kernels and 1 for 128-wide decoders.  The
// binned instantiation of the clustered workload takes 112 VGPRs (4 waves per
// SIMD); asking for 4 there makes the fp16-output and mip-blending
// instantiations spill.
template <int HID, bool BINNED>
constexpr int kMinBlocks = HID > 64 ? 1 : 16 / kWaves<HID, BINNED>;

template <int NL, int CH, int PE, int HID, int NH, bool MIP, int STORE, bool LEAKY>
__global__ void __launch_bounds__((kThreads<HID, true>), (kMinBlocks<HID, true>))
decode_binned(const DecodeArgs a) {
  constexpr int WAVES = kWaves<HID, true>;
  using S = Shape<NL, CH, PE, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t D = (uint32_t)a.n_decoders;
  const __amdgpu_buffer_rsrc_t out_rsrc = out_resource(a);
  // tiles of the permutation; never more than the buffer holds
  const uint64_t slots = min((uint64_t)bin_off(a, D), a.perm_capacity);
  const uint32_t total_tiles = (uint32_t)(slots / kWave);
  // This workgroup's contiguous range of tiles, in workgroups numbered XCD by
  // XCD.  Equal ranges, or with a.split (two workgroups per CU, the grid a
  // multiple of 16) twice the tiles for the first workgroup dispatched to each
  // CU (blockIdx < gridDim / 2): the SIMDs issue the older waves first, so two
  // co-resident workgroups with equal work finish a third apart and the second
  // runs its last third on half the waves.
  uint32_t t, t_end;
  if (a.split) {
    const uint32_t per_xcd = gridDim.x / 8, half = per_xcd / 2;
    const uint32_t xcd = blockIdx.x % 8, j = blockIdx.x / 8;  // j < half: first on its CU
    const uint64_t w0 = (uint64_t)xcd * half * 3 + (j < half ? 2 * j : 2 * half + (j - half));
    const uint64_t w1 = w0 + (j < half ? 2 : 1);
    const uint64_t W = (uint64_t)gridDim.x / 2 * 3;
    t = (uint32_t)(total_tiles * w0 / W);
    t_end = (uint32_t)(total_tiles * w1 / W);
  } else {
    const uint32_t per = (total_tiles + gridDim.x - 1) / gridDim.x;
    t = xcd_local_block(blockIdx.x, gridDim.x) * per;
    t_end = min(t + per, total_tiles);
  }
  if (t >= t_end) return;
  // bin holding slot 64 t: the last d with bin_offset[d] <= 64 t
  uint32_t lo = 0, hi = D;  // invariant: bin_offset[lo] <= 64 t < bin_offset[hi]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (bin_off(a, mid) <= t * kWave) lo = mid; else hi = mid;
  }
  // Tiles go in groups of consecutive tiles of one bin (weighted for 128-wide
  // decoders), tile t + w to wave w; every wave walks the same (uniform)
  // sequence of groups.  A wave without a tile in a group runs it with every
  // lane masked, or, weighted, skips its MLP and stores but still takes part in
  // its staging and prefetches.
  constexpr bool WEIGHTED = HID > 64;
  const uint32_t wu = __builtin_amdgcn_readfirstlane(w);
  auto advance = [&](const Group &g) {
    if constexpr (WEIGHTED) return next_wgroup<WAVES>(a, g, D, t_end);
    else return next_group<WAVES>(a, g, D, t_end);
  };
  Group g0 = group_at<WAVES>(a, t, lo, bin_off(a, lo + 1) / kWave, D, t_end);
  Group g1 = advance(g0);
  Group g2 = advance(g1);
  Group g3 = advance(g2);
  // perm entry of this wave's tile in group g.  The load is unconditional (slot
  // 0 exists whenever there is a tile) and the entry stays raw until it is
  // used, with `has` saying whether the wave has a tile in the group: selecting
  // right after the load would wait for it.
  struct Slot {
    uint32_t raw;
    bool has;
  };
  auto slot_query = [&](const Group &g) -> Slot {
    const bool has = w < g.n;
    return Slot{a.perm[has ? (g.t + w) * kWave + lane : 0u], has};
  };
  // Software pipeline.  Vector-memory operations complete in issue order as
  // far as the wait counter is concerned, and stores count too, so the order
  // at the end of tile k is: taps of tile k+1, query data of tile k+2,
  // permutation entry of tile k+3, and only then the stores of tile k.  Tile
  // k+1 then waits for its taps without waiting for those stores, and every
  // prefetch has a whole tile of work to land.
  auto restage = [&](uint32_t d) {
    __syncthreads();  // every wave is done with the previous decoder
    stage_decoder<NL, CH, PE, HID, kThreads<HID, true>>(a, d, lds);
    __syncthreads();
  };
  const Slot s0 = slot_query(g0);
  Query cur = validate(a, load_query<NL, MIP>(a, s0.raw, s0.has));  // tile 0
  restage(g0.d);
  uint32_t staged = g0.d;
  TileTaps<NL, CH> taps;
  if constexpr (!MIP) fetch_taps<NL, CH>(a, cur, taps);
  __builtin_amdgcn_sched_barrier(0);
  const Slot s1 = slot_query(g1);
  Query q_next = load_query<NL, MIP>(a, s1.raw, s1.has);  // tile 1
  Slot p_next = slot_query(g2);                            // tile 2
  __builtin_amdgcn_sched_barrier(0);
  // As many stores as a loop iteration issues, all past the range (dropped):
  // the loop is entered with the same operations in flight, in the same
  // order, as at its back edge, so the waits at its top need not drain.
  // Distinct offsets keep them from being merged.
#pragma unroll
  for (uint32_t i = 0; i < 2 * kStoresPerBlock<STORE>; ++i)
    __builtin_amdgcn_raw_buffer_store_b32(0u, out_rsrc, kDropOffset + 16u * i, 0, 0);
  // One tile: decode `cur` (taps already in flight), stage the next group's
  // decoder if it changes, fetch the next tile's taps from q_in (its query data),
  // prefetch query data of the tile after from p_in into q_out and the
  // permutation entry of the tile after that into p_out, then store.
  auto tile = [&](const Query &q_in, const Slot &p_in, Query &q_out, Slot &p_out) {
    const bool busy = !WEIGHTED || wu < g0.n;  // this wave has a tile in the group
    OutRows r0, r1;
    if (busy) {
      uint32_t x[S::F / 2];
      if constexpr (MIP)
        gather<NL, CH, PE, MIP>(a, cur, x);
      else {
        interp_taps<NL, CH, PE>(taps, x);
        if constexpr (PE > 0) pos_encoding<PE>(cur.u, cur.v, x + NL * CH / 2);
      }
      half8 xb0[S::KS0], xb1[S::KS0];
      to_b_operands<S::KS0>(x, xb0, xb1);
      floatx16 z0, z1;
      run_mlp<NL, CH, PE, HID, NH, LEAKY>(lds, xb0, xb1, z0, z1, a.slope_h2);
      const OutBias ob = load_out_bias<NL, CH, PE, HID, NH, STORE>(lds, a.out_dim);
      r0 = finish_rows<STORE>(z0, ob, a.out_dim);
      r1 = finish_rows<STORE>(z1, ob, a.out_dim);
    }
    __builtin_amdgcn_sched_barrier(0);
    // The next group's decoder is staged here, between this tile's MLP and the
    // next tile's fetches, so no fetched data is live across the staging.
    if (g1.n && g1.d != staged) {
      restage(g1.d);
      staged = g1.d;
    }
    // next tile: taps, then the prefetches, then this tile's stores
    const Query nxt = validate(a, q_in);
    if constexpr (!MIP) fetch_taps<NL, CH>(a, nxt, taps);
    __builtin_amdgcn_sched_barrier(0);
    q_out = load_query<NL, MIP>(a, p_in.raw, p_in.has);
    p_out = slot_query(g3);
    __builtin_amdgcn_sched_barrier(0);
    if (busy) store_tile<STORE>(out_rsrc, a.out_dim, cur.q, cur.valid, r0, r1, a.out_f16);
    cur = nxt;
    g0 = g1;
    g1 = g2;
    g2 = g3;
    g3 = advance(g3);
  };
  // Unrolled by two with the prefetch registers swapping roles, so a fetched
  // value is never copied between registers (a copy would wait for the fetch).
  Query q_b;
  Slot p_b;
  for (;;) {
    if (!g0.n) break;
    tile(q_next, p_next, q_b, p_b);
    if (!g0.n) break;
    tile(q_b, p_b, q_next, p_next);
  }
}

template <int NL, int CH, int PE, int HID, int NH, bool MIP, int STORE, bool LEAKY>
__global__ void __launch_bounds__((kThreads<HID, false>), (kMinBlocks<HID, false>))
decode_stream(const DecodeArgs a) {
  constexpr int WAVES = kWaves<HID, false>;
  using S = Shape<NL, CH, PE, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  __shared__ uint32_t next_dec[2][WAVES];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  const __amdgpu_buffer_rsrc_t out_rsrc = out_resource(a);
  const uint32_t n_tiles = (a.n + kWave - 1) / kWave;
  const uint32_t n_groups = (n_tiles + WAVES - 1) / WAVES;
  const uint32_t per = (n_groups + gridDim.x - 1) / gridDim.x;
  const uint32_t blk = xcd_local_block(blockIdx.x, gridDim.x);
  const uint32_t g_begin = blk * per, g_end = min(g_begin + per, n_groups);
  uint32_t staged = 0xFFFFFFFFu;
  int parity = 0;
  for (uint32_t g = g_begin; g < g_end; ++g) {
    const uint32_t q = (g * WAVES + w) * kWave + lane;
    const Query qq = validate(a, load_query<NL, MIP>(a, q, true));
    uint32_t dq = 0xFFFFFFFFu;
    bool live = qq.valid;
    if (live) {
      const uint32_t dd = a.tex_to_dec[qq.tex];
      live = dd < (uint32_t)a.n_decoders;
      dq = live ? dd : 0xFFFFFFFFu;
    }
    uint32_t x[S::F / 2];
    gather<NL, CH, PE, MIP>(a, qq, x);
    half8 xb0[S::KS0], xb1[S::KS0];
    to_b_operands<S::KS0>(x, xb0, xb1);
    uint64_t todo = ballot(live);
    for (;;) {
      const uint32_t mine =
          todo ? read_lane(dq, (uint32_t)__builtin_ctzll(todo)) : 0xFFFFFFFFu;
      if (lane == 0) next_dec[parity][w] = mine;
      __syncthreads();
      uint32_t d = next_dec[parity][0];
#pragma unroll
      for (int k = 1; k < WAVES; ++k) d = min(d, next_dec[parity][k]);
      parity ^= 1;
      if (d == 0xFFFFFFFFu) break;
      if (d != staged) {
        stage_decoder<NL, CH, PE, HID, kThreads<HID, false>>(a, d, lds);
        __syncthreads();
        staged = d;
      }
      const bool mine_now = live && dq == d;
      const uint64_t sel = ballot(mine_now);
      if (sel) {
        floatx16 z0, z1;
        run_mlp<NL, CH, PE, HID, NH, LEAKY>(lds, xb0, xb1, z0, z1, a.slope_h2);
        const OutBias ob = load_out_bias<NL, CH, PE, HID, NH, STORE>(lds, a.out_dim);
        store_tile<STORE>(out_rsrc, a.out_dim, q, mine_now,
                          finish_rows<STORE>(z0, ob, a.out_dim),
                          finish_rows<STORE>(z1, ob, a.out_dim), a.out_f16);
        todo &= ~sel;
        live = live && !mine_now;
      }
    }
  }
}

// ---------------------------------------------- stream mode, per-wave decoders
//
// The stream-mode decode for streams over several decoders.  A workgroup takes
// groups of consecutive tiles, one per wave, as decode_stream does.  At every
// kStreamVoteEvery-th group the waves vote: when all of them hold one and the
// same decoder, it is staged once in LDS, and every wave reads it from there
// until a later vote stages another.  Any other decoder a wave holds, the wave
// evaluates on its own, one decoder after another, reading every MFMA A
// fragment straight from that decoder's parameter block through a raw buffer
// (rows past the output width read as zero), with no restaging and no barrier.
// This is the paper's non-shared tensor decoder (Sec. 4.4): a wave pays one
// full MLP pass per decoder it holds.  Used when every decoder block is 16-byte
// aligned (the fragment loads are 16 and 8 bytes).  Restaging the union of a
// group's decoders in LDS, the only mode of decode_stream, makes every wave
// wait for every decoder of the group (on the 4K clustered frame, 16 decoders:
// 1.81 ms against 0.74 ms for per-wave reads); per-wave reads alone are twice
// as slow as one staged copy when waves share a decoder (3.2 ms against 1.6 ms
// on an 8192^2 image).
//
// Fragment (layer, row block mb, K-slice s) of lane (row r = 32 mb + lane % 32,
// half h = lane / 32): layer 0 reads the 8 features 16 s + 8 h .. + 7 of row r
// (one 16-byte load); later layers read units 16 s + 4 h .. + 3 and
// 16 s + 8 + 4 h .. + 3 (two 8-byte loads), the order the previous layer's
// accumulators leave its outputs in (sigma16).

__device__ __forceinline__ half8 load_frag16(__amdgpu_buffer_rsrc_t w, uint32_t off) {
  return as_half8(__builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(w, off, 0, 0)));
}

__device__ __forceinline__ half8 load_frag8x2(__amdgpu_buffer_rsrc_t w, uint32_t off) {
  const u32x2 lo = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(w, off, 0, 0));
  const u32x2 hi = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(w, off + 16u, 0, 0));
  return as_half8(u32x4{lo[0], lo[1], hi[0], hi[1]});
}

// The decoder's biases into this wave's region of LDS (fp32, the image's bias
// layout: the output layer's rows past its width zero and its biases scaled by
// -log2(e)); the wave's own earlier reads of the region precede these writes.
template <int NL, int CH, int PE, int HID>
__device__ __forceinline__ void stage_biases_wave(const DecodeArgs &a,
                                                  __amdgpu_buffer_rsrc_t w, float *bias) {
  using S = Shape<NL, CH, PE, HID>;
  const int n_layers = a.n_hidden + 2;
  const int n_bias = HID * (1 + a.n_hidden) + 32;
  for (int i = lane_id(); i < n_bias; i += kWave) {
    int layer, row, dout;
    if (i < HID * (1 + a.n_hidden)) {
      layer = i / HID; row = i % HID; dout = HID;
    } else {
      layer = n_layers - 1; row = i - HID * (1 + a.n_hidden); dout = a.out_dim;
    }
    const size_t off =
        layer == 0 ? 0 : (size_t)HID * (S::F + 1) + (size_t)(layer - 1) * HID * (HID + 1);
    const int din = layer == 0 ? S::F : HID;
    const uint32_t boff = row < dout ? (uint32_t)(off + (size_t)dout * din + row) * 2u : kPastBlock;
    const float v = (float)__builtin_bit_cast(_Float16, __builtin_amdgcn_raw_buffer_load_b16(w, boff, 0, 0));
    bias[i] = layer == n_layers - 1 ? v * -kLog2e : v;
  }
}

// run_mlp with the A fragments from the decoder block `w` and the biases from
// the wave's LDS region.
template <int NL, int CH, int PE, int HID, int NH, bool LEAKY>
__device__ __forceinline__ void run_mlp_direct(__amdgpu_buffer_rsrc_t w, const float *bias,
                                               int out_dim,
                                               const half8 (&xb0)[(NL * CH + PE) / 16],
                                               const half8 (&xb1)[(NL * CH + PE) / 16],
                                               floatx16 &y0, floatx16 &y1, uint32_t slope_h2) {
  using S = Shape<NL, CH, PE, HID>;
  const uint32_t lr = lane_id() & 31u, h = lane_id() >> 5;
  half8 h0[S::KSH], h1[S::KSH];
  // layer 0: F -> HID
#pragma unroll
  for (int mb = 0; mb < S::MB; ++mb) {
    floatx16 c0 = bias_frag(bias, mb), c1 = c0;
    const uint32_t base = ((mb * 32u + lr) * S::F + 8u * h) * 2u;
#pragma unroll
    for (int s = 0; s < S::KS0; ++s) {
      const half8 wf = load_frag16(w, base + 32u * s);
      c0 = mfma(wf, xb0[s], c0);
      c1 = mfma(wf, xb1[s], c1);
    }
    relu_pack<LEAKY>(c0, h0[2 * mb], h0[2 * mb + 1], slope_h2);
    relu_pack<LEAKY>(c1, h1[2 * mb], h1[2 * mb + 1], slope_h2);
  }
  uint32_t woff = HID * (S::F + 1);
  const float *bl = bias + HID;
  // hidden -> hidden
#pragma unroll
  for (int layer = 0; layer < NH; ++layer) {
    half8 n0[S::KSH], n1[S::KSH];
#pragma unroll
    for (int mb = 0; mb < S::MB; ++mb) {
      floatx16 c0 = bias_frag(bl, mb), c1 = c0;
      const uint32_t base = (woff + (mb * 32u + lr) * HID + 4u * h) * 2u;
#pragma unroll
      for (int s = 0; s < S::KSH; ++s) {
        const half8 wf = load_frag8x2(w, base + 32u * s);
        c0 = mfma(wf, h0[s], c0);
        c1 = mfma(wf, h1[s], c1);
      }
      relu_pack<LEAKY>(c0, n0[2 * mb], n0[2 * mb + 1], slope_h2);
      relu_pack<LEAKY>(c1, n1[2 * mb], n1[2 * mb + 1], slope_h2);
    }
#pragma unroll
    for (int s = 0; s < S::KSH; ++s) {
      h0[s] = n0[s];
      h1[s] = n1[s];
    }
    woff += HID * (HID + 1);
    bl += HID;
  }
  // output layer: rows past the width read zero; bias added by the sigmoid
  floatx16 c0 = {}, c1 = {};
  const uint32_t base = lr < (uint32_t)out_dim ? (woff + lr * HID + 4u * h) * 2u : kPastBlock;
#pragma unroll
  for (int s = 0; s < S::KSH; ++s) {
    const half8 wf = load_frag8x2(w, base + 32u * s);
    c0 = mfma(wf, h0[s], c0);
    c1 = mfma(wf, h1[s], c1);
  }
  y0 = c0;
  y1 = c1;
}

// groups between two votes on the staged decoder of decode_stream_mixed
constexpr uint32_t kStreamVoteEvery = 8;

template <int NL, int CH, int PE, int HID, int NH, bool MIP, int STORE, bool LEAKY>
__global__ void __launch_bounds__((kThreads<HID, false>), (kMinBlocks<HID, false>))
decode_stream_mixed(const DecodeArgs a, uint32_t image_bytes) {
  constexpr int WAVES = kWaves<HID, false>;
  constexpr uint32_t kNone = 0xFFFFFFFFu, kMixed = 0xFFFFFFFEu;
  using S = Shape<NL, CH, PE, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  __shared__ uint32_t wave_dec[2][WAVES];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  constexpr int n_bias = HID * (1 + NH) + 32;
  float *bias = (float *)(lds + image_bytes / 4) + (size_t)w * n_bias;  // this wave's region
  const __amdgpu_buffer_rsrc_t out_rsrc = out_resource(a);
  const uint32_t n_tiles = (a.n + kWave - 1) / kWave;
  const uint32_t n_groups = (n_tiles + WAVES - 1) / WAVES;
  const uint32_t per = (n_groups + gridDim.x - 1) / gridDim.x;
  const uint32_t blk = xcd_local_block(blockIdx.x, gridDim.x);
  const uint32_t g_begin = blk * per, g_end = min(g_begin + per, n_groups);
  const int block_bytes = (int)(a.dec_stride * 2);
  uint32_t staged = kNone;  // the decoder in the shared image; the same in every wave
  int parity = 0;
  for (uint32_t g = g_begin; g < g_end; ++g) {
    const uint32_t q = (g * WAVES + w) * kWave + lane;
    const Query qq = validate(a, load_query<NL, MIP>(a, q, true));
    uint32_t dq = kNone;
    bool live = qq.valid;
    if (live) {
      const uint32_t dd = a.tex_to_dec[qq.tex];
      live = dd < (uint32_t)a.n_decoders;
      dq = live ? dd : kNone;
    }
    uint32_t x[S::F / 2];
    gather<NL, CH, PE, MIP>(a, qq, x);
    half8 xb0[S::KS0], xb1[S::KS0];
    to_b_operands<S::KS0>(x, xb0, xb1);
    uint64_t todo = ballot(live);
    // the wave's one decoder, kMixed for several, kNone for none
    if ((g - g_begin) % kStreamVoteEvery == 0) {
      // the waves vote on the shared copy at every kStreamVoteEvery-th group only and
      // run on their own in between
      const uint32_t first = todo ? read_lane(dq, (uint32_t)__builtin_ctzll(todo)) : kNone;
      const uint32_t mine_one = ballot(live && dq != first) ? kMixed : first;
      if (lane == 0) wave_dec[parity][w] = mine_one;
      __syncthreads();  // also: every wave is done with its reads of the staged image
      uint32_t common = kNone;
      bool agree = true;
#pragma unroll
      for (int k = 0; k < WAVES; ++k) {
        const uint32_t v = wave_dec[parity][k];
        if (v == kNone) continue;
        if (v == kMixed || (common != kNone && v != common)) agree = false;
        common = v;
      }
      parity ^= 1;
      if (agree && common != kNone && common != staged) {
        // every wave of the group holds this one decoder: share one staged copy
        stage_decoder<NL, CH, PE, HID, kThreads<HID, false>>(a, common, lds);
        __syncthreads();
        staged = common;
      }
    }
    while (todo) {
      const uint32_t d = read_lane(dq, (uint32_t)__builtin_ctzll(todo));
      const bool mine = live && dq == d;
      floatx16 z0, z1;
      OutBias ob;
      if (d == staged) {
        run_mlp<NL, CH, PE, HID, NH, LEAKY>(lds, xb0, xb1, z0, z1, a.slope_h2);
        ob = load_out_bias<NL, CH, PE, HID, NH, STORE>(lds, a.out_dim);
      } else {
        const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(a.params + (size_t)d * (size_t)a.dec_stride), 0, block_bytes, 0x00020000);
        stage_biases_wave<NL, CH, PE, HID>(a, wrs, bias);
        run_mlp_direct<NL, CH, PE, HID, NH, LEAKY>(wrs, bias, a.out_dim, xb0, xb1, z0, z1,
                                                   a.slope_h2);
        const float *bo = bias + HID * (1 + NH);  // the output layer's scaled biases
        ob.lo = *(const floatx4 *)(bo + 4 * (lane >> 5));
        ob.hi = STORE == kStoreEach && a.out_dim > 8 ? *(const floatx4 *)(bo + 8 + 4 * (lane >> 5))
                                                     : ob.lo;
      }
      store_tile<STORE>(out_rsrc, a.out_dim, q, mine, finish_rows<STORE>(z0, ob, a.out_dim),
                        finish_rows<STORE>(z1, ob, a.out_dim), a.out_f16);
      todo &= ~ballot(mine);
    }
  }
}

// ------------------------------------------------- non-shared FMA decode
//
// The paper's Non-Shared FMA comparison (Sec. 4.4): every lane evaluates the
// decoder of its own query with vector instructions, so lanes that use
// different decoders share one instruction stream and differ only in the
// addresses their weights come from; the cost does not grow with the number of
// decoders in a wave, unlike the tensor path's one pass per decoder.  Products
// are v_dot2c_f32_f16 (two fp16 products added to an fp32 accumulator), with
// the tensor path's fp16 features and fp16-rounded activations, so both engines
// compute the same function within rounding.
//
// One thread per query, stream order.  Row j of W_i is read by the lane as
// din / 8 16-byte loads from the lane's decoder block (L1/L2-cached).  A layer
// takes its input from registers and writes its output, as fp16 pairs, to the
// thread's own LDS column (word i at i * kBlock + thread): the row loop is a
// runtime loop, and registers cannot be indexed at run time.

__device__ __forceinline__ float dot2(uint32_t w, uint32_t h, float c) {
  return __builtin_amdgcn_fdot2(as_h2(w), as_h2(h), c, false);
}

// fp16 pair of two fp32 values.
__device__ __forceinline__ float2 unpack_half2(uint32_t v) {
  const half2v h = as_h2(v);
  return float2{(float)h[0], (float)h[1]};
}

// Layer din -> dout (dout even) with its input h (fp16 pairs) in registers.
// Hidden layers (OUT = false) write the activated outputs as fp16 pairs, word
// j / 2 of the thread's LDS column; the output layer (OUT = true) writes the
// sigmoid of each output as a float, word j.
template <int DIN, bool OUT>
__device__ __forceinline__ void fma_layer(const uint16_t *W, int dout, const uint32_t (&h)[DIN / 2],
                                          uint32_t *col, bool leaky, uint32_t slope_h2) {
  const uint16_t *b = W + (size_t)dout * DIN;
#pragma unroll 2
  for (int j = 0; j < dout; j += 2) {
    const float2 bj = unpack_half2(*(const uint32_t *)(b + j));
    float acc0 = bj.x, acc1 = bj.y;
    const u32x4 *r0 = (const u32x4 *)(W + (size_t)j * DIN);
    const u32x4 *r1 = (const u32x4 *)(W + (size_t)(j + 1) * DIN);
#pragma unroll
    for (int k = 0; k < DIN / 8; ++k) {
      const u32x4 w0 = r0[k], w1 = r1[k];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc0 = dot2(w0[e], h[4 * k + e], acc0);
        acc1 = dot2(w1[e], h[4 * k + e], acc1);
      }
    }
    if constexpr (OUT) {
      col[j * kBlock] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(acc0 * -kLog2e)));
      col[(j + 1) * kBlock] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(acc1 * -kLog2e)));
    } else {
      col[(j / 2) * kBlock] = leaky ? leaky_pack2(acc0, acc1, slope_h2) : relu_pack2(acc0, acc1);
    }
  }
}

// Words of a thread's LDS column: the widest hidden layer as fp16 pairs, or the
// output row as floats.
template <int HID>
constexpr int kFmaColumn = HID / 2 > 16 ? HID / 2 : 16;

template <int NL, int CH, int PE, int HID, bool MIP>
__global__ void __launch_bounds__(kBlock, 2) decode_fma(const DecodeArgs a) {
  using S = Shape<NL, CH, PE, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  uint32_t *col = lds + threadIdx.x;  // this thread's activations, stride kBlock
  const uint64_t q64 = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
  if (q64 >= a.n) return;
  const uint32_t q = (uint32_t)q64;
  const Query qq = validate(a, load_query<NL, MIP>(a, q, true));
  if (!qq.valid) return;
  const uint32_t d = a.tex_to_dec[qq.tex];
  if (d >= (uint32_t)a.n_decoders) return;
  const uint16_t *p = a.params + (size_t)d * (size_t)a.dec_stride;
  const bool leaky = a.leaky != 0;
  {  // layer 0: F -> HID
    uint32_t x[S::F / 2];
    gather<NL, CH, PE, MIP>(a, qq, x);
    fma_layer<S::F, false>(p, HID, x, col, leaky, a.slope_h2);
    p += (size_t)HID * (S::F + 1);
  }
  // hidden -> hidden, then the output layer (8 or 16 wide, sigmoid)
  for (int l = 0; l <= a.n_hidden; ++l) {
    uint32_t h[HID / 2];
#pragma unroll
    for (int i = 0; i < HID / 2; ++i) h[i] = col[i * kBlock];
    if (l < a.n_hidden) {
      fma_layer<HID, false>(p, HID, h, col, leaky, a.slope_h2);
      p += (size_t)HID * (HID + 1);
    } else {
      fma_layer<HID, true>(p, a.out_dim, h, col, leaky, a.slope_h2);
    }
  }
  const int out_dim = a.out_dim;
  float y[16];
#pragma unroll
  for (int c = 0; c < 16; ++c) y[c] = c < out_dim ? __builtin_bit_cast(float, col[c * kBlock]) : 0.f;
  if (a.out_f16) {
    u32x2 *o = (u32x2 *)((uint16_t *)a.out + (size_t)q * out_dim);
#pragma unroll
    for (int c = 0; c < 16; c += 4)
      if (c < out_dim) o[c / 4] = u32x2{pack_half2(y[c], y[c + 1]), pack_half2(y[c + 2], y[c + 3])};
  } else {
    floatx4 *o = (floatx4 *)((float *)a.out + (size_t)q * out_dim);
#pragma unroll
    for (int c = 0; c < 16; c += 4)
      if (c < out_dim) o[c / 4] = floatx4{y[c], y[c + 1], y[c + 2], y[c + 3]};
  }
}

template <int NL, int CH, int PE, int HID, bool MIP>
int launch_fma(const DecodeArgs &a, hipStream_t stream) {
  const void *fn = (const void *)decode_fma<NL, CH, PE, HID, MIP>;
  const size_t lds = (size_t)kFmaColumn<HID> * kBlock * sizeof(uint32_t);
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return NTC_ERR_HIP;
  const uint64_t blocks = ((uint64_t)a.n + kBlock - 1) / kBlock;
  hipLaunchKernelGGL((decode_fma<NL, CH, PE, HID, MIP>), dim3((unsigned)blocks), dim3(kBlock), lds,
                     stream, a);
  return hip_status(hipGetLastError());
}

// ------------------------------------- non-shared FMA decode, LDS weight cache
//
// The same per-lane computation with the weights read from LDS: one workgroup
// of kFmaLdsThreads threads per CU walks tiles of that many consecutive
// queries and keeps up to `slots` whole decoders in an LDS cache.  For each
// tile it looks up every query's decoder, stages the missing ones into slots
// no pending query of the tile uses (one cooperative copy), and every lane
// whose decoder is cached evaluates its own query with v_dot2c_f32_f16 on rows
// read from its decoder's slot; a tile with more distinct decoders than slots
// takes several passes.  Lanes of one wave that use different decoders read
// different slots in one instruction.  Hidden width 64: activations stay in
// registers (the row loops are unrolled).
constexpr int kFmaLdsThreads = 1024;
constexpr int kFmaLdsWaves = kFmaLdsThreads / kWave;
constexpr size_t kFmaLdsWeightBytes = 144 * 1024;  // the decoder cache
constexpr uint32_t kFmaMaxSlots = 16;
constexpr uint32_t kNoSlotDecoder = 0xFFFFFFFFu;

struct FmaCache {
  uint32_t slot_dec[kFmaMaxSlots];  // decoder held by each slot
  uint32_t used[kFmaMaxSlots];      // a pending query of this pass hit the slot
  uint32_t want[kFmaLdsWaves][kFmaMaxSlots];  // per wave: distinct missing decoders
  uint32_t n_want[kFmaLdsWaves];
  uint32_t stage_slot[kFmaMaxSlots], stage_dec[kFmaMaxSlots];
  uint32_t n_stage;
};

// Layer DIN -> 64 (activated, fp16 pairs) from a decoder's weights in LDS.
template <int DIN>
__device__ __forceinline__ void fma_hidden_lds(const uint16_t *W, const uint32_t (&h)[DIN / 2],
                                               uint32_t (&o)[32], bool leaky, uint32_t slope_h2) {
  const uint16_t *b = W + 64 * DIN;
#pragma unroll
  for (int j = 0; j < 64; j += 2) {
    const float2 bj = unpack_half2(*(const uint32_t *)(b + j));
    float acc0 = bj.x, acc1 = bj.y;
    const u32x4 *r0 = (const u32x4 *)(W + j * DIN);
    const u32x4 *r1 = (const u32x4 *)(W + (j + 1) * DIN);
#pragma unroll
    for (int k = 0; k < DIN / 8; ++k) {
      const u32x4 w0 = r0[k], w1 = r1[k];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc0 = dot2(w0[e], h[4 * k + e], acc0);
        acc1 = dot2(w1[e], h[4 * k + e], acc1);
      }
    }
    o[j / 2] = leaky ? leaky_pack2(acc0, acc1, slope_h2) : relu_pack2(acc0, acc1);
  }
}

// Output layer 64 -> dout (8 or 16), logistic sigmoid, from LDS.
__device__ __forceinline__ void fma_out_lds(const uint16_t *W, int dout, const uint32_t (&h)[32],
                                            float (&y)[16]) {
  const uint16_t *b = W + dout * 64;
#pragma unroll
  for (int j = 0; j < 16; j += 2) {
    if (j < dout) {
      const float2 bj = unpack_half2(*(const uint32_t *)(b + j));
      float acc0 = bj.x, acc1 = bj.y;
      const u32x4 *r0 = (const u32x4 *)(W + j * 64);
      const u32x4 *r1 = (const u32x4 *)(W + (j + 1) * 64);
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const u32x4 w0 = r0[k], w1 = r1[k];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc0 = dot2(w0[e], h[4 * k + e], acc0);
          acc1 = dot2(w1[e], h[4 * k + e], acc1);
        }
      }
      y[j] = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(acc0 * -kLog2e));
      y[j + 1] = __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(acc1 * -kLog2e));
    } else {
      y[j] = y[j + 1] = 0.f;
    }
  }
}

template <int NL, int CH, int PE, bool MIP>
__global__ void __launch_bounds__(kFmaLdsThreads)
decode_fma_lds(const DecodeArgs a, uint32_t slots, uint32_t n_tiles) {
  using S = Shape<NL, CH, PE, 64>;
  extern __shared__ __attribute__((aligned(16))) uint16_t wcache[];
  __shared__ FmaCache c;
  const uint32_t tid = threadIdx.x, lane = lane_id();
  const uint32_t w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const uint32_t stride = (uint32_t)a.dec_stride;  // halves, a multiple of 8
  const uint32_t D = (uint32_t)a.n_decoders;
  const bool leaky = a.leaky != 0;
  if (tid < kFmaMaxSlots) {
    c.slot_dec[tid] = kNoSlotDecoder;
    c.used[tid] = 0;
  }
  for (uint32_t tile = blockIdx.x; tile < n_tiles; tile += gridDim.x) {
    const uint64_t q64 = (uint64_t)tile * kFmaLdsThreads + tid;
    const uint32_t q = (uint32_t)q64;
    const Query qq = validate(a, load_query<NL, MIP>(a, q, q64 < a.n));
    uint32_t d = qq.valid ? a.tex_to_dec[qq.tex] : kNoSlotDecoder;
    if (d >= D) d = kNoSlotDecoder;
    bool pending = d != kNoSlotDecoder;
    uint32_t x[S::F / 2];
    gather<NL, CH, PE, MIP>(a, qq, x);  // an invalid query gathers texture 0, unused
    while (__syncthreads_or(pending)) {
      // look the decoder up; mark the slots this pass reads; list the misses
      int slot = -1;
      if (pending)
        for (uint32_t k = 0; k < slots; ++k)
          if (c.slot_dec[k] == d) slot = (int)k;
      if (pending && slot >= 0) c.used[slot] = 1;
      const bool miss = pending && slot < 0;
      uint64_t todo = ballot(miss);
      uint32_t nw = 0;
      while (todo) {
        const uint32_t dl = read_lane(d, (uint32_t)__builtin_ctzll(todo));
        todo &= ~ballot(d == dl);
        if (lane == 0 && nw < kFmaMaxSlots) c.want[w][nw] = dl;
        ++nw;
      }
      if (lane == 0) c.n_want[w] = nw < kFmaMaxSlots ? nw : kFmaMaxSlots;
      __syncthreads();
      // one thread plans: distinct wanted decoders into slots no pending query hit
      if (tid == 0) {
        uint32_t ns = 0, next = 0;
        bool full = false;
        for (int wv = 0; wv < kFmaLdsWaves && !full; ++wv)
          for (uint32_t i = 0; i < c.n_want[wv] && !full; ++i) {
            const uint32_t dl = c.want[wv][i];
            bool dup = false;
            for (uint32_t k = 0; k < ns; ++k) dup = dup || c.stage_dec[k] == dl;
            if (dup) continue;
            while (next < slots && c.used[next]) ++next;
            if (next == slots) {
              full = true;
              break;
            }
            c.stage_slot[ns] = next;
            c.stage_dec[ns] = dl;
            ++ns;
            ++next;
          }
        c.n_stage = ns;
        for (uint32_t k = 0; k < ns; ++k) c.slot_dec[c.stage_slot[k]] = c.stage_dec[k];
        for (uint32_t k = 0; k < slots; ++k) c.used[k] = 0;
      }
      __syncthreads();
      // every thread copies 16-byte pieces of the staged decoders
      const uint32_t ns = c.n_stage;
      for (uint32_t k = 0; k < ns; ++k) {
        const u32x4 *src = (const u32x4 *)(a.params + (size_t)c.stage_dec[k] * stride);
        u32x4 *dst = (u32x4 *)(wcache + (size_t)c.stage_slot[k] * stride);
        for (uint32_t i = tid; i < stride / 8; i += kFmaLdsThreads) dst[i] = src[i];
      }
      __syncthreads();
      if (pending && slot < 0)
        for (uint32_t k = 0; k < slots; ++k)
          if (c.slot_dec[k] == d) slot = (int)k;
      if (pending && slot >= 0) {
        pending = false;
        const uint16_t *p = wcache + (size_t)slot * stride;
        uint32_t h[32], o[32];
        fma_hidden_lds<S::F>(p, x, h, leaky, a.slope_h2);
        p += 64 * (S::F + 1);
        for (int l = 0; l < a.n_hidden; ++l) {
          fma_hidden_lds<64>(p, h, o, leaky, a.slope_h2);
#pragma unroll
          for (int i = 0; i < 32; ++i) h[i] = o[i];
          p += 64 * 65;
        }
        float y[16];
        fma_out_lds(p, a.out_dim, h, y);
        const int out_dim = a.out_dim;
        if (a.out_f16) {
          u32x2 *o2 = (u32x2 *)((uint16_t *)a.out + (size_t)q * out_dim);
#pragma unroll
          for (int cc = 0; cc < 16; cc += 4)
            if (cc < out_dim)
              o2[cc / 4] = u32x2{pack_half2(y[cc], y[cc + 1]), pack_half2(y[cc + 2], y[cc + 3])};
        } else {
          floatx4 *o4 = (floatx4 *)((float *)a.out + (size_t)q * out_dim);
#pragma unroll
          for (int cc = 0; cc < 16; cc += 4)
            if (cc < out_dim) o4[cc / 4] = floatx4{y[cc], y[cc + 1], y[cc + 2], y[cc + 3]};
        }
      }
    }
  }
}

// Compute units of the current device (one LDS-cache workgroup each).
inline int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus < 1)
    return 256;
  return cus;
}

template <int NL, int CH, int PE, bool MIP>
int launch_fma_lds(const DecodeArgs &a, uint32_t slots, hipStream_t stream) {
  const void *fn = (const void *)decode_fma_lds<NL, CH, PE, MIP>;
  const size_t lds = (size_t)slots * (size_t)a.dec_stride * sizeof(uint16_t);
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return NTC_ERR_HIP;
  const uint64_t n_tiles = ((uint64_t)a.n + kFmaLdsThreads - 1) / kFmaLdsThreads;
  static const int cus = device_cus();
  const uint64_t groups = n_tiles < (uint64_t)cus ? n_tiles : (uint64_t)cus;
  hipLaunchKernelGGL((decode_fma_lds<NL, CH, PE, MIP>), dim3((unsigned)groups),
                     dim3(kFmaLdsThreads), lds, stream, a, slots, (uint32_t)n_tiles);
  return hip_status(hipGetLastError());
}

// Hidden width 64 takes the LDS weight cache when at least one decoder fits it;
// other shapes read their weights through the caches (decode_fma).
template <int NL, int CH, int PE, int HID, bool MIP>
int launch_fma_any(const DecodeArgs &a, hipStream_t stream) {
  if constexpr (HID == 64) {
    const size_t bytes = (size_t)a.dec_stride * sizeof(uint16_t);
    size_t slots = kFmaLdsWeightBytes / bytes;
    if (slots > kFmaMaxSlots) slots = kFmaMaxSlots;
    if (slots >= 1 && a.fma_cache) return launch_fma_lds<NL, CH, PE, MIP>(a, (uint32_t)slots, stream);
  }
  return launch_fma<NL, CH, PE, HID, MIP>(a, stream);
}

template <int NL, int CH, int PE, int HID>
int launch_fma_mip(const DecodeArgs &a, hipStream_t stream) {
  if constexpr (PE > 0) {
    return a.mip ? NTC_ERR_UNSUPPORTED : launch_fma_any<NL, CH, PE, HID, false>(a, stream);
  } else {
    return a.mip ? launch_fma_any<NL, CH, PE, HID, true>(a, stream)
                 : launch_fma_any<NL, CH, PE, HID, false>(a, stream);
  }
}

}  // namespace
}  // namespace ntc
