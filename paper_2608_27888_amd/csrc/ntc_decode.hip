// ntc_decode.hip -- fused latent gather + MLP decoder on MFMA (gfx950).
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
#include "ntc_internal.h"

namespace ntc {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kMaxHidden = 3;  // hidden -> hidden layers

__device__ __forceinline__ uint32_t pack_half2(float a, float b) {
  half2v h = {(_Float16)a, (_Float16)b};  // round to nearest even
  return __builtin_bit_cast(uint32_t, h);
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

template <int NL, int CH, int HID>
struct Shape {
  static constexpr int F = NL * CH;          // features per query
  static constexpr int KS0 = F / 16;         // K-slices of layer 0
  static constexpr int MB = HID / 32;        // 32-row output blocks of a hidden layer
  static constexpr int KSH = HID / 16;       // K-slices of a layer fed by a hidden layer
  static_assert(F % 16 == 0, "feature count must be a multiple of 16");
  static_assert(HID % 32 == 0, "hidden width must be a multiple of 32");
  static_assert(CH == 8 || CH == 16, "8 or 16 channels per level");
};

// LDS image of one decoder: A fragments (64 lanes x 16 B each), then fp32
// biases (rows padded to 32 per block).
struct Image {
  int n_frags;    // fragments
  int bias_off;   // float offset of the biases inside the image (after fragments)
  int n_bias;     // floats
  int bytes;
};

template <int NL, int CH, int HID>
__host__ __device__ inline Image image_of(int n_hidden) {
  using S = Shape<NL, CH, HID>;
  Image im;
  im.n_frags = S::MB * S::KS0 + n_hidden * S::MB * S::KSH + S::KSH;
  im.bias_off = im.n_frags * 256;  // 1024 B = 256 floats per fragment
  im.n_bias = HID * (1 + n_hidden) + 32;
  im.bytes = (im.bias_off + im.n_bias) * 4;
  return im;
}

// Copies decoder `dec` into the LDS image, re-arranged into A fragments; all
// threads of the workgroup take part; the caller brackets it with barriers.
template <int NL, int CH, int HID>
__device__ void stage_decoder(const DecodeArgs &a, uint32_t dec, uint32_t *lds) {
  using S = Shape<NL, CH, HID>;
  const Image im = image_of<NL, CH, HID>(a.n_hidden);
  const uint16_t *p = a.params + (size_t)dec * (size_t)a.dec_stride;
  const int n_layers = a.n_hidden + 2;
  // fragment lane-slices: one 16-byte lane slice per iteration
  for (int lf = threadIdx.x; lf < im.n_frags * kWave; lf += kBlock) {
    const int f = lf / kWave, lane = lf % kWave;
    int layer, mb, s, ks, din, dout;
    if (f < S::MB * S::KS0) {
      layer = 0; mb = f / S::KS0; s = f % S::KS0; ks = S::KS0; din = S::F; dout = HID;
    } else if (f < S::MB * S::KS0 + a.n_hidden * S::MB * S::KSH) {
      const int g = f - S::MB * S::KS0;
      layer = 1 + g / (S::MB * S::KSH);
      const int r = g % (S::MB * S::KSH);
      mb = r / S::KSH; s = r % S::KSH; ks = S::KSH; din = HID; dout = HID;
    } else {
      layer = n_layers - 1; mb = 0; s = f - S::MB * S::KS0 - a.n_hidden * S::MB * S::KSH;
      ks = S::KSH; din = HID; dout = a.out_dim;
    }
    (void)ks;
    // offset of W_layer inside the decoder's parameter block
    size_t woff = 0;
    for (int i = 0; i < layer; ++i) {
      const int di = i == 0 ? S::F : HID;
      woff += (size_t)HID * (di + 1);
    }
    const int row = mb * 32 + (lane & 31), h = lane >> 5;
    uint32_t packed[4];
#pragma unroll
    for (int e2 = 0; e2 < 4; ++e2) {
      uint32_t two = 0;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int e = 2 * e2 + j;
        const int kap = 8 * h + e;
        const int unit = 16 * s + (layer == 0 ? kap : sigma16(kap));
        uint16_t v = 0;
        if (row < dout && unit < din) v = p[woff + (size_t)row * din + unit];
        two |= (uint32_t)v << (16 * j);
      }
      packed[e2] = two;
    }
    u32x4 *dst = (u32x4 *)(lds + (size_t)f * 256 + lane * 4);
    *dst = u32x4{packed[0], packed[1], packed[2], packed[3]};
  }
  // biases, converted to fp32; rows past the layer width are zero
  float *bias = (float *)(lds + im.bias_off);
  for (int i = threadIdx.x; i < im.n_bias; i += kBlock) {
    int layer, row, dout;
    if (i < HID * (1 + a.n_hidden)) {
      layer = i / HID; row = i % HID; dout = HID;
    } else {
      layer = n_layers - 1; row = i - HID * (1 + a.n_hidden); dout = a.out_dim;
    }
    size_t off = 0;
    for (int k = 0; k < layer; ++k) {
      const int di = k == 0 ? S::F : HID;
      off += (size_t)HID * (di + 1);
    }
    const int din = layer == 0 ? S::F : HID;
    float v = 0.f;
    if (row < dout) {
      const uint16_t hb = p[off + (size_t)dout * din + row];
      v = (float)__builtin_bit_cast(_Float16, hb);
    }
    bias[i] = v;
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

// -------------------------------------------------------------------- gather

struct Query {
  uint32_t q;      // query index (only meaningful when valid)
  bool valid;
  uint32_t tex;
  float u, v, mip;
};

// Bilinear sample of one level: CH fp32 values, weights in fp32, latents fed
// to mixed-precision FMAs as fp16.
template <int CH>
__device__ __forceinline__ void sample_level(const uint16_t *level, int res, float resf, float u,
                                             float v, float *f) {
  const float x = __builtin_fmaf(u, resf, -0.5f), y = __builtin_fmaf(v, resf, -0.5f);
  const float x0f = __builtin_floorf(x), y0f = __builtin_floorf(y);
  const float fx = x - x0f, fy = y - y0f;
  // bound before converting so that any finite (or NaN) coordinate stays in range
  const int xi = (int)__builtin_fminf(__builtin_fmaxf(x0f, -1.f), resf);
  const int yi = (int)__builtin_fminf(__builtin_fmaxf(y0f, -1.f), resf);
  // xi, yi in [-1, res]: both taps clamp into [0, res - 1] (clamp-to-edge)
  const int x0 = min(max(xi, 0), res - 1), x1 = min(max(xi + 1, 0), res - 1);
  const int y0 = min(max(yi, 0), res - 1), y1 = min(max(yi + 1, 0), res - 1);
  const float w00 = (1.f - fx) * (1.f - fy), w10 = fx * (1.f - fy);
  const float w01 = (1.f - fx) * fy, w11 = fx * fy;
  const u32x4 *t00 = (const u32x4 *)(level + ((size_t)(y0 * res + x0)) * CH);
  const u32x4 *t10 = (const u32x4 *)(level + ((size_t)(y0 * res + x1)) * CH);
  const u32x4 *t01 = (const u32x4 *)(level + ((size_t)(y1 * res + x0)) * CH);
  const u32x4 *t11 = (const u32x4 *)(level + ((size_t)(y1 * res + x1)) * CH);
  constexpr int NV = CH / 8;  // 16-byte vectors per texel
  u32x4 l00[NV], l10[NV], l01[NV], l11[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    l00[i] = t00[i];
    l10[i] = t10[i];
    l01[i] = t01[i];
    l11[i] = t11[i];
  }
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const half8 a = as_half8(l00[i]), b = as_half8(l10[i]);
    const half8 c = as_half8(l01[i]), d = as_half8(l11[i]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float s = w00 * (float)a[e];
      s = __builtin_fmaf(w10, (float)b[e], s);
      s = __builtin_fmaf(w01, (float)c[e], s);
      s = __builtin_fmaf(w11, (float)d[e], s);
      f[8 * i + e] = s;
    }
  }
}

template <int NL>
__device__ __forceinline__ int pick(const int32_t (&v)[NTC_MAX_LEVELS], int k) {
  int r = v[0];
#pragma unroll
  for (int i = 1; i < NL; ++i) r = k == i ? v[i] : r;
  return r;
}

template <int NL>
__device__ __forceinline__ float pickf(const float (&v)[NTC_MAX_LEVELS], int k) {
  float r = v[0];
#pragma unroll
  for (int i = 1; i < NL; ++i) r = k == i ? v[i] : r;
  return r;
}

// Feature vector of the lane's query, packed as fp16 pairs: x[c/2] holds
// features c and c+1; slot l occupies features [l*CH, (l+1)*CH).
template <int NL, int CH, bool MIP>
__device__ __forceinline__ void gather(const DecodeArgs &a, const Query &qq,
                                       uint32_t (&x)[NL * CH / 2]) {
  const uint16_t *tex = a.latents + (size_t)qq.tex * (size_t)a.tex_stride;
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    float f[CH];
    if (!MIP) {
      sample_level<CH>(tex + a.level_off[l], a.res[l], a.resf[l], qq.u, qq.v, f);
    } else {
      float m = __builtin_fminf(__builtin_fmaxf(qq.mip, 0.f), (float)(NL - 1));
      const float lod = __builtin_fmaxf((float)l, m);
      const int k0 = (int)__builtin_floorf(lod);
      const int k1 = min(k0 + 1, NL - 1);
      const float t = lod - (float)k0;
      sample_level<CH>(tex + pick<NL>(a.level_off, k0), pick<NL>(a.res, k0),
                       pickf<NL>(a.resf, k0), qq.u, qq.v, f);
      if (__builtin_amdgcn_ballot_w64(t != 0.f)) {
        float g[CH];
        sample_level<CH>(tex + pick<NL>(a.level_off, k1), pick<NL>(a.res, k1),
                         pickf<NL>(a.resf, k1), qq.u, qq.v, g);
#pragma unroll
        for (int c = 0; c < CH; ++c) f[c] = __builtin_fmaf(t, g[c] - f[c], f[c]);
      }
    }
#pragma unroll
    for (int c = 0; c < CH; c += 2) x[(l * CH + c) / 2] = pack_half2(f[c], f[c + 1]);
  }
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

// ReLU + fp16 of one 32-row output block -> two K-slices of the next layer.
__device__ __forceinline__ void relu_pack(const floatx16 &acc, half8 &s0, half8 &s1) {
  u32x4 a, b;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = pack_half2(__builtin_fmaxf(acc[2 * i], 0.f), __builtin_fmaxf(acc[2 * i + 1], 0.f));
    b[i] = pack_half2(__builtin_fmaxf(acc[8 + 2 * i], 0.f),
                      __builtin_fmaxf(acc[8 + 2 * i + 1], 0.f));
  }
  s0 = as_half8(a);
  s1 = as_half8(b);
}

__device__ __forceinline__ float sigmoid(float z) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-z * kLog2e));
}

// Runs the staged decoder on the tile's features; returns the output layer's
// accumulators (sigmoid applied) for the two column blocks.
template <int NL, int CH, int HID>
__device__ __forceinline__ void run_mlp(const uint32_t *lds, int n_hidden,
                                        const half8 (&xb0)[NL * CH / 16],
                                        const half8 (&xb1)[NL * CH / 16], floatx16 &y0,
                                        floatx16 &y1) {
  using S = Shape<NL, CH, HID>;
  const float *bias = (const float *)(lds) + image_of<NL, CH, HID>(n_hidden).bias_off;
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
    relu_pack(c0, h0[2 * mb], h0[2 * mb + 1]);
    relu_pack(c1, h1[2 * mb], h1[2 * mb + 1]);
  }
  int frag = S::MB * S::KS0;
  const float *bl = bias + HID;
  // hidden -> hidden
  for (int layer = 0; layer < n_hidden; ++layer) {
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
      relu_pack(c0, n0[2 * mb], n0[2 * mb + 1]);
      relu_pack(c1, n1[2 * mb], n1[2 * mb + 1]);
    }
#pragma unroll
    for (int s = 0; s < S::KSH; ++s) {
      h0[s] = n0[s];
      h1[s] = n1[s];
    }
    frag += S::MB * S::KSH;
    bl += HID;
  }
  // output layer: HID -> out (rows padded to 32)
  floatx16 c0 = bias_frag(bl, 0), c1 = c0;
#pragma unroll
  for (int s = 0; s < S::KSH; ++s) {
    const half8 w = a_frag(lds, frag + s);
    c0 = mfma(w, h0[s], c0);
    c1 = mfma(w, h1[s], c1);
  }
  y0 = c0;
  y1 = c1;
}

// Sigmoid and store of the output rows held by this lane for column block nb.
__device__ __forceinline__ void store_out(float *out, int out_dim, uint32_t q, bool ok,
                                          const floatx16 &z) {
  if (!ok) return;
  const int h = lane_id() >> 5;
  float *row = out + (size_t)q * out_dim;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int r0 = 8 * g + 4 * h;
    if (r0 >= out_dim) continue;
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) y[r] = sigmoid(z[4 * g + r]);
    if (r0 + 4 <= out_dim && (out_dim & 3) == 0) {
      *(floatx4 *)(row + r0) = floatx4{y[0], y[1], y[2], y[3]};
    } else {
      for (int r = 0; r < 4 && r0 + r < out_dim; ++r) row[r0 + r] = y[r];
    }
  }
}

template <int NL, bool MIP>
__device__ __forceinline__ Query load_query(const DecodeArgs &a, uint32_t q, bool in_range) {
  Query r;
  r.q = q;
  r.valid = in_range && q < a.n;
  r.tex = r.valid ? a.tex_id[q] : 0u;
  r.valid = r.valid && r.tex < (uint32_t)a.n_textures;
  if (!r.valid) r.tex = 0;
  r.u = 0.f;
  r.v = 0.f;
  r.mip = 0.f;
  if (r.valid) {
    const float2 uv = ((const float2 *)a.uv)[q];
    r.u = uv.x;
    r.v = uv.y;
    if (MIP) r.mip = a.mip[q];
  }
  return r;
}

// ------------------------------------------------------------------- kernels

template <int NL, int CH, int HID, bool MIP>
__global__ void __launch_bounds__(kBlock)
decode_binned(const DecodeArgs a) {
  using S = Shape<NL, CH, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t D = (uint32_t)a.n_decoders;
  // tiles of the permutation; never more than the buffer holds
  const uint64_t slots = min((uint64_t)a.bin_offset[D], a.perm_capacity);
  const uint32_t total_tiles = (uint32_t)(slots / kWave);
  const uint32_t per = (total_tiles + gridDim.x - 1) / gridDim.x;
  const uint32_t blk = xcd_local_block(blockIdx.x, gridDim.x);
  uint32_t t = blk * per;
  const uint32_t t_end = min(t + per, total_tiles);
  if (t >= t_end) return;
  // bin holding slot 64 t: the last d with bin_offset[d] <= 64 t
  uint32_t lo = 0, hi = D;  // invariant: bin_offset[lo] <= 64 t < bin_offset[hi]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (a.bin_offset[mid] <= t * kWave) lo = mid; else hi = mid;
  }
  uint32_t d = lo, bin_end = a.bin_offset[d + 1] / kWave;
  uint32_t staged = 0xFFFFFFFFu;
  while (t < t_end) {
    while (t >= bin_end && d + 1 < D) {  // next non-empty bin
      ++d;
      bin_end = a.bin_offset[d + 1] / kWave;
    }
    if (t >= bin_end) break;  // offsets not ascending: nothing sensible left to do
    const uint32_t group = min(min((uint32_t)kWavesPerBlock, bin_end - t), t_end - t);
    if (d != staged) {
      __syncthreads();
      stage_decoder<NL, CH, HID>(a, d, lds);
      __syncthreads();
      staged = d;
    }
    if (w < group) {
      const uint32_t slot = (t + w) * kWave + lane;
      const Query qq = load_query<NL, MIP>(a, a.perm[slot], true);
      uint32_t x[S::F / 2];
      gather<NL, CH, MIP>(a, qq, x);
      half8 xb0[S::KS0], xb1[S::KS0];
      to_b_operands<S::KS0>(x, xb0, xb1);
      floatx16 y0, y1;
      run_mlp<NL, CH, HID>(lds, a.n_hidden, xb0, xb1, y0, y1);
      const uint32_t q_other = (uint32_t)__shfl_xor((int)qq.q, 32, kWave);
      const bool ok_other = __shfl_xor((int)qq.valid, 32, kWave) != 0;
      const bool h = lane >= 32;
      store_out(a.out, a.out_dim, h ? q_other : qq.q, h ? ok_other : qq.valid, y0);
      store_out(a.out, a.out_dim, h ? qq.q : q_other, h ? qq.valid : ok_other, y1);
    }
    t += group;
  }
}

template <int NL, int CH, int HID, bool MIP>
__global__ void __launch_bounds__(kBlock)
decode_stream(const DecodeArgs a) {
  using S = Shape<NL, CH, HID>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  __shared__ uint32_t next_dec[2][kWavesPerBlock];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t n_tiles = (a.n + kWave - 1) / kWave;
  const uint32_t n_groups = (n_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
  const uint32_t per = (n_groups + gridDim.x - 1) / gridDim.x;
  const uint32_t blk = xcd_local_block(blockIdx.x, gridDim.x);
  const uint32_t g_begin = blk * per, g_end = min(g_begin + per, n_groups);
  uint32_t staged = 0xFFFFFFFFu;
  int parity = 0;
  const bool h = lane >= 32;
  for (uint32_t g = g_begin; g < g_end; ++g) {
    const uint32_t q = (g * kWavesPerBlock + w) * kWave + lane;
    const Query qq = load_query<NL, MIP>(a, q, true);
    uint32_t dq = 0xFFFFFFFFu;
    bool live = qq.valid;
    if (live) {
      const uint32_t dd = a.tex_to_dec[qq.tex];
      live = dd < (uint32_t)a.n_decoders;
      dq = live ? dd : 0xFFFFFFFFu;
    }
    uint32_t x[S::F / 2];
    gather<NL, CH, MIP>(a, qq, x);
    half8 xb0[S::KS0], xb1[S::KS0];
    to_b_operands<S::KS0>(x, xb0, xb1);
    const uint32_t q_other = (uint32_t)__shfl_xor((int)q, 32, kWave);
    uint64_t todo = ballot(live);
    for (;;) {
      const uint32_t mine =
          todo ? read_lane(dq, (uint32_t)__builtin_ctzll(todo)) : 0xFFFFFFFFu;
      if (lane == 0) next_dec[parity][w] = mine;
      __syncthreads();
      uint32_t d = next_dec[parity][0];
#pragma unroll
      for (int k = 1; k < kWavesPerBlock; ++k) d = min(d, next_dec[parity][k]);
      parity ^= 1;
      if (d == 0xFFFFFFFFu) break;
      if (d != staged) {
        stage_decoder<NL, CH, HID>(a, d, lds);
        __syncthreads();
        staged = d;
      }
      const bool mine_now = live && dq == d;
      const uint64_t sel = ballot(mine_now);
      if (sel) {
        floatx16 y0, y1;
        run_mlp<NL, CH, HID>(lds, a.n_hidden, xb0, xb1, y0, y1);
        const bool sel_other = __shfl_xor((int)mine_now, 32, kWave) != 0;
        store_out(a.out, a.out_dim, h ? q_other : q, h ? sel_other : mine_now, y0);
        store_out(a.out, a.out_dim, h ? q : q_other, h ? mine_now : sel_other, y1);
        todo &= ~sel;
        live = live && !mine_now;
      }
    }
  }
}

template <int NL, int CH, int HID, bool MIP>
int launch_shape(const DecodeArgs &a, hipStream_t stream) {
  const Image im = image_of<NL, CH, HID>(a.n_hidden);
  const size_t lds = (size_t)im.bytes;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const void *fn = a.bin_offset ? (const void *)decode_binned<NL, CH, HID, MIP>
                                : (const void *)decode_stream<NL, CH, HID, MIP>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return NTC_ERR_HIP;
  }
  if (a.bin_offset) {
    uint64_t blocks = ((uint64_t)a.max_tiles + kWavesPerBlock - 1) / kWavesPerBlock;
    const uint64_t cap = (uint64_t)cus * 4;
    if (blocks > cap) blocks = cap;
    if (blocks == 0) return NTC_OK;
    hipLaunchKernelGGL((decode_binned<NL, CH, HID, MIP>), dim3((unsigned)blocks), dim3(kBlock),
                       lds, stream, a);
  } else {
    const uint64_t tiles = ((uint64_t)a.n + kWave - 1) / kWave;
    uint64_t blocks = (tiles + kWavesPerBlock - 1) / kWavesPerBlock;
    const uint64_t cap = (uint64_t)cus * 4;
    if (blocks > cap) blocks = cap;
    if (blocks == 0) return NTC_OK;
    hipLaunchKernelGGL((decode_stream<NL, CH, HID, MIP>), dim3((unsigned)blocks), dim3(kBlock),
                       lds, stream, a);
  }
  return hip_status(hipGetLastError());
}

template <int NL, int CH, int HID>
int launch_mip(const DecodeArgs &a, hipStream_t stream) {
  return a.mip ? launch_shape<NL, CH, HID, true>(a, stream)
               : launch_shape<NL, CH, HID, false>(a, stream);
}

}  // namespace

int launch_decode(const DecodeArgs &a, int n_levels, int channels, int feat, int hidden,
                  hipStream_t stream) {
  (void)feat;
  if (a.n_hidden < 0 || a.n_hidden > kMaxHidden) return NTC_ERR_UNSUPPORTED;
  if (hidden == 64) {
    if (n_levels == 2 && channels == 8) return launch_mip<2, 8, 64>(a, stream);
    if (n_levels == 2 && channels == 16) return launch_mip<2, 16, 64>(a, stream);
    if (n_levels == 3 && channels == 16) return launch_mip<3, 16, 64>(a, stream);
  } else if (hidden == 128) {
    if (n_levels == 2 && channels == 8) return launch_mip<2, 8, 128>(a, stream);
    if (n_levels == 2 && channels == 16) return launch_mip<2, 16, 128>(a, stream);
    if (n_levels == 3 && channels == 16) return launch_mip<3, 16, 128>(a, stream);
  }
  return NTC_ERR_UNSUPPORTED;
}

}  // namespace ntc
