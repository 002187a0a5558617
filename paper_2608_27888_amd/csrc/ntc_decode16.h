// ntc_decode16.h -- binned decode on v_mfma_f32_16x16x32_f16 with an
// LDS-staged latent gather (gfx950).
//
// The decode of a 64-query tile of one bin (one decoder, the shared or
// clustered decoder of Sec. 1 and Sec. 4.4): latent sampling, then the MLP.
// Two departures from the 32x32 kernels of ntc_decode_kernels.h, both measured
// on MI355X:
//
//  * The MLP runs on the 16x16x32 MFMA, which issues at 2.1-2.2 PFLOP/s over
//    the chip against 1.7-1.8 for 32x32x16, and pads an 8-wide output layer to
//    16 rows instead of 32.  Lane l = (g = l / 16, n = l % 16): the B operand of
//    column block j (queries 16j .. 16j+15) holds K-values 8g .. 8g+7 of query
//    16j + n, the A operand row n with the same K-values, the accumulator rows
//    4g .. 4g+3 of column n.  Converted to fp16, the accumulators of row blocks
//    2t and 2t+1 are directly the next layer's B operand for K-step t once that
//    layer's weight columns are permuted (position 8g + e reads unit
//    32t + 4g + e for e < 4 and 32t + 16 + 4g + e - 4 otherwise); the
//    permutation is applied when the weights are staged, so activations never
//    leave registers.  Biases are the first MFMA's accumulator input, 4 floats
//    per lane and row block.
//
//  * Latent taps come from a wave-private LDS region instead of one 16-byte
//    global load per tap and lane.  A vector-memory instruction costs the CU
//    16 cycles of L1 return bandwidth for 64 lanes x 16 bytes whether or not
//    the lanes share addresses, and in binned order the 64 queries of a tile
//    touch about 13 distinct bilinear quads at the finest level (not 64): a
//    query whose quad differs from the previous lane's is a leader, each
//    leader's quad is fetched once by a few lanes (1-4 loads per level instead
//    of 8), written to LDS, and every lane reads its four taps from there.  The
//    fetch for tile k+1 is issued at the start of tile k into a few registers,
//    so its latency is hidden by a whole tile of work.  A level whose tile has
//    more leaders than the region holds is fetched tap by tap from memory for
//    that tile.
//
// Selected with NTC_GATHER_STAGED for binned decode without mip blending.  On
// MI355X it is slower than the direct gather of ntc_decode_kernels.h: the
// planning (leaders, slots, the exchange of quad addresses) adds about 40 VALU
// instructions per tile, more than the 8-10 % of decode time that tap loads
// cost there.
#pragma once

#include "ntc_decode_kernels.h"

namespace ntc {
namespace {

__device__ __forceinline__ floatx4 mfma16(half8 a, half8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

template <int NL, int CH, int PE, int HID>
struct Shape16 {
  static constexpr int FL = NL * CH;         // latent features per query
  static constexpr int F = FL + PE;          // + positional-encoding features
  static constexpr int KS0 = (F + 31) / 32;  // 32-wide K-steps of layer 0 (zero padded)
  static constexpr int MB = HID / 16;        // 16-row blocks of a hidden layer
  static constexpr int KSH = HID / 32;       // K-steps of a layer fed by a hidden layer
  static_assert(F % 16 == 0, "feature count must be a multiple of 16");
  static_assert(HID % 32 == 0, "hidden width must be a multiple of 32");
  static_assert(CH == 8 || CH == 16, "8 or 16 channels per level");
};

// LDS image of one decoder in the 16x16 layout: fragments (64 lanes x 16 B),
// then fp32 biases: HID per layer fed to a hidden activation, then 16 for the
// output layer (scaled by -log2(e), rows past the width zero).
template <int NL, int CH, int PE, int HID>
__host__ __device__ inline Image image16_of(int n_hidden) {
  using S = Shape16<NL, CH, PE, HID>;
  Image im;
  im.n_frags = S::MB * S::KS0 + n_hidden * S::MB * S::KSH + S::KSH;
  im.bias_off = im.n_frags * 256;
  im.n_bias = HID * (1 + n_hidden) + 16;
  im.bytes = (im.bias_off + im.n_bias) * 4;
  return im;
}

// Weight unit that element e of lane group g reads in K-step s of a layer:
// layer 0 reads the features in order, later layers the order in which the
// previous layer's accumulators leave its outputs.
__device__ __forceinline__ int unit16(int layer, int s, int g, int e) {
  return layer == 0 ? 32 * s + 8 * g + e : 32 * s + (e < 4 ? 4 * g + e : 16 + 4 * g + e - 4);
}

// Copies decoder `dec` into the LDS image (all threads of the workgroup; the
// caller brackets it with barriers).  Weights outside their layer read as zero
// (raw buffer loads past the block return zero).
template <int NL, int CH, int PE, int HID, int THREADS>
__device__ void stage_decoder16(const DecodeArgs &a, uint32_t dec, uint32_t *lds) {
  using S = Shape16<NL, CH, PE, HID>;
  const Image im = image16_of<NL, CH, PE, HID>(a.n_hidden);
  const uint16_t *p = a.params + (size_t)dec * (size_t)a.dec_stride;
  const __amdgpu_buffer_rsrc_t rsrc =
      __builtin_amdgcn_make_buffer_rsrc((void *)p, 0, (int)(a.dec_stride * 2), 0x00020000);
  const int n_layers = a.n_hidden + 2;
  const int f_hid = S::MB * S::KS0, f_out = f_hid + a.n_hidden * S::MB * S::KSH;
  auto layer_off = [&](int layer) -> size_t {
    return layer == 0 ? 0 : (size_t)HID * (S::F + 1) + (size_t)(layer - 1) * HID * (HID + 1);
  };
  const int n_slices = im.n_frags * kWave;
  for (int base = threadIdx.x; base < n_slices; base += kStageSlices * THREADS) {
    uint32_t v[kStageSlices][8];
#pragma unroll
    for (int i = 0; i < kStageSlices; ++i) {
      int lf = base + i * THREADS;
      lf = lf < n_slices ? lf : 0;
      const int f = lf / kWave, lane = lf % kWave, g = lane >> 4, n = lane & 15;
      int layer, mb, s, din, dout;
      if (f < f_hid) {
        layer = 0; mb = f / S::KS0; s = f % S::KS0; din = S::F; dout = HID;
      } else if (f < f_out) {
        const int q = f - f_hid;
        layer = 1 + q / (S::MB * S::KSH);
        mb = (q % (S::MB * S::KSH)) / S::KSH;
        s = q % S::KSH;
        din = HID; dout = HID;
      } else {
        layer = n_layers - 1; mb = 0; s = f - f_out; din = HID; dout = a.out_dim;
      }
      const int row = 16 * mb + n;
      const size_t woff = layer_off(layer);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int unit = unit16(layer, s, g, e);
        const bool in = row < dout && unit < din;
        const uint32_t off = in ? (uint32_t)(woff + (size_t)row * din + unit) * 2u : kPastBlock;
        v[i][e] = __builtin_amdgcn_raw_buffer_load_b16(rsrc, off, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < kStageSlices; ++i) {
      const int lf = base + i * THREADS;
      if (lf < n_slices) {
        const u32x4 packed = {v[i][0] | v[i][1] << 16, v[i][2] | v[i][3] << 16,
                              v[i][4] | v[i][5] << 16, v[i][6] | v[i][7] << 16};
        *(u32x4 *)(lds + (size_t)lf * 4) = packed;
      }
    }
  }
  float *bias = (float *)(lds + im.bias_off);
  for (int i = threadIdx.x; i < im.n_bias; i += THREADS) {
    int layer, row, dout;
    if (i < HID * (1 + a.n_hidden)) {
      layer = i / HID; row = i % HID; dout = HID;
    } else {
      layer = n_layers - 1; row = i - HID * (1 + a.n_hidden); dout = a.out_dim;
    }
    const int din = layer == 0 ? S::F : HID;
    const uint32_t boff =
        row < dout ? (uint32_t)(layer_off(layer) + (size_t)dout * din + row) * 2u : kPastBlock;
    const uint16_t hb = __builtin_amdgcn_raw_buffer_load_b16(rsrc, boff, 0, 0);
    const float v = (float)__builtin_bit_cast(_Float16, hb);
    bias[i] = layer == n_layers - 1 ? v * -kLog2e : v;
  }
}

__device__ __forceinline__ half8 frag16(const uint32_t *lds, int f) {
  return as_half8(*(const u32x4 *)(lds + (size_t)f * 256 + lane_id() * 4));
}

// The 4 biases of this lane's rows in row block mb of a layer.
__device__ __forceinline__ floatx4 bias16(const float *bias_layer, int mb) {
  return *(const floatx4 *)(bias_layer + 16 * mb + 4 * (lane_id() >> 4));
}

// Hidden activation and fp16 of row blocks 2t (lo) and 2t+1 (hi): the next
// layer's B operand for K-step t.
template <bool LEAKY>
__device__ __forceinline__ half8 act_pack16(const floatx4 &lo, const floatx4 &hi,
                                            uint32_t slope_h2) {
  if constexpr (LEAKY) {
    return as_half8(u32x4{leaky_pack2(lo[0], lo[1], slope_h2), leaky_pack2(lo[2], lo[3], slope_h2),
                          leaky_pack2(hi[0], hi[1], slope_h2), leaky_pack2(hi[2], hi[3], slope_h2)});
  } else {
    return as_half8(u32x4{relu_pack2(lo[0], lo[1]), relu_pack2(lo[2], lo[3]),
                          relu_pack2(hi[0], hi[1]), relu_pack2(hi[2], hi[3])});
  }
}

// B operands of layer 0 from the features of the lane's own query (lane =
// query slot; x[c/2] holds features c, c+1): a 4x4 transpose of (16-lane row,
// 8-feature group) blocks per K-step, one v_permlane32_swap stage and one
// v_permlane16_swap stage.  Afterwards xb[j][s] holds, in lane (g, n),
// features 32s + 8g .. +7 of query 16j + n.
template <int KS0, int XW>
__device__ __forceinline__ void to_b16(const uint32_t (&x)[XW], half8 (&xb)[4][KS0]) {
#pragma unroll
  for (int s = 0; s < KS0; ++s) {
    uint32_t e[4][4];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int w = 16 * s + 4 * g + v;
        e[g][v] = w < XW ? x[w] : 0u;
      }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const auto a = __builtin_amdgcn_permlane32_swap(e[0][v], e[2][v], false, false);
      const auto b = __builtin_amdgcn_permlane32_swap(e[1][v], e[3][v], false, false);
      e[0][v] = a[0]; e[2][v] = a[1];
      e[1][v] = b[0]; e[3][v] = b[1];
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const auto a = __builtin_amdgcn_permlane16_swap(e[0][v], e[1][v], false, false);
      const auto b = __builtin_amdgcn_permlane16_swap(e[2][v], e[3][v], false, false);
      e[0][v] = a[0]; e[1][v] = a[1];
      e[2][v] = b[0]; e[3][v] = b[1];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) xb[j][s] = as_half8(u32x4{e[j][0], e[j][1], e[j][2], e[j][3]});
  }
}

// Layer 0 of the staged decoder (F -> HID) on the tile's 4 column blocks:
// h[j][t] is the next layer's B operand for K-step t.
template <int NL, int CH, int PE, int HID, int NH, bool LEAKY>
__device__ __forceinline__ void mlp16_layer0(const uint32_t *lds,
                                             const half8 (&xb)[4][Shape16<NL, CH, PE, HID>::KS0],
                                             half8 (&h)[4][HID / 32], uint32_t slope_h2) {
  using S = Shape16<NL, CH, PE, HID>;
  const float *bias = (const float *)(lds) + image16_of<NL, CH, PE, HID>(NH).bias_off;
#pragma unroll
  for (int t = 0; t < S::KSH; ++t) {
    const floatx4 blo = bias16(bias, 2 * t), bhi = bias16(bias, 2 * t + 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      floatx4 lo = blo, hi = bhi;
#pragma unroll
      for (int s = 0; s < S::KS0; ++s) {
        lo = mfma16(frag16(lds, (2 * t) * S::KS0 + s), xb[j][s], lo);
        hi = mfma16(frag16(lds, (2 * t + 1) * S::KS0 + s), xb[j][s], hi);
      }
      h[j][t] = act_pack16<LEAKY>(lo, hi, slope_h2);
    }
  }
}

// The hidden and output layers; y[j] holds the output layer's accumulators
// (rows 4g .. 4g+3 of query 16j + n), bias not yet added.
template <int NL, int CH, int PE, int HID, int NH, bool LEAKY>
__device__ __forceinline__ void mlp16_rest(const uint32_t *lds, half8 (&h)[4][HID / 32],
                                           floatx4 (&y)[4], uint32_t slope_h2) {
  using S = Shape16<NL, CH, PE, HID>;
  const float *bias = (const float *)(lds) + image16_of<NL, CH, PE, HID>(NH).bias_off;
  int frag = S::MB * S::KS0;
  const float *bl = bias + HID;
  // hidden -> hidden
#pragma unroll
  for (int layer = 0; layer < NH; ++layer) {
    half8 m[4][S::KSH];
#pragma unroll
    for (int t = 0; t < S::KSH; ++t) {
      const floatx4 blo = bias16(bl, 2 * t), bhi = bias16(bl, 2 * t + 1);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        floatx4 lo = blo, hi = bhi;
#pragma unroll
        for (int s = 0; s < S::KSH; ++s) {
          lo = mfma16(frag16(lds, frag + (2 * t) * S::KSH + s), h[j][s], lo);
          hi = mfma16(frag16(lds, frag + (2 * t + 1) * S::KSH + s), h[j][s], hi);
        }
        m[j][t] = act_pack16<LEAKY>(lo, hi, slope_h2);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < S::KSH; ++t) h[j][t] = m[j][t];
    frag += S::MB * S::KSH;
    bl += HID;
  }
  // output layer: HID -> 16 rows (rows past the width have zero weights)
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    floatx4 c = {};
#pragma unroll
    for (int s = 0; s < S::KSH; ++s) c = mfma16(frag16(lds, frag + s), h[j][s], c);
    y[j] = c;
  }
}

// ----------------------------------------------------------------- staging

// Wave-private LDS staging of the bilinear quads of one tile.  A quad is the
// 2x2 texels of one level around a query: 4 * CH / 8 pieces of 16 bytes,
// (x0, y0), (x0 + 1, y0), (x0, y0 + 1), (x0 + 1, y0 + 1), each texel's pieces
// in channel order.  Region of level l: cap(l) quad slots of QS bytes (a quad
// and 16 bytes of padding: the lanes of one read instruction address
// different slots at the same piece offset, and the padding spreads those
// slots over distinct LDS banks); then an exchange table of 8 bytes per slot
// (the quad's fp16 element offset).
template <int CH>
struct Staging {
  static constexpr int NV = CH / 8;          // pieces per texel
  static constexpr int PIECES = 4 * NV;      // pieces per quad
  static constexpr int QB = PIECES * 16;     // bytes per quad
  static constexpr int QS = QB + 16;         // bytes per slot
  static constexpr int loads(int l) { return l == 0 ? 4 : 3; }   // 16-byte loads per lane and level
  static constexpr int cap(int l) { return loads(l) * kWave / PIECES; }  // quads per level
  static constexpr int region(int l) {
    int b = 0;
    for (int i = 0; i < l; ++i) b += cap(i) * QS;
    return b;
  }
  template <int NL>
  static constexpr int bytes() {
    return region(NL) + xchg_bytes<NL>();
  }
  template <int NL>
  static constexpr int xchg_bytes() {
    int b = 0;
    for (int l = 0; l < NL; ++l) b += cap(l) * 8;
    return b;
  }
  template <int NL>
  static constexpr int xchg(int l) {
    int b = region(NL);
    for (int i = 0; i < l; ++i) b += cap(i) * 8;
    return b;
  }
  // LDS byte offset, inside its level's region, of piece 64 m + lane of the
  // level's staged quads (quad (64 m + lane) / PIECES, piece (64 m + lane) %
  // PIECES).
  static constexpr int piece_pos(int m, int lane) {
    return ((m * kWave + lane) / PIECES) * QS + ((m * kWave + lane) % PIECES) * 16;
  }
};

// Per-lane plan of one tile: for each level, the byte offset of the lane's
// quad in the wave's staging region (or of nothing when the level is fetched
// tap by tap) and its bilinear position; plus the query's texture and uv for
// such a level.
template <int NL>
struct TilePlan {
  uint32_t tap_off[NL];  // word offset in LDS of the lane's quad (staged levels)
  float fx[NL], fy[NL];
  uint32_t staged;       // wave-uniform: bit l set when level l is staged
};

// Global data of the leaders' quads of the next tile, in registers until they
// are written to LDS.
template <int NL>
struct StageData {
  u32x4 v[NL][4];
};

// Plans the tile whose (validated) query data is `qq`: bilinear positions,
// leaders (a valid query whose quad differs from the previous lane's, or whose
// previous lane holds no valid query), slots, and the loads of the leaders'
// quads into `sd` (issued, not waited for).  wave_w is the word offset of the
// wave's staging region in `lds`.  A wave's LDS operations execute in order,
// so the exchange table written and read back here needs no barrier.
template <int NL, int CH>
__device__ __forceinline__ TilePlan<NL> plan_tile(const DecodeArgs &a, const Query &qq,
                                                  uint32_t *lds, uint32_t wave_w,
                                                  const uint32_t (&piece_off)[NL],
                                                  StageData<NL> &sd) {
  using St = Staging<CH>;
  TilePlan<NL> P;
  P.staged = 0;
  const uint32_t lane = lane_id();
  // previous lane's texture and validity (lane 0 has none)
  const uint32_t valid = qq.valid ? 1u : 0u;
  const uint32_t prev_valid = __builtin_amdgcn_update_dpp(0u, valid, 0x138, 0xf, 0xf, false);
  const uint32_t prev_tex = __builtin_amdgcn_update_dpp(0u, qq.tex, 0x138, 0xf, 0xf, false);
  const bool new_run = qq.valid && (!prev_valid || prev_tex != qq.tex);
  const uint64_t tex_base = (uint64_t)qq.tex * (uint64_t)a.tex_stride;
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const float resf = a.resf[l];
    const float x = __builtin_fmaf(qq.u, resf, -0.5f), y = __builtin_fmaf(qq.v, resf, -0.5f);
    const float hi = resf - 2.f;
    const float x0 = __builtin_amdgcn_fmed3f(__builtin_floorf(x), 0.f, hi);
    const float y0 = __builtin_amdgcn_fmed3f(__builtin_floorf(y), 0.f, hi);
    P.fx[l] = __builtin_amdgcn_fmed3f(x - x0, 0.f, 1.f);
    P.fy[l] = __builtin_amdgcn_fmed3f(y - y0, 0.f, 1.f);
    const uint32_t idx = (uint32_t)y0 * (uint32_t)a.res[l] + (uint32_t)x0;
    const uint32_t prev_idx = __builtin_amdgcn_update_dpp(0u, idx, 0x138, 0xf, 0xf, false);
    const bool lead = new_run || (qq.valid && prev_idx != idx);
    const uint64_t mask = ballot(lead);
    const uint32_t nlead = (uint32_t)__builtin_popcountll(mask);
    // slot of the lane's leader (lanes before the first leader hold no valid query)
    const uint32_t rank = lanes_below(mask) + (lead ? 1u : 0u);
    const uint32_t slot = rank ? rank - 1u : 0u;
    P.tap_off[l] = wave_w + (St::region(l) + slot * St::QS) / 4;
    if (nlead <= (uint32_t)St::cap(l)) P.staged |= 1u << l;
    // The leaders' quad addresses (fp16 element offsets) go through the exchange
    // table; every load of the level is issued whatever the number of leaders
    // (no branch: a conditional load would be waited for right away), pieces
    // past the last leader's repeating its quad.  A level with more leaders than
    // the table holds is not staged; its loads only fill registers.
    uint64_t *xchg = (uint64_t *)(lds + wave_w + St::template xchg<NL>(l) / 4);
    const uint64_t elem = tex_base + a.level_off[l] + (uint64_t)idx * CH;
    // a wave without a valid query (no leader) has lane 0 enter texture 0's
    // first texels, which always exist; entries 0 .. last are written here
    if (nlead ? lead && slot < (uint32_t)St::cap(l) : lane == 0u) xchg[nlead ? slot : 0u] = nlead ? elem : 0ull;
    const uint32_t last = nlead ? min(nlead, (uint32_t)St::cap(l)) - 1u : 0u;
#pragma unroll
    for (int m = 0; m < St::loads(l); ++m) {
      const uint32_t k = min((m * kWave + lane) / St::PIECES, last);
      const char *src = (const char *)(a.latents + xchg[k]) + piece_off[l];
      sd.v[l][m] = *(const u32x4 *)src;
    }
  }
  return P;
}

// Writes the staged quads of a plan into the wave's region (after the wave is
// done reading the previous tile's taps from it).
template <int NL, int CH>
__device__ __forceinline__ void write_staged(const TilePlan<NL> &P, const StageData<NL> &sd,
                                             uint32_t *lds, uint32_t wave_w) {
  using St = Staging<CH>;
  const uint32_t lane = lane_id();
#pragma unroll
  for (int l = 0; l < NL; ++l) {
#pragma unroll
    for (int m = 0; m < St::loads(l); ++m)
      *(u32x4 *)(lds + wave_w + (St::region(l) + St::piece_pos(m, (int)lane)) / 4) = sd.v[l][m];
  }
}

// Features of the lane's query (lane = query slot) from the staged quads, or,
// for a level that was not staged, from taps loaded here.
template <int NL, int CH, int PE>
__device__ __forceinline__ void gather_staged(const DecodeArgs &a, const Query &qq,
                                              const TilePlan<NL> &P, const uint32_t *lds,
                                              uint32_t (&x)[(NL * CH + PE) / 2]) {
  using St = Staging<CH>;
  if constexpr (PE > 0) pos_encoding<PE>(qq.u, qq.v, x + NL * CH / 2);
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    LevelTaps<CH> L;
    if (P.staged & (1u << l)) {
      const u32x4 *q = (const u32x4 *)(lds + P.tap_off[l]);
#pragma unroll
      for (int i = 0; i < St::NV; ++i) {
        L.t00[i] = q[0 * St::NV + i];
        L.t10[i] = q[1 * St::NV + i];
        L.t01[i] = q[2 * St::NV + i];
        L.t11[i] = q[3 * St::NV + i];
      }
      L.fx = P.fx[l];
      L.fy = P.fy[l];
    } else {
      const uint16_t *tex = a.latents + (size_t)qq.tex * (size_t)a.tex_stride;
      fetch_level<CH>(tex, a.level_off[l], a.res[l], a.resf[l], qq.u, qq.v, L);
    }
    interp_level_h2<CH>(L, x + l * CH / 2);
  }
}

// ----------------------------------------------------------------- output

// Decoded values of one lane for the store: rows r0 .. r0+3 of one query.
// Output widths up to 8 use the rows of lane groups 0 and 1 only; the upper
// half-wave of y[0] / y[1] takes y[2] / y[3]'s lower half first, so every lane
// finishes 4 values of y01[0] (queries 16n, blocks 0 / 2) and 4 of y01[1]
// (blocks 1 / 3).
// Bit casts through by-value helpers: a __builtin_bit_cast applied directly to
// an element of an ext_vector inside an unrolled loop is folded to element 0 by
// this compiler.
__device__ __forceinline__ uint32_t f32_bits(float f) { return __builtin_bit_cast(uint32_t, f); }
__device__ __forceinline__ float bits_f32(uint32_t u) { return __builtin_bit_cast(float, u); }

__device__ __forceinline__ void compact_out(floatx4 (&y)[4]) {
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const auto a = __builtin_amdgcn_permlane32_swap(f32_bits(y[0][r]), f32_bits(y[2][r]), false,
                                                    false);
    const auto b = __builtin_amdgcn_permlane32_swap(f32_bits(y[1][r]), f32_bits(y[3][r]), false,
                                                    false);
    y[0][r] = bits_f32(a[0]);
    y[1][r] = bits_f32(b[0]);
  }
}

// Store of rows r0 .. r0 + 3 of query q (of the output's first 16 rows) in the
// given mode; rows at or past out_dim, and queries that are not ok, are
// dropped.
template <int STORE>
__device__ __forceinline__ void store4(__amdgpu_buffer_rsrc_t out, int out_dim, uint32_t q,
                                       bool ok, int r0, const u32x4 &v, uint32_t out_f16) {
  if constexpr (STORE == kStoreF32x4) {
    const uint32_t off = ok && r0 < out_dim ? (q * (uint32_t)out_dim + (uint32_t)r0) * 4u
                                            : kDropOffset;
    __builtin_amdgcn_raw_buffer_store_b128(v, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF16x4) {
    const uint32_t off = ok && r0 < out_dim ? (q * (uint32_t)out_dim + (uint32_t)r0) * 2u
                                            : kDropOffset;
    const float4 f = __builtin_bit_cast(float4, v);
    const u32x2 h = {pack_half2(f.x, f.y), pack_half2(f.z, f.w)};
    __builtin_amdgcn_raw_buffer_store_b64(h, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF32x3) {
    const uint32_t off = ok && r0 == 0 ? q * 12u : kDropOffset;
    const u32x3 w = {v[0], v[1], v[2]};
    __builtin_amdgcn_raw_buffer_store_b96(w, out, off, 0, kOutPolicy);
  } else if constexpr (STORE == kStoreF16x3) {
    const float4 f = __builtin_bit_cast(float4, v);
    const bool even = (q & 1u) == 0;
    const uint32_t base = q * 6u;
    const bool st = ok && r0 == 0;
    const uint32_t off32 = st ? (even ? base : base + 2u) : kDropOffset;
    const uint32_t off16 = st ? (even ? base + 4u : base) : kDropOffset;
    const uint32_t pair = even ? pack_half2(f.x, f.y) : pack_half2(f.y, f.z);
    const _Float16 single = (_Float16)(even ? f.z : f.x);
    __builtin_amdgcn_raw_buffer_store_b32(pair, out, off32, 0, kOutPolicy);
    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, single), out, off16, 0,
                                           kOutPolicy);
  } else {
    const uint32_t row = q * (uint32_t)out_dim;
    const uint32_t es = out_f16 ? 2u : 4u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int rr = r0 + i;
      const uint32_t off = ok && rr < out_dim ? (row + (uint32_t)rr) * es : kDropOffset;
      if (out_f16) {
        const _Float16 f = (_Float16)bits_f32(v[i]);
        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(uint16_t, f), out, off, 0,
                                               kOutPolicy);
      } else {
        __builtin_amdgcn_raw_buffer_store_b32(v[i], out, off, 0, kOutPolicy);
      }
    }
  }
}

// Finished output of a tile: sigmoid applied, with the query index and
// validity of each stored row group.  Widths up to 8 (WIDE = false) hold two
// 4-row groups per lane (after compact_out), wider outputs four.
template <bool WIDE>
struct TileOut {
  static constexpr int G = WIDE ? 4 : 2;
  u32x4 v[G];
  uint32_t q[G];
  uint32_t ok;   // bit i: group i is valid
};

// Sigmoid of the output accumulators with the scaled output biases; q and ok
// of the lane's own query slot (lane = query slot) are redistributed to the
// lanes that store its rows.
template <bool WIDE>
__device__ __forceinline__ TileOut<WIDE> finish16(floatx4 (&y)[4], const float *out_bias,
                                                  uint32_t q, bool ok) {
  TileOut<WIDE> o;
  const uint32_t lane = lane_id(), g = lane >> 4;
  const uint32_t okw = ok ? 1u : 0u;
  o.ok = 0;
  if constexpr (!WIDE) {
    compact_out(y);
    const floatx4 b = *(const floatx4 *)(out_bias + 4 * (g & 1));
    // lane (g, n) stores query slots (g < 2 ? n : 32 + n) and (g < 2 ? 16 + n : 48 + n)
    const auto qs = __builtin_amdgcn_permlane16_swap(q, q, false, false);
    const auto oks = __builtin_amdgcn_permlane16_swap(okw, okw, false, false);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int r = 0; r < 4; ++r) o.v[i][r] = f32_bits(sigmoid(y[i][r], b[r]));
      o.q[i] = qs[i];
      o.ok |= (oks[i] & 1u) << i;
    }
  } else {
    const floatx4 b = *(const floatx4 *)(out_bias + 4 * g);
    // lane (g, n) stores rows 4g .. 4g+3 of query slot 16j + n of each block j:
    // a 4x4 transpose of (row, block) of the query index and its validity
    uint32_t tq[4] = {q, q, q, q}, tk[4] = {okw, okw, okw, okw};
    {
      auto a = __builtin_amdgcn_permlane32_swap(tq[0], tq[2], false, false);
      auto b2 = __builtin_amdgcn_permlane32_swap(tq[1], tq[3], false, false);
      tq[0] = a[0]; tq[2] = a[1]; tq[1] = b2[0]; tq[3] = b2[1];
      a = __builtin_amdgcn_permlane16_swap(tq[0], tq[1], false, false);
      b2 = __builtin_amdgcn_permlane16_swap(tq[2], tq[3], false, false);
      tq[0] = a[0]; tq[1] = a[1]; tq[2] = b2[0]; tq[3] = b2[1];
      a = __builtin_amdgcn_permlane32_swap(tk[0], tk[2], false, false);
      b2 = __builtin_amdgcn_permlane32_swap(tk[1], tk[3], false, false);
      tk[0] = a[0]; tk[2] = a[1]; tk[1] = b2[0]; tk[3] = b2[1];
      a = __builtin_amdgcn_permlane16_swap(tk[0], tk[1], false, false);
      b2 = __builtin_amdgcn_permlane16_swap(tk[2], tk[3], false, false);
      tk[0] = a[0]; tk[1] = a[1]; tk[2] = b2[0]; tk[3] = b2[1];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int r = 0; r < 4; ++r) o.v[j][r] = f32_bits(sigmoid(y[j][r], b[r]));
      o.q[j] = tq[j];
      o.ok |= (tk[j] & 1u) << j;
    }
  }
  return o;
}

template <int STORE, bool WIDE>
__device__ __forceinline__ void store_out16(__amdgpu_buffer_rsrc_t out, int out_dim,
                                            const TileOut<WIDE> &o, uint32_t out_f16) {
  const uint32_t g = lane_id() >> 4;
  const int r0 = WIDE ? 4 * (int)g : 4 * (int)(g & 1);
#pragma unroll
  for (int i = 0; i < TileOut<WIDE>::G; ++i)
    store4<STORE>(out, out_dim, o.q[i], (o.ok >> i) & 1u, r0, o.v[i], out_f16);
}

// Store instructions of one store_out16 call, fixed per mode.
// ----------------------------------------------------------------- kernel

// Waves per workgroup and per SIMD of the 16x16 binned kernel.  A wave holds
// the MLP's activations, the next tile's plan and the query prefetches in at
// most 168 VGPRs (3 waves per SIMD) for 64-wide decoders: one 12-wave
// workgroup per CU shares one staged decoder.  128-wide decoders use 8-wave
// workgroups, 2 waves per SIMD.
template <int HID>
constexpr int kWaves16 = HID > 64 ? 8 : 12;
template <int HID>
constexpr int kThreads16 = kWaves16<HID> * kWave;
template <int HID>
constexpr int kWavesPerEu16 = HID > 64 ? 2 : 3;

// Where the next tile's staged quads are written: right after this tile's taps
// are read (their loads have the least time to land, their registers are free
// for layer 0), or after layer 0.
constexpr bool kStageAfterLayer0 = false;

template <int NL, int CH, int PE, int HID, int NH, int STORE, bool LEAKY>
__global__ void __launch_bounds__((kThreads16<HID>), (kWavesPerEu16<HID>))
decode_binned16(const DecodeArgs a, uint32_t image_bytes) {
  constexpr int WAVES = kWaves16<HID>;
  constexpr int THREADS = kThreads16<HID>;
  constexpr bool WIDE = false;  // widths up to 8 (wider outputs use the 32x32 kernel)
  using S = Shape16<NL, CH, PE, HID>;
  using St = Staging<CH>;
  extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
  const uint32_t w = threadIdx.x / kWave, lane = lane_id();
  const uint32_t D = (uint32_t)a.n_decoders;
  const __amdgpu_buffer_rsrc_t out_rsrc = out_resource(a);
  // this wave's staging region: a word offset in `lds`, past the decoder image
  const uint32_t wave_w = (image_bytes + w * (uint32_t)St::template bytes<NL>()) / 4;
  // byte offset of this lane's piece inside a quad, per level
  uint32_t piece_off[NL];
#pragma unroll
  for (int l = 0; l < NL; ++l) {
    const uint32_t p = lane % St::PIECES, tap = p / St::NV, vec = p % St::NV;
    piece_off[l] = (tap & 1u) * CH * 2u + (tap >> 1) * (uint32_t)a.res[l] * CH * 2u + vec * 16u;
  }
  const uint64_t slots = min((uint64_t)bin_off(a, D), a.perm_capacity);
  const uint32_t total_tiles = (uint32_t)(slots / kWave);
  const uint32_t per = (total_tiles + gridDim.x - 1) / gridDim.x;
  const uint32_t blk = xcd_local_block(blockIdx.x, gridDim.x);
  const uint32_t t = blk * per;
  const uint32_t t_end = min(t + per, total_tiles);
  if (t >= t_end) return;
  uint32_t lo = 0, hi = D;  // bin holding slot 64 t: bin_offset[lo] <= 64 t < bin_offset[hi]
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) / 2;
    if (bin_off(a, mid) <= t * kWave) lo = mid; else hi = mid;
  }
  Group g0 = group_at<WAVES>(a, t, lo, bin_off(a, lo + 1) / kWave, D, t_end);
  Group g1 = next_group<WAVES>(a, g0, D, t_end);
  Group g2 = next_group<WAVES>(a, g1, D, t_end);
  Group g3 = next_group<WAVES>(a, g2, D, t_end);
  struct Slot {
    uint32_t raw;
    bool has;
  };
  auto slot_query = [&](const Group &g) -> Slot {
    const bool has = w < g.n;
    return Slot{a.perm[has ? (g.t + w) * kWave + lane : 0u], has};
  };
  auto restage = [&](uint32_t d) {
    __syncthreads();
    stage_decoder16<NL, CH, PE, HID, THREADS>(a, d, lds);
    __syncthreads();
  };
  // prologue: tile 0 planned and staged, tile 1's query data and tile 2's
  // permutation entry in flight
  const Slot s0 = slot_query(g0);
  Query cur = validate(a, load_query<NL, false>(a, s0.raw, s0.has));
  restage(g0.d);
  uint32_t staged_dec = g0.d;
  StageData<NL> sd;
  TilePlan<NL> plan = plan_tile<NL, CH>(a, cur, lds, wave_w, piece_off, sd);
  write_staged<NL, CH>(plan, sd, lds, wave_w);
  const Slot s1 = slot_query(g1);
  Query q_next = load_query<NL, false>(a, s1.raw, s1.has);
  Slot p_next = slot_query(g2);
  // the previous tile's output, stored one tile late (none before the first:
  // its stores are dropped, so every tile issues the same stores)
  TileOut<WIDE> pending;
#pragma unroll
  for (int i = 0; i < TileOut<WIDE>::G; ++i) {
    pending.v[i] = u32x4{0u, 0u, 0u, 0u};
    pending.q[i] = 0u;
  }
  pending.ok = 0u;
  auto tile = [&](const Query &q_in, const Slot &p_in, Query &q_out, Slot &p_out) {
    // prefetches: query data two tiles ahead, the permutation entry three ahead
    q_out = load_query<NL, false>(a, p_in.raw, p_in.has);
    p_out = slot_query(g3);
    __builtin_amdgcn_sched_barrier(0);
    // plan of the next tile; its quads' loads go out now
    const Query nxt = validate(a, q_in);
    const TilePlan<NL> plan_next = plan_tile<NL, CH>(a, nxt, lds, wave_w, piece_off, sd);
    __builtin_amdgcn_sched_barrier(0);
    // the previous tile's stores, after every load of this tile in issue order
    store_out16<STORE, WIDE>(out_rsrc, a.out_dim, pending, a.out_f16);
    __builtin_amdgcn_sched_barrier(0);
    // this tile: features from the staged quads
    uint32_t x[S::F / 2];
    gather_staged<NL, CH, PE>(a, cur, plan, lds, x);
    half8 xb[4][S::KS0];
    to_b16<S::KS0, S::F / 2>(x, xb);
    __builtin_amdgcn_sched_barrier(0);
    half8 h[4][S::KSH];
    if constexpr (!kStageAfterLayer0) write_staged<NL, CH>(plan_next, sd, lds, wave_w);
    mlp16_layer0<NL, CH, PE, HID, NH, LEAKY>(lds, xb, h, a.slope_h2);
    // the region is free now (this tile's taps are read): the next tile's quads go in
    if constexpr (kStageAfterLayer0) write_staged<NL, CH>(plan_next, sd, lds, wave_w);
    floatx4 y[4];
    mlp16_rest<NL, CH, PE, HID, NH, LEAKY>(lds, h, y, a.slope_h2);
    const float *ob = (const float *)lds + image16_of<NL, CH, PE, HID>(NH).bias_off + HID * (1 + NH);
    pending = finish16<WIDE>(y, ob, cur.q, cur.valid);
    __builtin_amdgcn_sched_barrier(0);
    if (g1.n && g1.d != staged_dec) {
      restage(g1.d);
      staged_dec = g1.d;
    }
    cur = nxt;
    plan = plan_next;
    g0 = g1;
    g1 = g2;
    g2 = g3;
    g3 = next_group<WAVES>(a, g3, D, t_end);
  };
  Query q_b;
  Slot p_b;
  for (;;) {
    if (!g0.n) break;
    tile(q_next, p_next, q_b, p_b);
    if (!g0.n) break;
    tile(q_b, p_b, q_next, p_next);
  }
  store_out16<STORE, WIDE>(out_rsrc, a.out_dim, pending, a.out_f16);
}

// LDS bytes of a decode_binned16 workgroup: the decoder image (16-byte
// aligned), then every wave's staging region.
template <int NL, int CH, int PE, int HID, int NH>
inline size_t binned16_lds_bytes(uint32_t *image_bytes) {
  const Image im = image16_of<NL, CH, PE, HID>(NH);
  const uint32_t ib = ((uint32_t)im.bytes + 15u) & ~15u;
  if (image_bytes) *image_bytes = ib;
  return (size_t)ib + (size_t)kWaves16<HID> * Staging<CH>::template bytes<NL>();
}

template <int NL, int CH, int PE, int HID, int NH, int STORE, bool LEAKY>
int launch_binned16(const DecodeArgs &a, hipStream_t stream) {
  uint32_t image_bytes = 0;
  const size_t lds = binned16_lds_bytes<NL, CH, PE, HID, NH>(&image_bytes);
  const void *fn = (const void *)decode_binned16<NL, CH, PE, HID, NH, STORE, LEAKY>;
  if (lds > 64 * 1024 &&
      hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
    return NTC_ERR_HIP;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  constexpr int threads = kThreads16<HID>;
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  const uint64_t cap = (uint64_t)cus * (uint64_t)per_cu;
  uint64_t blocks = ((uint64_t)a.max_tiles + kWaves16<HID> - 1) / kWaves16<HID>;
  if (blocks > cap) blocks = cap;
  if (blocks == 0) return NTC_OK;
  hipLaunchKernelGGL((decode_binned16<NL, CH, PE, HID, NH, STORE, LEAKY>), dim3((unsigned)blocks),
                     dim3(threads), lds, stream, a, image_bytes);
  return hip_status(hipGetLastError());
}

}  // namespace
}  // namespace ntc
