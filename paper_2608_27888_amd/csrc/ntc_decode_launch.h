// ntc_decode_launch.h -- launches of the decode kernels of one decoder shape
// family: the kernel chosen by mode (binned, stream, per-wave stream), output
// store mode and activation.  Included by the per-family translation units.
#pragma once

#include "ntc_decode16.h"

namespace ntc {
namespace {

template <int NL, int CH, int PE, int HID, int NH, bool MIP, int STORE, bool LEAKY>
int launch_shape(const DecodeArgs &a, hipStream_t stream) {
  const Image im = image_of<NL, CH, PE, HID>(NH);
  const size_t lds = (size_t)im.bytes;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess)
    (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (!a.bin_offset && a.n_decoders > 1 && a.dec_stride % 8 == 0 &&
      ((uintptr_t)a.params & 15) == 0) {
    // stream mode over several decoders, every block 16-byte aligned: a shared staged
    // decoder where a whole group agrees on one, per-wave fragment reads elsewhere
    constexpr int waves = kWaves<HID, false>, threads = waves * kWave;
    const uint32_t image_bytes = ((uint32_t)im.bytes + 15u) & ~15u;
    const size_t mlds = image_bytes + (size_t)waves * (HID * (1 + NH) + 32) * sizeof(float);
    const void *fm = (const void *)decode_stream_mixed<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>;
    if (mlds > 64 * 1024 &&
        hipFuncSetAttribute(fm, hipFuncAttributeMaxDynamicSharedMemorySize, (int)mlds) != hipSuccess)
      return NTC_ERR_HIP;
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fm, threads, mlds) != hipSuccess ||
        per_cu < 1)
      per_cu = 1;
    const uint64_t tiles = ((uint64_t)a.n + kWave - 1) / kWave;
    uint64_t blocks = (tiles + waves - 1) / waves;
    if (blocks > (uint64_t)cus * per_cu) blocks = (uint64_t)cus * per_cu;
    if (blocks == 0) return NTC_OK;
    hipLaunchKernelGGL((decode_stream_mixed<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>),
                       dim3((unsigned)blocks), dim3(threads), mlds, stream, a, image_bytes);
    return hip_status(hipGetLastError());
  }
  if (a.gather == NTC_GATHER_STAGED) {
    // the LDS-staged gather: binned, no mip blending, 2 levels, widths up to 8
    // (checked by the caller)
    if constexpr (!MIP && NL == 2)
      if (a.bin_offset && a.out_dim <= 8) return launch_binned16<NL, CH, PE, HID, NH, STORE, LEAKY>(a, stream);
    return NTC_ERR_UNSUPPORTED;
  }
  const void *fn = a.bin_offset ? (const void *)decode_binned<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>
                                : (const void *)decode_stream<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>;
  if (lds > 64 * 1024) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return NTC_ERR_HIP;
  }
  // every workgroup resident at once: one round, no tail of late workgroups
  int per_cu = 0;
  const bool binned = a.bin_offset != nullptr;
  const int waves = binned ? kWaves<HID, true> : kWaves<HID, false>;
  const int threads = waves * kWave;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, lds) != hipSuccess ||
      per_cu < 1)
    per_cu = 1;
  const uint64_t cap = (uint64_t)cus * (uint64_t)per_cu;
  const uint64_t tiles = a.bin_offset ? (uint64_t)a.max_tiles : ((uint64_t)a.n + kWave - 1) / kWave;
  uint64_t blocks = (tiles + waves - 1) / waves;
  if (blocks > cap) blocks = cap;
  if (blocks == 0) return NTC_OK;
  if (a.bin_offset) {
    // two workgroups on every CU: the first dispatched to a CU takes two
    // thirds of the CU's tiles (measured 3-4 % less time on the 4K clustered
    // frame than equal ranges; 3:1 is slower again)
    DecodeArgs b = a;
    b.split = per_cu == 2 && blocks == cap && blocks % 16 == 0 ? 1u : 0u;
    hipLaunchKernelGGL((decode_binned<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>), dim3((unsigned)blocks),
                       dim3(threads), lds, stream, b);
  } else
    hipLaunchKernelGGL((decode_stream<NL, CH, PE, HID, NH, MIP, STORE, LEAKY>), dim3((unsigned)blocks),
                       dim3(threads), lds, stream, a);
  return hip_status(hipGetLastError());
}

template <int NL, int CH, int PE, int HID, int NH, bool MIP, bool LEAKY>
int launch_store(const DecodeArgs &a, hipStream_t stream) {
  if (a.out_dim == 3)
    return a.out_f16 ? launch_shape<NL, CH, PE, HID, NH, MIP, kStoreF16x3, LEAKY>(a, stream)
                     : launch_shape<NL, CH, PE, HID, NH, MIP, kStoreF32x3, LEAKY>(a, stream);
  if (a.out_dim != 4 && a.out_dim != 8)
    return launch_shape<NL, CH, PE, HID, NH, MIP, kStoreEach, LEAKY>(a, stream);
  return a.out_f16 ? launch_shape<NL, CH, PE, HID, NH, MIP, kStoreF16x4, LEAKY>(a, stream)
                   : launch_shape<NL, CH, PE, HID, NH, MIP, kStoreF32x4, LEAKY>(a, stream);
}

template <int NL, int CH, int PE, int HID, int NH, bool MIP>
int launch_act(const DecodeArgs &a, hipStream_t stream) {
  return a.leaky ? launch_store<NL, CH, PE, HID, NH, MIP, true>(a, stream)
                 : launch_store<NL, CH, PE, HID, NH, MIP, false>(a, stream);
}

// Positional-encoding kernels exist for the Sec. 4 setup's decoder only: one
// hidden -> hidden layer, no mip blending.
template <int NL, int CH, int PE, int HID, int NH>
int launch_mip(const DecodeArgs &a, hipStream_t stream) {
  if constexpr (PE > 0) {
    return a.mip ? NTC_ERR_UNSUPPORTED : launch_act<NL, CH, PE, HID, NH, false>(a, stream);
  } else {
    return a.mip ? launch_act<NL, CH, PE, HID, NH, true>(a, stream)
                 : launch_act<NL, CH, PE, HID, NH, false>(a, stream);
  }
}

template <int NL, int CH, int PE, int HID>
int launch_hidden(const DecodeArgs &a, hipStream_t stream) {
  switch (a.n_hidden) {
    case 1: return launch_mip<NL, CH, PE, HID, 1>(a, stream);
    case 2:
      if constexpr (PE > 0) return NTC_ERR_UNSUPPORTED;
      else return launch_mip<NL, CH, PE, HID, 2>(a, stream);
    default: return NTC_ERR_UNSUPPORTED;
  }
}

}  // namespace

// One decoder shape family: every kernel variant (hidden layers, mip, store
// mode, activation) of the MFMA engine, and of the FMA engine.  Each family
// is instantiated in a translation unit of its own so that they compile in
// parallel.
template <int NL, int CH, int PE, int HID>
int launch_decode_shape(const DecodeArgs &a, hipStream_t stream) {
  return launch_hidden<NL, CH, PE, HID>(a, stream);
}

template <int NL, int CH, int PE, int HID>
int launch_decode_fma_shape(const DecodeArgs &a, hipStream_t stream) {
  return launch_fma_mip<NL, CH, PE, HID>(a, stream);
}

}  // namespace ntc
