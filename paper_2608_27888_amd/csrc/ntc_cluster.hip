// ntc_cluster.hip -- Stage 2 of the paper's texture pipeline (Alg. "Overall
// texture processing pipeline"): k-means clustering of one feature vector per
// texture into m groups; the group labels are the texture -> decoder map c(i)
// that the decode path reads.  The paper clusters CLIP embeddings (Stage 1);
// any per-texture features can be given.
//
// Lloyd's algorithm in fp64, run for up to max_iter iterations without host
// synchronisation: iteration t is an assignment launch and an update launch,
// and a per-iteration flag lets every launch after convergence return at once.
//   seed   : centroid j = features of texture init[j]; flags cleared.
//   assign : one wave per texture; squared Euclidean distance to each
//            centroid (lanes stride the dimensions, butterfly sum, so every
//            lane holds the same bits), nearest centroid with ties to the lower
//            index; flags[t] = 1 if any label changed (always at t = 0).
//   update : one workgroup per cluster; if nothing changed at t, return;
//            otherwise each dimension sums its members in ascending texture
//            order and divides by the count; an empty cluster keeps its
//            centroid.  Sizes k_g go to counts[j].
#include "ntc_internal.h"

namespace ntc {
namespace {

__global__ void __launch_bounds__(kBlock)
kmeans_seed(const float *__restrict__ features, int32_t dim, const uint32_t *__restrict__ init,
            double *__restrict__ centroids, uint32_t *__restrict__ flags, int32_t max_iter) {
  const uint32_t j = blockIdx.x;
  const float *x = features + (size_t)init[j] * dim;
  for (int k = threadIdx.x; k < dim; k += kBlock) centroids[(size_t)j * dim + k] = (double)x[k];
  if (j == 0)
    for (int t = threadIdx.x; t < max_iter; t += kBlock) flags[t] = 0;
}

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int s = 1; s < kWave; s <<= 1) v += __shfl_xor(v, s, kWave);
  return v;
}

__global__ void __launch_bounds__(kBlock)
kmeans_assign(const float *__restrict__ features, int32_t n, int32_t dim, int32_t m,
              const double *__restrict__ centroids, uint32_t *__restrict__ assign,
              uint32_t *__restrict__ flags, int32_t t) {
  if (t > 0 && flags[t - 1] == 0) return;  // converged at an earlier iteration
  const uint32_t i = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave, lane = lane_id();
  if (i >= (uint32_t)n) return;
  const float *x = features + (size_t)i * dim;
  double best = __builtin_inf();
  uint32_t bj = 0;
  for (int j = 0; j < m; ++j) {
    const double *c = centroids + (size_t)j * dim;
    double s = 0.0;
    for (int k = lane; k < dim; k += kWave) {
      const double d = (double)x[k] - c[k];
      s = __builtin_fma(d, d, s);
    }
    s = wave_sum(s);
    if (s < best) {
      best = s;
      bj = (uint32_t)j;
    }
  }
  if (lane == 0) {
    if (t == 0 || assign[i] != bj) flags[t] = 1u;
    assign[i] = bj;
  }
}

__global__ void __launch_bounds__(kBlock)
kmeans_update(const float *__restrict__ features, int32_t n, int32_t dim,
              const uint32_t *__restrict__ assign, double *__restrict__ centroids,
              uint32_t *__restrict__ counts, const uint32_t *__restrict__ flags, int32_t t) {
  if (flags[t] == 0) return;  // no label changed: the centroids stand
  const uint32_t j = blockIdx.x;
  for (int k0 = 0; k0 < dim; k0 += kBlock) {  // uniform trip count: every thread counts
    const int k = k0 + (int)threadIdx.x;
    double s = 0.0;
    uint32_t cnt = 0;
    for (int i = 0; i < n; ++i) {
      if (assign[i] == j) {
        if (k < dim) s += (double)features[(size_t)i * dim + k];
        ++cnt;
      }
    }
    if (cnt && k < dim) centroids[(size_t)j * dim + k] = s / (double)cnt;
    if (k0 == 0 && threadIdx.x == 0) counts[j] = cnt;
  }
}

}  // namespace

size_t kmeans_workspace_bytes(int32_t m, int32_t max_iter) {
  return ((size_t)m + (size_t)max_iter) * sizeof(uint32_t);
}

int launch_kmeans(const float *features, int32_t n, int32_t dim, int32_t m, const uint32_t *init,
                  int32_t max_iter, uint32_t *assign, double *centroids, uint32_t *counts,
                  void *workspace, hipStream_t stream) {
  uint32_t *dinit = (uint32_t *)workspace;  // [m] seed textures, then [max_iter] flags
  uint32_t *flags = dinit + m;
  // the seed list is the caller's host memory: it is read before this call returns
  if (hipMemcpyAsync(dinit, init, (size_t)m * sizeof(uint32_t), hipMemcpyHostToDevice, stream) !=
          hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return NTC_ERR_HIP;
  hipLaunchKernelGGL(kmeans_seed, dim3((unsigned)m), dim3(kBlock), 0, stream, features, dim, dinit,
                     centroids, flags, max_iter);
  const unsigned assign_blocks = (unsigned)((n + kWavesPerBlock - 1) / kWavesPerBlock);
  for (int32_t t = 0; t < max_iter; ++t) {
    hipLaunchKernelGGL(kmeans_assign, dim3(assign_blocks), dim3(kBlock), 0, stream, features, n,
                       dim, m, centroids, assign, flags, t);
    hipLaunchKernelGGL(kmeans_update, dim3((unsigned)m), dim3(kBlock), 0, stream, features, n, dim,
                       assign, centroids, counts, flags, t);
  }
  return hip_status(hipGetLastError());
}

int read_kmeans_state(const void *workspace, int32_t m, int32_t max_iter, int32_t *iterations,
                      int32_t *converged, hipStream_t stream) {
  const uint32_t *flags = (const uint32_t *)workspace + m;
  uint32_t buf[64];
  int32_t done = max_iter, conv = 0;
  for (int32_t t0 = 0; t0 < max_iter && !conv; t0 += 64) {
    const int32_t len = max_iter - t0 < 64 ? max_iter - t0 : 64;
    hipError_t e = hipMemcpyAsync(buf, flags + t0, (size_t)len * sizeof(uint32_t),
                                  hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess) e = hipStreamSynchronize(stream);
    if (e != hipSuccess) return NTC_ERR_HIP;
    for (int32_t k = 0; k < len; ++k) {
      if (buf[k] == 0) {
        done = t0 + k + 1;
        conv = 1;
        break;
      }
    }
  }
  if (iterations) *iterations = done;
  if (converged) *converged = conv;
  return NTC_OK;
}

}  // namespace ntc
