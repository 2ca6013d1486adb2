// Probe dump, initialisation and the parameter update of the CD-RGE step.
#include <hip/hip_runtime.h>

#include "zo_kernels.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

__global__ __launch_bounds__(256) void debug_probe_kernel(int kind, Key key, uint32_t i,
                                                          uint64_t j0, uint64_t n, float* out) {
  const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n) return;
  out[t] = probe_value(kind, key, i, j0 + t);
}

__global__ __launch_bounds__(256) void debug_gauss_kernel(const uint32_t* words, uint64_t n_pairs,
                                                          float* out) {
  const uint64_t p = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n_pairs) return;
  float z0, z1;
  gauss_pair(words[2 * p], words[2 * p + 1], z0, z1);
  out[2 * p] = z0;
  out[2 * p + 1] = z1;
}

// theta_j ~ U(-1/sqrt(H), 1/sqrt(H)); one Philox block (tag 2) per 4 elements.
template <typename T>
__global__ __launch_bounds__(256) void init_kernel(T* theta, uint64_t P, Key key, float scale) {
  const uint64_t blk = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint64_t j0 = blk << 2;
  if (j0 >= P) return;
  const Words x = stream_block(key, blk, 0u, kTagInit);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (j0 + e < P) {
      const float v = init_value(x.w[e], scale);
      if constexpr (sizeof(T) == 2) theta[j0 + e] = bf16_rne(v);
      else theta[j0 + e] = v;
    }
  }
}

// Eq. 7 step size of probe n: fp32 of (lr / N) * (L+ - L-) / (2 eps), in double.
__device__ __forceinline__ float update_coeff(float lr, int N, float lp, float lm, float eps) {
  const double c = ((double)lr / (double)N) * (((double)lp - (double)lm) / (2.0 * (double)eps));
  return (float)c;
}

// Workgroup-wide check that every loss is finite (all workgroups agree).
__device__ bool losses_finite(const float* Lp, const float* Lm, int N, int* flag) {
  if (threadIdx.x == 0) *flag = 0;
  __syncthreads();
  int bad = 0;
  for (int n = threadIdx.x; n < N; n += blockDim.x)
    bad |= !(isfinite(Lp[n]) && isfinite(Lm[n]));
  if (bad) atomicOr(flag, 1);
  __syncthreads();
  return *flag == 0;
}

template <typename T>
__device__ __forceinline__ void load4(const T* theta, uint64_t j, uint64_t P, float v[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] = 0.0f;
    if (j + e < P) {
      if constexpr (sizeof(T) == 2) v[e] = bf16_to_f32(theta[j + e]);
      else v[e] = theta[j + e];
    }
  }
}

template <typename T>
__device__ __forceinline__ void store4(T* theta, uint64_t j, uint64_t P, const float v[4]) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (j + e < P) {
      if constexpr (sizeof(T) == 2) theta[j + e] = bf16_rne(v[e]);
      else theta[j + e] = v[e];
    }
  }
}

// Rademacher update. A workgroup owns 1024 consecutive parameters (8 Philox
// blocks per probe); for each group of 32 probes every thread computes one
// Philox block into LDS, then each thread applies the 32 signed step sizes to
// its 4 parameters in ascending probe order.
constexpr int kUpdChunk = 1024;

template <typename T>
__global__ __launch_bounds__(256) void update_rademacher_kernel(T* theta, uint64_t P, Key key,
                                                                float eps, float lr, int N,
                                                                uint32_t i0, const float* Lp,
                                                                const float* Lm, int32_t* skipped) {
  __shared__ uint32_t words[32][8][4];
  __shared__ float coef[32];
  __shared__ int flag;
  const bool ok = losses_finite(Lp, Lm, N, &flag);
  if (blockIdx.x == 0 && threadIdx.x == 0 && skipped) *skipped = ok ? 0 : 1;
  if (!ok) return;
  const int t = threadIdx.x;
  const uint64_t base = (uint64_t)blockIdx.x * kUpdChunk;
  const uint64_t j = base + 4u * (uint64_t)t;
  float th[4];
  load4(theta, j, P, th);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  const int wsel_blk = t >> 5;        // which of the 8 blocks holds this thread's elements
  const int wsel_word = (t >> 3) & 3;  // which word of that block
  const int shift = (t & 7) * 4;       // bit position of the first of the 4 elements
  for (int n0 = 0; n0 < N; n0 += 32) {
    __syncthreads();
    {
      const int pn = t >> 3, pb = t & 7;
      if (n0 + pn < N) {
        const Words x = stream_block(key, (base >> 7) + pb, i0 + (uint32_t)(n0 + pn), kTagRademacher);
#pragma unroll
        for (int w = 0; w < 4; ++w) words[pn][pb][w] = x.w[w];
      }
      if (t < 32 && n0 + t < N) coef[t] = update_coeff(lr, N, Lp[n0 + t], Lm[n0 + t], eps);
    }
    __syncthreads();
    const int cnt = N - n0 < 32 ? N - n0 : 32;
    for (int pn = 0; pn < cnt; ++pn) {
      const uint32_t w = words[pn][wsel_blk][wsel_word] >> shift;
      const float c = coef[pn];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[e] += ((w >> e) & 1u) ? c : -c;
    }
  }
  float out[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = th[e] - acc[e];
  store4(theta, j, P, out);
}

// Normal-probe update: each thread owns one Philox block (4 parameters) and
// regenerates its 4 values of every probe in ascending order.
template <typename T>
__global__ __launch_bounds__(256) void update_gaussian_kernel(T* theta, uint64_t P, Key key,
                                                              float eps, float lr, int N,
                                                              uint32_t i0, const float* Lp,
                                                              const float* Lm, int32_t* skipped) {
  __shared__ float coef[256];
  __shared__ int flag;
  const bool ok = losses_finite(Lp, Lm, N, &flag);
  if (blockIdx.x == 0 && threadIdx.x == 0 && skipped) *skipped = ok ? 0 : 1;
  if (!ok) return;
  const int t = threadIdx.x;
  const uint64_t blk = (uint64_t)blockIdx.x * blockDim.x + t;
  const uint64_t j = blk << 2;
  float th[4];
  load4(theta, j, P, th);
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int n0 = 0; n0 < N; n0 += 256) {
    __syncthreads();
    if (n0 + t < N) coef[t] = update_coeff(lr, N, Lp[n0 + t], Lm[n0 + t], eps);
    __syncthreads();
    const int cnt = N - n0 < 256 ? N - n0 : 256;
    if (j < P) {
      for (int pn = 0; pn < cnt; ++pn) {
        float z[4];
        gauss_block(key, i0 + (uint32_t)(n0 + pn), blk, z);
        const float c = coef[pn];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[e] = fmaf(c, z[e], acc[e]);
      }
    }
  }
  float out[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = th[e] - acc[e];
  store4(theta, j, P, out);
}

}  // namespace

hipError_t launch_debug_probe(int kind, uint64_t seed, uint32_t i, uint64_t j0, uint64_t n,
                              float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const uint64_t grid = (n + 255) / 256;
  debug_probe_kernel<<<dim3((unsigned)grid), dim3(256), 0, s>>>(kind, make_key(seed), i, j0, n, out);
  return hipGetLastError();
}

hipError_t launch_debug_gauss_pairs(const uint32_t* words, uint64_t n_pairs, float* out,
                                    hipStream_t s) {
  if (n_pairs == 0) return hipSuccess;
  const uint64_t grid = (n_pairs + 255) / 256;
  debug_gauss_kernel<<<dim3((unsigned)grid), dim3(256), 0, s>>>(words, n_pairs, out);
  return hipGetLastError();
}

hipError_t launch_init(int wdtype, void* theta, uint64_t P, uint64_t seed, float scale,
                       hipStream_t s) {
  const uint64_t grid = ((P + 3) / 4 + 255) / 256;
  if (wdtype == ZO_WBF16)
    init_kernel<uint16_t><<<dim3((unsigned)grid), dim3(256), 0, s>>>((uint16_t*)theta, P, make_key(seed), scale);
  else
    init_kernel<float><<<dim3((unsigned)grid), dim3(256), 0, s>>>((float*)theta, P, make_key(seed), scale);
  return hipGetLastError();
}

hipError_t launch_update(int wdtype, int kind, void* theta, uint64_t P, uint64_t seed, float eps,
                         float lr, int32_t N, uint32_t i0, const float* Lp, const float* Lm,
                         int32_t* skipped, hipStream_t s) {
  const Key key = make_key(seed);
  ProfScope ps(kKUpdate, s);
  if (kind == ZO_RADEMACHER) {
    const uint64_t grid = (P + kUpdChunk - 1) / kUpdChunk;
    if (wdtype == ZO_WBF16)
      update_rademacher_kernel<uint16_t><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (uint16_t*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped);
    else
      update_rademacher_kernel<float><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (float*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped);
  } else {
    const uint64_t grid = ((P + 3) / 4 + 255) / 256;
    if (wdtype == ZO_WBF16)
      update_gaussian_kernel<uint16_t><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (uint16_t*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped);
    else
      update_gaussian_kernel<float><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (float*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped);
  }
  return hipGetLastError();
}

}  // namespace zo
