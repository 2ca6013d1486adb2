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

// Rademacher update. sum_n c_n z_n[j] with z = +-1 is, for each group of 8
// probes, a table lookup: T_g[m] = sum over the group of (bit n of m ? +c_n :
// -c_n) for the 256 sign patterns m (built once per workgroup and group).
// A workgroup owns 8192 consecutive parameters (256 Philox words per probe);
// each thread loads its 4 sets of 8 parameters up front (four 16-byte loads
// in flight per thread), then for each group of up to 16 probes the
// workgroup computes their Philox blocks into LDS (4 per thread), and each
// thread takes, for each set of 8 parameters, one byte of sign bits from
// each of 8 probes, transposes that 8x8 bit block (three swap stages) so that
// byte e holds parameter e's signs, and adds one table entry per parameter
// and group of 8. theta is read and written once.
constexpr int kUpdChunk = 8192;   // parameters per workgroup (32 per thread, 4 sets of 8)
constexpr int kUpdWords = kUpdChunk / 32;
constexpr int kUpdGroup = 16;     // probes per pass over the LDS tables

// 8x8 bit transpose of the bytes of (lo, hi) (byte j = row j): byte e of the
// result holds bit e of every input byte.
__device__ __forceinline__ void transpose8x8(uint32_t& lo, uint32_t& hi) {
  uint32_t t;
  t = (lo ^ (lo >> 7)) & 0x00AA00AAu;
  lo = lo ^ t ^ (t << 7);
  t = (hi ^ (hi >> 7)) & 0x00AA00AAu;
  hi = hi ^ t ^ (t << 7);
  t = (lo ^ (lo >> 14)) & 0x0000CCCCu;
  lo = lo ^ t ^ (t << 14);
  t = (hi ^ (hi >> 14)) & 0x0000CCCCu;
  hi = hi ^ t ^ (t << 14);
  t = (lo ^ (hi << 4)) & 0xF0F0F0F0u;
  lo = lo ^ t;
  hi = hi ^ (t >> 4);
}

template <typename T>
__device__ __forceinline__ void load8(const T* theta, uint64_t j, uint64_t P, float v[8]) {
  if (j + 8 <= P) {
    if constexpr (sizeof(T) == 2) {
      const uint4 q = *(const uint4*)(theta + j);
      const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = bf16_to_f32((uint16_t)w[e]);
        v[2 * e + 1] = bf16_to_f32((uint16_t)(w[e] >> 16));
      }
    } else {
      const float4 a = *(const float4*)(theta + j), b = *(const float4*)(theta + j + 4);
      v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
      v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
  } else {
    load4(theta, j, P, v);
    load4(theta, j + 4, P, v + 4);
  }
}

template <typename T>
__device__ __forceinline__ void store8(T* theta, uint64_t j, uint64_t P, const float v[8]) {
  if (j + 8 <= P) {
    if constexpr (sizeof(T) == 2) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = (uint32_t)bf16_rne(v[2 * e]) | ((uint32_t)bf16_rne(v[2 * e + 1]) << 16);
      *(uint4*)(theta + j) = uint4{w[0], w[1], w[2], w[3]};
    } else {
      *(float4*)(theta + j) = float4{v[0], v[1], v[2], v[3]};
      *(float4*)(theta + j + 4) = float4{v[4], v[5], v[6], v[7]};
    }
  } else {
    store4(theta, j, P, v);
    store4(theta, j + 4, P, v + 4);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void update_rademacher_kernel(T* theta, uint64_t P, Key key,
                                                                float eps, float lr, int N,
                                                                uint32_t i0, const float* Lp,
                                                                const float* Lm, int32_t* skipped) {
  // sign words laid out [word][probe] (rows padded by 4 words) so that one
  // thread reads 8 probes' words of its parameters with two 128-bit loads
  constexpr int kRow = kUpdGroup + 4;
  constexpr int kSets = kUpdChunk / (8 * 256);
  __shared__ uint32_t words[kUpdWords * kRow];     // 20 KiB
  __shared__ float table[kUpdGroup / 8][256];      // signed-sum tables
  __shared__ float half_table[kUpdGroup / 8][32];  // 4-probe partial sums
  __shared__ float coef[kUpdGroup];
  __shared__ int flag;
  const bool ok = losses_finite(Lp, Lm, N, &flag);
  if (blockIdx.x == 0 && threadIdx.x == 0 && skipped) *skipped = ok ? 0 : 1;
  if (!ok) return;
  const int t = threadIdx.x;
  const uint64_t base = (uint64_t)blockIdx.x * kUpdChunk;
  float th[kSets][8];
#pragma unroll
  for (int q = 0; q < kSets; ++q) load8(theta, base + 2048u * q + 8u * t, P, th[q]);
  float acc[kSets][8];
#pragma unroll
  for (int q = 0; q < kSets; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[q][e] = 0.f;
  const uint32_t k = (uint32_t)(t & 3);  // this thread's byte within each of its words
  // byte-gather selectors for v_perm: byte k of the low and high source -> bytes 0, 1
  const uint32_t sel = k | ((4u + k) << 8) | 0x0C0C0000u;
  for (int n0 = 0; n0 < N; n0 += kUpdGroup) {
    const int cnt = N - n0 < kUpdGroup ? N - n0 : kUpdGroup;
    const int ngroups = (cnt + 7) / 8;
    __syncthreads();
    if (t < kUpdGroup) coef[t] = t < cnt ? update_coeff(lr, N, Lp[n0 + t], Lm[n0 + t], eps) : 0.f;
    // Philox blocks: cnt probes x 64 blocks (probes past cnt only ever meet zero coefficients)
    for (int q = t; q < cnt * (kUpdWords / 4); q += 256) {
      const int pn = q / (kUpdWords / 4), pb = q % (kUpdWords / 4);
      const Words x = stream_block(key, (base >> 7) + pb, i0 + (uint32_t)(n0 + pn), kTagRademacher);
#pragma unroll
      for (int w = 0; w < 4; ++w) words[(4 * pb + w) * kRow + pn] = x.w[w];
    }
    __syncthreads();
    // 4-probe partial tables, then T[m] = low[m & 15] + high[m >> 4]
    if (t < ngroups * 32) {
      const int g = t >> 5, h = (t >> 4) & 1, m = t & 15;
      float v = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float c = coef[8 * g + 4 * h + b];
        v += ((m >> b) & 1) ? c : -c;
      }
      half_table[g][16 * h + m] = v;
    }
    __syncthreads();
    for (int q = t; q < ngroups * 256; q += 256) {
      const int g = q >> 8, m = q & 255;
      table[g][m] = half_table[g][m & 15] + half_table[g][16 + (m >> 4)];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < kSets; ++q) {
      const uint32_t* wrow = words + (64 * q + (t >> 2)) * kRow;
      for (int g = 0; g < ngroups; ++g) {
        const uint4 a = *(const uint4*)(wrow + 8 * g);
        const uint4 b = *(const uint4*)(wrow + 8 * g + 4);
        // byte k of each of the 8 probes' words, probe order, into (lo, hi)
        uint32_t lo = __builtin_amdgcn_perm(a.y, a.x, sel) | (__builtin_amdgcn_perm(a.w, a.z, sel) << 16);
        uint32_t hi = __builtin_amdgcn_perm(b.y, b.x, sel) | (__builtin_amdgcn_perm(b.w, b.z, sel) << 16);
        transpose8x8(lo, hi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[q][e] += table[g][(lo >> (8 * e)) & 0xFFu];
          acc[q][4 + e] += table[g][(hi >> (8 * e)) & 0xFFu];
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < kSets; ++q) {
    float out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = th[q][e] - acc[q][e];
    store8(theta, base + 2048u * q + 8u * t, P, out);
  }
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
