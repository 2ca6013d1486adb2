// Probe dump, initialisation and the parameter update of the CD-RGE step.
#include <hip/hip_runtime.h>

#include <type_traits>

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
__device__ bool losses_finite(const float* Lp, const float* Lm, int N, int lm_stride, int* flag) {
  if (threadIdx.x == 0) *flag = 0;
  __syncthreads();
  int bad = 0;
  for (int n = threadIdx.x; n < N; n += blockDim.x)
    bad |= !(isfinite(Lp[n]) && isfinite(Lm[n * lm_stride]));
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

// Rademacher update for any N (the kernel below takes N <= 16, the common
// case, faster). sum_n c_n z_n[j] with z = +-1 is, for each group of 8
// probes, a table lookup: T_g[m] = sum over the group of (bit n of m ? +c_n :
// -c_n) for the 256 sign patterns m. Persistent workgroups (as many as fit
// at once) walk chunks of 8192 consecutive parameters (256 Philox words per
// probe); a thread owns 4 sets of 8 parameters of a chunk, and the next
// chunk's theta loads are issued when the current chunk starts, so they run
// during its probe work. With at most 16 probes the coefficients and tables
// are built once per workgroup. Per chunk and group of up to 16 probes, the
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

// Two fp32 values to packed bf16 (round to nearest even) with one
// v_cvt_pk_bf16_f32; the same rounding as bf16_rne for finite values.
__device__ __forceinline__ uint32_t pack_bf16x2_rne(float lo, float hi) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  typedef float f2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){lo, hi}, bf2));
}

template <typename T>
__device__ __forceinline__ void store8(T* theta, uint64_t j, uint64_t P, const float v[8]) {
  if (j + 8 <= P) {
    if constexpr (sizeof(T) == 2) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2_rne(v[2 * e], v[2 * e + 1]);
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

// Eight parameters j .. j + 7 as stored (bf16 or fp32 bit patterns; zeros
// past P). Whole-workgroup chunks inside theta take plain 16-byte loads
// with no bounds checks, so that a thread's loads issue back to back.
template <typename T>
struct Raw8 {
  uint4 w[8 * sizeof(T) / 16];
};
template <typename T>
__device__ __forceinline__ Raw8<T> load_raw8(const T* theta, uint64_t j, uint64_t P, bool full) {
  Raw8<T> r;
  constexpr int kW = 8 * sizeof(T) / 16, kPer = 16 / sizeof(T);
  if (full) {
#pragma unroll
    for (int w = 0; w < kW; ++w) r.w[w] = *(const uint4*)(theta + j + (uint64_t)w * kPer);
  } else {
    T v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = j + e < P ? theta[j + e] : (T)0;
    __builtin_memcpy(&r, v, sizeof(v));
  }
  return r;
}
template <typename T>
__device__ __forceinline__ void decode_raw8(const Raw8<T>& r, float v[8]) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t x = w == 0 ? r.w[0].x : w == 1 ? r.w[0].y : w == 2 ? r.w[0].z : r.w[0].w;
      v[2 * w] = bf16_to_f32((uint16_t)x);
      v[2 * w + 1] = bf16_to_f32((uint16_t)(x >> 16));
    }
  } else {
    __builtin_memcpy(v, &r, 32);
  }
}

// The 4 sign words of Philox block blk of probe n from the sign-probe cache
// (layout: bit_words; its words are stored unshuffled, so they are shuffled
// back into the generator's order); zeros past the parameters, as their signs
// only ever meet parameters that are not stored.
__device__ __forceinline__ Words cached_block(const uint32_t* bits, uint64_t P, int n, uint64_t blk) {
  if (blk >= (P + 127) / 128) return Words{{0u, 0u, 0u, 0u}};
  const uint4 v = *(const uint4*)(bits + (uint64_t)n * bit_words(P) + 4 * blk);
  return Words{{sign_word_shuffle(v.x), sign_word_shuffle(v.y), sign_word_shuffle(v.z), sign_word_shuffle(v.w)}};
}

// Workgroup barrier for LDS data only: waits for this thread's LDS accesses
// (lgkmcnt(0)), not for its global loads, which stay in flight across it.
// The empty asm statements keep the compiler from moving memory accesses
// across the barrier.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt, expcnt at their maxima; lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <typename T, bool kBits>
__global__ __launch_bounds__(256) void update_rademacher_kernel(T* __restrict__ theta, uint64_t P, Key key,
                                                                float eps, float lr, int N, uint32_t i0,
                                                                const float* __restrict__ Lp,
                                                                const float* __restrict__ Lm,
                                                                int32_t* __restrict__ skipped,
                                                                uint64_t nchunks, int lm_stride,
                                                                const uint32_t* __restrict__ bits) {
  // sign words laid out [word][probe] (rows padded by 4 words) so that one
  // thread reads 8 probes' words of its parameters with two 128-bit loads
  constexpr int kRow = kUpdGroup + 4;
  constexpr int kSets = kUpdChunk / (8 * 256);
  __shared__ uint32_t words[kUpdWords * kRow];     // 20 KiB
  __shared__ float table[kUpdGroup / 8][256];      // signed-sum tables
  __shared__ float half_table[kUpdGroup / 8][32];  // 4-probe partial sums
  __shared__ float coef[kUpdGroup];
  __shared__ int bad;  // some loss is not finite
  const int t = threadIdx.x;
  const uint32_t k = (uint32_t)(t & 3);  // this thread's byte within each of its words
  // byte-gather selectors for v_perm: byte k of the low and high source -> bytes 0, 1
  const uint32_t sel = k | ((4u + k) << 8) | 0x0C0C0000u;
  const bool one_group = N <= kUpdGroup;  // coefficients and tables built once

  // The workgroup walks its chunks (8192 parameters each) blockIdx.x,
  // blockIdx.x + gridDim.x, ...; the next chunk's theta loads are issued at
  // the start of the current one, so they run during its probe work.
  auto load_chunk = [&](uint64_t chunk, Raw8<T> (&r)[kSets]) {
    const uint64_t base = chunk * kUpdChunk;
    if (base + kUpdChunk <= P) {  // the same for the whole workgroup
#pragma unroll
      for (int q = 0; q < kSets; ++q) r[q] = load_raw8(theta, base + 2048u * q + 8u * t, P, true);
    } else {
#pragma unroll
      for (int q = 0; q < kSets; ++q) r[q] = load_raw8(theta, base + 2048u * q + 8u * t, P, false);
    }
  };
  // coefficients of probes n0 .. n0 + cnt - 1 into LDS and the finite flag
  // (threads t < cnt; needs a barrier after)
  auto coefficients = [&](int n0, int cnt, float lp, float lm) {
    if (t < kUpdGroup) {
      coef[t] = t < cnt ? update_coeff(lr, N, lp, lm, eps) : 0.f;
      if (t < cnt && !(isfinite(lp) && isfinite(lm))) atomicOr(&bad, 1);
    }
  };
  // signed-sum tables of the current coefficients: 4-probe partial tables,
  // then T[m] = low[m & 15] + high[m >> 4] (two barriers)
  auto tables = [&](int ngroups) {
    if (t < ngroups * 32) {
      const int g = t >> 5, h = (t >> 4) & 1, m = t & 15;
      float v = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const float cb = coef[8 * g + 4 * h + b];
        v += ((m >> b) & 1) ? cb : -cb;
      }
      half_table[g][16 * h + m] = v;
    }
    lds_barrier();
    for (int q = t; q < ngroups * 256; q += 256) {
      const int g = q >> 8, m = q & 255;
      table[g][m] = half_table[g][m & 15] + half_table[g][16 + (m >> 4)];
    }
    lds_barrier();
  };

  // the first group's losses, then the first chunk's theta: loads complete
  // in issue order, so waiting for the losses leaves theta in flight
  float lp = 0.f, lm = 0.f;
  if (t < kUpdGroup && t < N) {
    lp = Lp[t];
    lm = Lm[t * lm_stride];
  }
  uint64_t chunk = blockIdx.x;
  Raw8<T> raw[kSets];
  if (chunk < nchunks) load_chunk(chunk, raw);
  if (t == 0) bad = 0;  // set before the first barrier
  if (one_group) {
    lds_barrier();
    coefficients(0, N, lp, lm);
    lds_barrier();
    tables((N + 7) / 8);
  }
  for (; chunk < nchunks; chunk += gridDim.x) {
    const uint64_t base = chunk * kUpdChunk;
    Raw8<T> next[kSets];
    const uint64_t nxt = chunk + gridDim.x;
    if (nxt < nchunks) load_chunk(nxt, next);
    float acc[kSets][8];
#pragma unroll
    for (int q = 0; q < kSets; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[q][e] = 0.f;
    for (int n0 = 0; n0 < N; n0 += kUpdGroup) {
      const int cnt = N - n0 < kUpdGroup ? N - n0 : kUpdGroup;
      const int ngroups = (cnt + 7) / 8;
      if (!one_group && t < cnt) {
        lp = Lp[n0 + t];
        lm = Lm[(n0 + t) * lm_stride];
      }
      lds_barrier();  // the previous lookups no longer read the words or tables
      if (!one_group) coefficients(n0, cnt, lp, lm);
      // Philox blocks: cnt probes x 64 blocks (probes past cnt only ever meet zero coefficients)
      for (int q = t; q < cnt * (kUpdWords / 4); q += 256) {
        const int pn = q / (kUpdWords / 4), pb = q % (kUpdWords / 4);
        const Words x = kBits ? cached_block(bits, P, n0 + pn, (base >> 7) + pb)
                              : stream_block(key, (base >> 7) + pb, i0 + (uint32_t)(n0 + pn), kTagRademacher);
#pragma unroll
        for (int w = 0; w < 4; ++w) words[(4 * pb + w) * kRow + pn] = x.w[w];
      }
      lds_barrier();
      if (!one_group) tables(ngroups);
      // lookups: for each set of 8 parameters and group of 8 probes, byte k
      // of each probe's word, transposed so that byte e holds parameter e's
      // 8 signs, then one table entry per parameter (groups of a full pass
      // of 16 probes unrolled)
      auto lookup = [&](int q, int g) {
        const uint32_t* wrow = words + (64 * q + (t >> 2)) * kRow + 8 * g;
        const uint4 a = *(const uint4*)(wrow);
        const uint4 b = *(const uint4*)(wrow + 4);
        // byte k of each of the 8 probes' words, probe order, into (lo, hi)
        uint32_t lo = __builtin_amdgcn_perm(a.y, a.x, sel) | (__builtin_amdgcn_perm(a.w, a.z, sel) << 16);
        uint32_t hi = __builtin_amdgcn_perm(b.y, b.x, sel) | (__builtin_amdgcn_perm(b.w, b.z, sel) << 16);
        transpose8x8(lo, hi);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[q][e] += table[g][(lo >> (8 * e)) & 0xFFu];
          acc[q][4 + e] += table[g][(hi >> (8 * e)) & 0xFFu];
        }
      };
      if (ngroups == kUpdGroup / 8) {
#pragma unroll
        for (int q = 0; q < kSets; ++q)
#pragma unroll
          for (int g = 0; g < kUpdGroup / 8; ++g) lookup(q, g);
      } else {
#pragma unroll
        for (int q = 0; q < kSets; ++q)
          for (int g = 0; g < ngroups; ++g) lookup(q, g);
      }
    }
    // a non-finite loss leaves theta untouched (every workgroup decides
    // alike; the flag was last written before a barrier already passed)
    const bool finite = bad == 0;
    if (chunk == 0 && t == 0 && skipped) *skipped = finite ? 0 : 1;
    if (finite) {
#pragma unroll
      for (int q = 0; q < kSets; ++q) {
        float th[8], out[8];
        decode_raw8(raw[q], th);
#pragma unroll
        for (int e = 0; e < 8; ++e) out[e] = th[e] - acc[q][e];
        store8(theta, base + 2048u * q + 8u * t, P, out);
      }
    }
#pragma unroll
    for (int q = 0; q < kSets; ++q) raw[q] = next[q];
  }
}

// Rademacher update for N <= 16 probes. Persistent workgroups of 512
// threads (two per CU) walk tiles of 8192 parameters (64 Philox blocks),
// tile blockIdx.x + i * gridDim.x. theta moves in coalesced 16-byte pieces
// with non-temporal loads and stores: lane t owns the 8-parameter chunks t
// and t + 512 of a tile, so every wave instruction covers 1 KiB of
// consecutive memory (lanes owning 32 consecutive parameters instead measured
// 40-80% slower for this read-modify-write).
//
// The sign work is done in a transposed role: lane t = 2 wg + g transposes
// word-group wg (sign word w = wg & 3 of block wg >> 2, 32 parameters) for
// probe group g (probes 8g .. 8g+7). The 8 lanes of a block each compute two
// of its 16 Philox blocks and swap words through LDS; three delta-swap stages
// transpose the 8x8 bit blocks of the 8 probe words in all four bytes at once
// (afterwards byte k of word r holds the 8 signs of parameter 8k + r), and the
// result goes back to the lane's LDS row. After a barrier each chunk owner
// reads the two rows of its word-group (one per probe group) and takes byte k
// of word i as the table index of its parameter i.
//
// The signed-sum tables of probes 0-7 (T0) and 8-15 (T1) are built once per
// workgroup and replicated 32 times: entry e is 256 bytes, [32 copies of
// T0[e]][32 copies of T1[e]], copy (lane & 31) in bank (lane & 31), so the
// lookups of 32 lanes never meet in a bank, and one v_perm builds a lookup
// address (the entry in byte 1, the lane's copy in byte 0). The sums, and the
// order in which they are formed, are those of the general kernel above.
constexpr int kR16Threads = 512;
constexpr int kR16Tile = kR16Threads * 16;  // parameters per tile
constexpr int kR16Copies = 32;
constexpr int kR16Row = 8;                  // LDS row: the 8 words of one (word-group, probe group)
constexpr int kR16PerCu = 2;                // resident workgroups per CU (LDS: 80 KiB each)

// Three delta swaps: transposes the 8x8 bit block in each byte lane of the 8
// words s[0..7] (row r = word r, column c = bit c of the byte).
__device__ __forceinline__ void transpose8_words(uint32_t s[8]) {
#pragma unroll
  for (int d = 1; d < 8; d <<= 1) {
    // columns c with bit d clear (m) of row r + d <-> columns c + d of row r
    const uint32_t m = d == 1 ? 0x55555555u : d == 2 ? 0x33333333u : 0x0F0F0F0Fu;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if (r & d) continue;
      const uint32_t a = s[r], b = s[r + d];
      s[r + d] = ((a >> d) & m) | (b & ~m);
      s[r] = ((b << d) & (m << d)) | (a & ~(m << d));
    }
  }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Orders this wave's LDS accesses: the writes and reads before it complete
// (lgkmcnt(0)) before any after it issue. Lanes of one wave exchange data
// through LDS this way without a workgroup barrier; the empty asm statements
// keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void wave_lds_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // vmcnt, expcnt at their maxima; lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  asm volatile("" ::: "memory");
}

template <typename T, bool kBits>
__global__ __launch_bounds__(kR16Threads) void update_rad16_kernel(
    T* __restrict__ theta, uint64_t P, Key key, float eps, float lr, int N, uint32_t i0,
    const float* __restrict__ Lp, const float* __restrict__ Lm, int32_t* __restrict__ skipped,
    int lm_stride, const uint32_t* __restrict__ bits) {
  // tables (64 KiB) first, so that a lookup address fits a 16-bit LDS offset;
  // then the rows (16 KiB), which also hold the coefficients and the 4-probe
  // partial sums while the tables are built
  __shared__ __align__(16) uint32_t lds[256 * 2 * kR16Copies + kR16Threads * kR16Row];
  float* tab = (float*)lds;
  uint32_t* rows = lds + 256 * 2 * kR16Copies;
  float* coef = (float*)rows;             // [16]
  float* half_table = (float*)rows + 32;  // [2][32]
  int* bad = (int*)rows + 96;
  const int t = threadIdx.x;
  constexpr int kVec = 8 * (int)sizeof(T) / 16;  // 16-byte vectors per chunk
  const bool two = N > 8;

  // wave 0: coefficients (lanes 0-15) and the 4-probe partial sums of both
  // probe groups; then every thread builds one table entry's 32 copies
  if (__builtin_amdgcn_readfirstlane(t >> 6) == 0) {
    float c = 0.f;
    int nonfinite = 0;
    if (t < N && t < kUpdGroup) {
      const float lp = Lp[t], lm = Lm[t * lm_stride];
      c = update_coeff(lr, N, lp, lm, eps);
      nonfinite = !(isfinite(lp) && isfinite(lm));
    }
    if (t < kUpdGroup) coef[t] = c;
    const int any = __builtin_amdgcn_readfirstlane(__any(nonfinite) ? 1 : 0);
    if (t == 0) *bad = any;
    wave_lds_sync();
    const int gg = t >> 5, h = (t >> 4) & 1, m = t & 15;
    float v = 0.f;
#pragma unroll
    for (int bb = 0; bb < 4; ++bb) {
      const float cb = coef[8 * gg + 4 * h + bb];
      v += ((m >> bb) & 1) ? cb : -cb;
    }
    half_table[32 * gg + 16 * h + m] = v;
  }
  lds_barrier();
  {
    // entry e of group gt: the sums of the low and the high nibble, added
    // (with at most 8 probes both halves of an entry hold T0)
    const int e = t & 255, gt = t >> 8, gs = two ? gt : 0;
    const float v = half_table[32 * gs + (e & 15)] + half_table[32 * gs + 16 + (e >> 4)];
    float4* dst = (float4*)&tab[e * 2 * kR16Copies + gt * kR16Copies];
#pragma unroll
    for (int c = 0; c < kR16Copies / 4; ++c) dst[c] = float4{v, v, v, v};
  }
  const bool finite = *bad == 0;
  if (blockIdx.x == 0 && t == 0 && skipped) *skipped = finite ? 0 : 1;
  lds_barrier();  // the rows are free again
  if (!finite) return;  // the same in every lane

  const int b = t >> 3, w = (t >> 1) & 3, g = t & 1;  // transposer role
  const bool transposer = g == 0 || two;
  const uint32_t k = (uint32_t)(t & 3);               // owner role: byte k of each word
  const uint32_t sel = 0x0C0C0000u | ((4u + k) << 8);  // byte 0 of the base, byte k of the word
  const uint32_t base0 = (uint32_t)(t & 31) * 4u, base1 = 128u + base0;
  const uint64_t ntiles = (P + kR16Tile - 1) / kR16Tile;
  for (uint64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const uint64_t tile0 = tile * kR16Tile;
    // chunk q of this lane holds parameters tile0 + 8 (t + 512 q) .. + 7
    u32x4 raw[2][kVec];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const uint64_t j = tile0 + 8u * (uint64_t)(t + kR16Threads * q);
      if (j + 8 <= P) {
#pragma unroll
        for (int v = 0; v < kVec; ++v)
          raw[q][v] = __builtin_nontemporal_load((const u32x4*)(theta + j) + v);
      } else {
        T x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = j + e < P ? theta[j + e] : (T)0;
        __builtin_memcpy(raw[q], x, sizeof(x));
      }
    }
    if (transposer) {
      const uint64_t blk = tile0 / 128 + (uint64_t)b;
      Words x[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const int p = 8 * g + 2 * w + m;  // zeros past N: their coefficients are 0
        if (p < N) x[m] = kBits ? cached_block(bits, P, p, blk) : stream_block(key, blk, i0 + (uint32_t)p, kTagRademacher);
        else x[m] = Words{{0u, 0u, 0u, 0u}};
      }
      // word v of these two probes goes to the row of lane (b, v, g), at 2 w
#pragma unroll
      for (int v = 0; v < 4; ++v)
        *(uint2*)&rows[(8 * b + 2 * v + g) * kR16Row + 2 * w] = uint2{x[0].w[v], x[1].w[v]};
    }
    wave_lds_sync();  // the 8 lanes of a block are in one wave
    if (transposer) {
      uint32_t s[8];
      const uint4 lo = *(const uint4*)&rows[t * kR16Row], hi = *(const uint4*)&rows[t * kR16Row + 4];
      s[0] = lo.x; s[1] = lo.y; s[2] = lo.z; s[3] = lo.w;
      s[4] = hi.x; s[5] = hi.y; s[6] = hi.z; s[7] = hi.w;
      transpose8_words(s);  // the row is this lane's own from here on
      *(uint4*)&rows[t * kR16Row] = uint4{s[0], s[1], s[2], s[3]};
      *(uint4*)&rows[t * kR16Row + 4] = uint4{s[4], s[5], s[6], s[7]};
    }
    lds_barrier();
    // owner role: parameter i of chunk q is parameter 8k + i of word-group wg
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int wg = (t + kR16Threads * q) >> 2;
      const uint4 a0 = *(const uint4*)&rows[(2 * wg) * kR16Row];
      const uint4 a1 = *(const uint4*)&rows[(2 * wg) * kR16Row + 4];
      const uint32_t sa[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
      float acc[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        acc[i] = *(const float*)((const char*)tab + __builtin_amdgcn_perm(sa[i], base0, sel));
      if (two) {
        const uint4 b0 = *(const uint4*)&rows[(2 * wg + 1) * kR16Row];
        const uint4 b1 = *(const uint4*)&rows[(2 * wg + 1) * kR16Row + 4];
        const uint32_t sb[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
#pragma unroll
        for (int i = 0; i < 8; ++i)
          acc[i] += *(const float*)((const char*)tab + __builtin_amdgcn_perm(sb[i], base1, sel));
      }
      const uint64_t j = tile0 + 8u * (uint64_t)(t + kR16Threads * q);
      u32x4 out[kVec];
      if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          out[0][e] = pack_bf16x2_rne(bf16_to_f32((uint16_t)raw[q][0][e]) - acc[2 * e],
                                      bf16_to_f32((uint16_t)(raw[q][0][e] >> 16)) - acc[2 * e + 1]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          out[e >> 2][e & 3] = __float_as_uint(__uint_as_float(raw[q][e >> 2][e & 3]) - acc[e]);
      }
      if (j + 8 <= P) {
#pragma unroll
        for (int v = 0; v < kVec; ++v) __builtin_nontemporal_store(out[v], (u32x4*)(theta + j) + v);
      } else {
        T x[8];
        __builtin_memcpy(x, out, sizeof(x));
        for (int e = 0; e < 8; ++e)
          if (j + e < P) theta[j + e] = x[e];
      }
    }
    lds_barrier();  // every owner has read the rows before the next tile writes them
  }
}

// Normal-probe update: each thread owns one Philox block (4 parameters) and
// regenerates its 4 values of every probe in ascending order.
template <typename T>
__global__ __launch_bounds__(256) void update_gaussian_kernel(T* theta, uint64_t P, Key key,
                                                              float eps, float lr, int N,
                                                              uint32_t i0, const float* Lp,
                                                              const float* Lm, int32_t* skipped,
                                                              int lm_stride) {
  __shared__ float coef[256];
  __shared__ int flag;
  const bool ok = losses_finite(Lp, Lm, N, lm_stride, &flag);
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
    if (n0 + t < N) coef[t] = update_coeff(lr, N, Lp[n0 + t], Lm[(n0 + t) * lm_stride], eps);
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

template <typename T>
struct TypeTag {
  using type = T;
};

// The sign-probe cache: probe n's Philox blocks (tag 0), 4 words each,
// unshuffled, at n * bit_words(P) + 4 blk. One thread per block and probe.
__global__ __launch_bounds__(256) void bits_fill_kernel(uint32_t* bits, uint64_t P, Key key, uint32_t i0, int N) {
  const uint64_t nblk = (P + 127) / 128;
  for (int n = blockIdx.y; n < N; n += gridDim.y)
    for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nblk; b += (uint64_t)gridDim.x * blockDim.x) {
      const Words x = stream_block(key, b, i0 + (uint32_t)n, kTagRademacher);
      *(uint4*)(bits + (uint64_t)n * bit_words(P) + 4 * b) =
          uint4{sign_word_unshuffle(x.w[0]), sign_word_unshuffle(x.w[1]), sign_word_unshuffle(x.w[2]),
                sign_word_unshuffle(x.w[3])};
    }
}

}  // namespace

hipError_t launch_bits_fill(uint32_t* bits, uint64_t P, uint64_t seed, uint32_t i0, int32_t N, hipStream_t s) {
  const uint64_t nblk = (P + 127) / 128;
  uint64_t gx = (nblk + 255) / 256;
  if (gx > 8192) gx = 8192;
  const unsigned gy = (unsigned)(N < 65535 ? N : 65535);
  ProfScope ps(kKProbeCache, s);
  bits_fill_kernel<<<dim3((unsigned)gx, gy), dim3(256), 0, s>>>(bits, P, make_key(seed), i0, N);
  return hipGetLastError();
}

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
                         int32_t* skipped, hipStream_t s, int lm_stride, const uint32_t* bits) {
  const Key key = make_key(seed);
  ProfScope ps(kKUpdate, s);
  if (kind == ZO_RADEMACHER && N <= kUpdGroup) {
    // persistent workgroups, kR16PerCu per CU, never more than there are tiles
    const uint64_t tiles = (P + kR16Tile - 1) / kR16Tile;
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    const uint64_t slots = (uint64_t)(cus > 0 ? cus : 1) * kR16PerCu;
    const unsigned grid = (unsigned)(tiles < slots ? tiles : slots);
    auto go = [&](auto t_tag, auto b_tag) {
      using T = typename decltype(t_tag)::type;
      constexpr bool kB = decltype(b_tag)::value;
      update_rad16_kernel<T, kB><<<dim3(grid), dim3(kR16Threads), 0, s>>>((T*)theta, P, key, eps, lr, N, i0, Lp,
                                                                        Lm, skipped, lm_stride, bits);
    };
    using std::integral_constant;
    if (wdtype == ZO_WBF16)
      bits ? go(TypeTag<uint16_t>{}, integral_constant<bool, true>{})
           : go(TypeTag<uint16_t>{}, integral_constant<bool, false>{});
    else
      bits ? go(TypeTag<float>{}, integral_constant<bool, true>{})
           : go(TypeTag<float>{}, integral_constant<bool, false>{});
  } else if (kind == ZO_RADEMACHER) {
    // persistent workgroups: as many as fit on the device at once, each
    // walking chunks of kUpdChunk parameters
    const uint64_t nchunks = (P + kUpdChunk - 1) / kUpdChunk;
    int dev = 0, cus = 0, per_cu = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = wdtype == ZO_WBF16
              ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, update_rademacher_kernel<uint16_t, false>, 256, 0)
              : hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, update_rademacher_kernel<float, false>, 256, 0);
    if (e != hipSuccess) return e;
    const uint64_t slots = (uint64_t)(cus > 0 ? cus : 1) * (uint64_t)(per_cu > 0 ? per_cu : 1);
    const unsigned grid = (unsigned)(nchunks < slots ? nchunks : slots);
    auto go = [&](auto t_tag, auto b_tag) {
      using T = typename decltype(t_tag)::type;
      constexpr bool kB = decltype(b_tag)::value;
      update_rademacher_kernel<T, kB><<<dim3(grid), dim3(256), 0, s>>>((T*)theta, P, key, eps, lr, N, i0, Lp, Lm,
                                                                     skipped, nchunks, lm_stride, bits);
    };
    using std::integral_constant;
    if (wdtype == ZO_WBF16)
      bits ? go(TypeTag<uint16_t>{}, integral_constant<bool, true>{})
           : go(TypeTag<uint16_t>{}, integral_constant<bool, false>{});
    else
      bits ? go(TypeTag<float>{}, integral_constant<bool, true>{})
           : go(TypeTag<float>{}, integral_constant<bool, false>{});
  } else {
    const uint64_t grid = ((P + 3) / 4 + 255) / 256;
    if (wdtype == ZO_WBF16)
      update_gaussian_kernel<uint16_t><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (uint16_t*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped, lm_stride);
    else
      update_gaussian_kernel<float><<<dim3((unsigned)grid), dim3(256), 0, s>>>(
          (float*)theta, P, key, eps, lr, N, i0, Lp, Lm, skipped, lm_stride);
  }
  return hipGetLastError();
}

}  // namespace zo
