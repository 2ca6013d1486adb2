// Device-side random stream of the CD-RGE step: Philox4x32-10 and the
// transforms from its 32-bit words to probe values and initial weights.
//
// The paper draws one seeded probe per perturbation and regenerates it every
// time it is applied (Algorithm 2, reconstructed several times per step,
// Section 3.1), never holding a whole probe. A counter-based generator gives
// the same property with random access: any element z_i[j] is a pure
// function of (seed, i, j), so a tile of z can be produced wherever a kernel
// needs it.
//
// The fp32 operation sequences below (ln, sin/cos of a 24-bit angle, the
// Box-Muller pair and the initial-weight scaling) are a fixed contract: every
// operation is a single correctly rounded fp32 operation, so that every
// implementation of the contract yields the same bits. HIP compiles with
// floating-point contraction on by default; the helpers fmul/fadd/fdiv turn
// it off (a multiply followed by an add must not become one fma).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zo {

enum : uint32_t { kTagRademacher = 0u, kTagGaussian = 1u, kTagInit = 2u };

struct Key {
  uint32_t k0, k1;
};
__host__ __device__ inline Key make_key(uint64_t seed) {
  return Key{(uint32_t)seed, (uint32_t)(seed >> 32)};
}

struct Words {
  uint32_t w[4];
};

// a ^ b ^ k in one v_bitop3_b32 (truth table 0x96); the compiler would emit
// two v_xor_b32. k must be the same in every lane (a Philox round key: the
// seed is a launch argument), since it is read from a scalar register.
__device__ __forceinline__ uint32_t xor3_key(uint32_t a, uint32_t b, uint32_t k) {
  uint32_t d;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(d) : "v"(a), "v"(b), "s"(k));
  return d;
}

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror and Shaw, SC'11): each
// round multiplies counter words 0 and 2 by two fixed odd constants, swaps
// the halves of the 64-bit products across the lanes and mixes in the key;
// the key advances by the two Weyl constants after every round. The key must
// be wave-uniform (xor3_key).
__device__ __forceinline__ Words philox(uint32_t x0, uint32_t x1, uint32_t x2, uint32_t x3,
                                        Key key) {
  uint32_t k0 = key.k0, k1 = key.k1;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t pa = (uint64_t)0xD2511F53u * (uint64_t)x0;
    const uint64_t pb = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
    const uint32_t y0 = xor3_key((uint32_t)(pb >> 32), x1, k0);
    const uint32_t y1 = (uint32_t)pb;
    const uint32_t y2 = xor3_key((uint32_t)(pa >> 32), x3, k1);
    const uint32_t y3 = (uint32_t)pa;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return Words{{x0, x1, x2, x3}};
}

// Block `blk` of probe stream `i` under `tag`: counter (blk lo, blk hi, i, tag).
__device__ __forceinline__ Words stream_block(Key key, uint64_t blk, uint32_t i, uint32_t tag) {
  return philox((uint32_t)blk, (uint32_t)(blk >> 32), i, tag, key);
}

// 32 Rademacher signs z_i[32q .. 32q+31] (q = j >> 5) as one word; bit b set
// means z = +1 for element 32q + b.
__device__ __forceinline__ uint32_t rademacher_word(Key key, uint32_t i, uint64_t q) {
  const Words x = stream_block(key, q >> 2, i, kTagRademacher);
  const uint32_t s = (uint32_t)(q & 3u);
  return s == 0 ? x.w[0] : s == 1 ? x.w[1] : s == 2 ? x.w[2] : x.w[3];
}

// ---- fixed fp32 sequences ------------------------------------------------

// Single rounded operations. The contraction pragma sits inside each helper
// (an fma can only form when both the multiply and the add allow it), and
// sqrt / division use the compiler's correctly rounded expansions
// (__fsqrt_rn would map to the 1-ulp hardware square root).
__device__ __forceinline__ float fmul(float a, float b) {
#pragma clang fp contract(off)
  return a * b;
}
__device__ __forceinline__ float fadd(float a, float b) {
#pragma clang fp contract(off)
  return a + b;
}
__device__ __forceinline__ float fdiv(float a, float b) {
#pragma clang fp contract(off)
  return a / b;
}
__device__ __forceinline__ float fsqrt(float a) { return __builtin_sqrtf(a); }

// Natural log of a normal float u in (0, 1]. Write u = 2^e m with m folded
// into (sqrt(1/2), sqrt(2)]; then ln m = 2 atanh(s) with s = (m-1)/(m+1),
// summed as s * (2 + s^2 (2/3 + s^2 (2/5 + s^2 (2/7 + s^2 2/9)))), and
// ln u = e ln2_hi + (e ln2_lo + ln m) with ln 2 split into a 16-bit head and
// its remainder.
__device__ __forceinline__ float ln_u(float u) {
  const uint32_t bits = __float_as_uint(u);
  int e = (int)((bits >> 23) & 0xFFu) - 127;
  float m = __uint_as_float((bits & 0x007FFFFFu) | 0x3F800000u);
  if (m > __uint_as_float(0x3FB504F3u)) {  // largest float <= sqrt(2)
    m = fmul(m, 0.5f);
    e += 1;
  }
  const float s = fdiv(fadd(m, -1.0f), fadd(m, 1.0f));
  const float s2 = fmul(s, s);
  float p = (float)(2.0 / 9.0);
  p = fadd(fmul(p, s2), (float)(2.0 / 7.0));
  p = fadd(fmul(p, s2), (float)(2.0 / 5.0));
  p = fadd(fmul(p, s2), (float)(2.0 / 3.0));
  p = fadd(fmul(p, s2), 2.0f);
  const float lnm = fmul(s, p);
  const float ef = (float)e;
  const float ln2_head = __uint_as_float(0x3F317200u);  // 0.693145751953125
  const float ln2_tail = (float)(0.6931471805599453094 - 0.693145751953125);
  const float lo = fadd(fmul(ef, ln2_tail), lnm);
  return fadd(fmul(ef, ln2_head), lo);
}

// sin and cos of 2 pi k / 2^24 for a 24-bit integer k. Exact integer split
// into the nearest quarter turn q and a remainder d in [-1/2, 1/2) quarter
// turns; phi = d pi/2 in [-pi/4, pi/4); odd Taylor series of sin through
// phi^9 and even series of cos through phi^10, then rotation by q.
__device__ __forceinline__ void sincos_turn24(uint32_t k24, float& s_out, float& c_out) {
  const int32_t k = (int32_t)(k24 & 0xFFFFFFu);
  const int32_t qn = (k + (1 << 21)) >> 22;
  const int32_t dk = k - (qn << 22);
  const int q = qn & 3;
  const float d = fmul((float)dk, __uint_as_float(0x34800000u));  // 2^-22, exact
  const float phi = fmul(d, (float)1.57079632679489661923);
  const float p2 = fmul(phi, phi);
  float sp = (float)(1.0 / 362880.0);
  sp = fadd(fmul(sp, p2), (float)(-1.0 / 5040.0));
  sp = fadd(fmul(sp, p2), (float)(1.0 / 120.0));
  sp = fadd(fmul(sp, p2), (float)(-1.0 / 6.0));
  sp = fmul(fmul(sp, p2), phi);
  const float sn = fadd(phi, sp);
  float cp = (float)(-1.0 / 3628800.0);
  cp = fadd(fmul(cp, p2), (float)(1.0 / 40320.0));
  cp = fadd(fmul(cp, p2), (float)(-1.0 / 720.0));
  cp = fadd(fmul(cp, p2), (float)(1.0 / 24.0));
  cp = fadd(fmul(cp, p2), -0.5f);
  cp = fmul(cp, p2);
  const float cs = fadd(1.0f, cp);
  switch (q) {
    case 0: s_out = sn;  c_out = cs;  break;
    case 1: s_out = cs;  c_out = -sn; break;
    case 2: s_out = -sn; c_out = -cs; break;
    default: s_out = -cs; c_out = sn; break;
  }
}

// Box-Muller (1958) on two words: u1 = (x0>>8 + 1) 2^-24 in (0, 1],
// angle x1>>8 of 2^24; returns (r cos, r sin) with r = sqrt(-2 ln u1).
__device__ __forceinline__ void gauss_pair(uint32_t x0, uint32_t x1, float& z0, float& z1) {
  const float u1 = fmul((float)((x0 >> 8) + 1u), __uint_as_float(0x33800000u));  // 2^-24
  const float r = fsqrt(fmul(-2.0f, ln_u(u1)));
  float s, c;
  sincos_turn24(x1 >> 8, s, c);
  z0 = fmul(r, c);
  z1 = fmul(r, s);
}

// The four normal probe values z_i[4b .. 4b+3] of block b.
__device__ __forceinline__ void gauss_block(Key key, uint32_t i, uint64_t b, float z[4]) {
  const Words x = stream_block(key, b, i, kTagGaussian);
  gauss_pair(x.w[0], x.w[1], z[0], z[1]);
  gauss_pair(x.w[2], x.w[3], z[2], z[3]);
}

// One probe element (slow path: a whole Philox block per element).
__device__ __forceinline__ float probe_value(int kind, Key key, uint32_t i, uint64_t j) {
  if (kind == 0) {
    const uint32_t w = rademacher_word(key, i, j >> 5);
    return ((w >> (uint32_t)(j & 31u)) & 1u) ? 1.0f : -1.0f;
  }
  float z[4];
  gauss_block(key, i, j >> 2, z);
  const uint32_t r = (uint32_t)(j & 3u);
  return r == 0 ? z[0] : r == 1 ? z[1] : r == 2 ? z[2] : z[3];
}

// Initial weight from one word: (2m + 1 - 2^24) 2^-24 with m = w >> 8, an
// exact odd multiple of 2^-24 in (-1, 1), times fp32(1/sqrt(H)).
__device__ __forceinline__ float init_value(uint32_t w, float scale) {
  const int32_t m = (int32_t)(w >> 8);
  const float v = fmul((float)(2 * m + 1 - (1 << 24)), __uint_as_float(0x33800000u));
  return fmul(v, scale);
}

// fp32 -> bf16, round to nearest even (NaN kept quiet).
__host__ __device__ inline uint16_t bf16_rne(float f) {
  uint32_t b;
  __builtin_memcpy(&b, &f, 4);
  if ((b & 0x7F800000u) == 0x7F800000u && (b & 0x007FFFFFu)) return (uint16_t)((b >> 16) | 0x40u);
  b += 0x7FFFu + ((b >> 16) & 1u);
  return (uint16_t)(b >> 16);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// fp32 -> fp16 bits, round to nearest even (subnormals kept, overflow to
// infinity, NaN kept quiet); the host's conversion of eps, bit-equal to the
// device's v_cvt_f16_f32 under its default rounding.
__host__ __device__ inline uint16_t f16_rne(float f) {
  uint32_t x;
  __builtin_memcpy(&x, &f, 4);
  const uint32_t sign = (x >> 16) & 0x8000u;
  x &= 0x7FFFFFFFu;
  if (x >= 0x7F800000u) return (uint16_t)(sign | (x > 0x7F800000u ? 0x7E00u : 0x7C00u));
  if (x >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u);  // >= 65520 rounds to infinity
  uint32_t h, rem, half;
  if (x >= 0x38800000u) {  // normal: rebias the exponent (127 -> 15), round off 13 bits
    const uint32_t r = x - 0x38000000u;
    h = r >> 13;
    rem = r & 0x1FFFu;
    half = 0x1000u;
  } else {  // subnormal or zero: round(|f| 2^24)
    const int shift = 126 - (int)(x >> 23);
    if (shift > 24) return (uint16_t)sign;
    const uint32_t m = (x & 0x007FFFFFu) | 0x00800000u;
    h = m >> shift;
    rem = m & ((1u << shift) - 1u);
    half = 1u << (shift - 1);
  }
  if (rem > half || (rem == half && (h & 1u))) ++h;
  return (uint16_t)(sign | h);
}

// Two fp32 values to packed fp16 (round to nearest even), low half first.
__device__ __forceinline__ uint32_t pack_f16x2(float lo, float hi) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  typedef float f2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f2){lo, hi}, h2));
}
__device__ __forceinline__ uint16_t f16_bits(float x) { return __builtin_bit_cast(uint16_t, (_Float16)x); }

}  // namespace zo
