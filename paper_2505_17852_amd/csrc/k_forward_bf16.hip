// bf16 kernels of the batched perturbed forward (bf16 weights, bf16 MFMA
// operands, fp32 accumulation and fp32 cell state).
//
// A bf16 weight cannot carry a perturbation of eps = 1e-3 (its spacing near
// |w| = 1/64 is 6e-5, and a rounded w + eps z would lose several percent of
// eps z). So every product keeps the two terms apart, as two MFMA streams
// that share the activation fragment:
//     accW = A . W        (bf16 x bf16, fp32 accumulate)
//     accZ = A . z        (z = +-1 exactly, or the bf16 of a normal value)
//     a    = accW + s eps accZ   (fp32, in the epilogue)
// so the probe term is formed at fp32 precision relative to itself.
//
// Tiles: a workgroup computes 256 rows x 128 columns with K tiles of 64;
// 4 waves each own 64 rows x 128 columns as 2 x 4 tiles of
// v_mfma_f32_32x32x16_bf16 for each of the two streams (256 accumulator
// registers). Lane l feeds row/column l % 32 and k block l / 32 of each
// 32x32x16 step. LDS (dynamic, 72 KiB) holds the A tile [256][72], the weight
// tile [128][72] and the probe tile [128][72] (bf16, rows padded to 144 B so
// that 16 lanes' 128-bit reads hit distinct banks). The next K tile's global
// loads and probe generation are issued before the current tile's MFMAs.
#include <hip/hip_runtime.h>

#include "zo_kernels.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int TM = 256;  // rows per workgroup
constexpr int TN = 128;  // columns per workgroup
constexpr int TK = 64;   // K per tile
constexpr int LDB = TK + 8;  // LDS row stride in bf16 elements (144 B)
constexpr size_t kSmemBytes = (size_t)(TM + 2 * TN) * LDB * 2;

static_assert(2 * kRowGranuleBF16 % TM == 0, "a probe's rows must be a whole number of row tiles");
static_assert(TN == kVocabTile, "head vocabulary tile");

__device__ __forceinline__ bf8 as_bf8(u4 v) { return __builtin_bit_cast(bf8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)bf16_rne(lo) | ((uint32_t)bf16_rne(hi) << 16);
}

struct SegB {
  const uint16_t* A;  // row r of the tile at A + r * lda (bf16)
  int64_t lda;
  const uint16_t* W;  // weight row n at W + n * ldw (bf16, inside theta)
  int64_t ldw;
  uint64_t zoff;      // offset of W inside theta (probe coordinates)
  int K;
};

// accW / accZ: [2 row tiles][4 column tiles] of 32x32 fp32.
template <int kind, typename ColMap>
__device__ __forceinline__ void mainloop_bf16(f16v (&accW)[2][4], f16v (&accZ)[2][4], const SegB s0,
                                              const SegB s1, int nseg, ColMap colmap, Key key,
                                              uint32_t probe, uint16_t* sm) {
  uint16_t* sa = sm;
  uint16_t* sw = sm + TM * LDB;
  uint16_t* sz = sw + TN * LDB;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  // loader roles: A chunk idx = t + 256 q (q < 8): row idx >> 3, 8 bf16 at 8 (idx & 7);
  // weight / probe row rho = t >> 1, 32 consecutive k at 32 (t & 1)
  const int rho = t >> 1, half = t & 1;
  int wn;
  const bool wok = colmap(rho, wn);
  const int ntiles = s0.K / TK + (nseg > 1 ? s1.K / TK : 0);

  u4 ra[8], rw[4], rz[4];
  Words zcache{{0u, 0u, 0u, 0u}};
  int seg = 0, k0 = 0;

  auto fetch = [&]() {
    const SegB sg = seg == 0 ? s0 : s1;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = t + 256 * q;
      ra[q] = *(const u4*)(sg.A + (int64_t)(idx >> 3) * sg.lda + k0 + 8 * (idx & 7));
    }
    const uint16_t* wp = sg.W + (int64_t)wn * sg.ldw + k0 + 32 * half;
#pragma unroll
    for (int q = 0; q < 4; ++q) rw[q] = wok ? *(const u4*)(wp + 8 * q) : u4{0u, 0u, 0u, 0u};
    const uint64_t j0 = sg.zoff + (uint64_t)wn * (uint64_t)sg.ldw + (uint64_t)k0 + 32 * half;
    if constexpr (kind == ZO_RADEMACHER) {
      uint32_t word;
      const bool aligned = (sg.zoff % 128u) == 0 && (sg.ldw % 128) == 0;
      if (aligned) {
        if ((k0 & 127) == 0) zcache = stream_block(key, j0 >> 7, probe, kTagRademacher);
        const int q = (int)((j0 >> 5) & 3u);
        word = q == 0 ? zcache.w[0] : q == 1 ? zcache.w[1] : q == 2 ? zcache.w[2] : zcache.w[3];
      } else {
        word = rademacher_word(key, probe, j0 >> 5);
      }
      // bit 1 -> +1 (0x3F80), bit 0 -> -1 (0xBF80)
      const uint32_t nb = ~word;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        u4 v;
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const int e = 8 * q + 2 * d;
          v[d] = 0x3F803F80u | (((nb >> e) & 1u) << 15) | (((nb >> (e + 1)) & 1u) << 31);
        }
        rz[q] = v;
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float za[4], zb[4];
        gauss_block(key, probe, (j0 >> 2) + 2 * q, za);
        gauss_block(key, probe, (j0 >> 2) + 2 * q + 1, zb);
        rz[q] = u4{pack_bf16x2(za[0], za[1]), pack_bf16x2(za[2], za[3]), pack_bf16x2(zb[0], zb[1]),
                   pack_bf16x2(zb[2], zb[3])};
      }
    }
    if (!wok) {
#pragma unroll
      for (int q = 0; q < 4; ++q) rz[q] = u4{0u, 0u, 0u, 0u};
    }
    k0 += TK;
    if (k0 == sg.K) {
      k0 = 0;
      ++seg;
    }
  };

  fetch();
  for (int it = 0; it < ntiles; ++it) {
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int idx = t + 256 * q;
      *(u4*)(sa + (idx >> 3) * LDB + 8 * (idx & 7)) = ra[q];
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *(u4*)(sw + rho * LDB + 32 * half + 8 * q) = rw[q];
      *(u4*)(sz + rho * LDB + 32 * half + 8 * q) = rz[q];
    }
    __syncthreads();
    if (it + 1 < ntiles) fetch();

#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      const int kk = 16 * s + 8 * lg;
      bf8 a[2], w[4], z[4];
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        a[mt] = as_bf8(*(const u4*)(sa + (64 * wave + 32 * mt + lr) * LDB + kk));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        w[q] = as_bf8(*(const u4*)(sw + (32 * q + lr) * LDB + kk));
        z[q] = as_bf8(*(const u4*)(sz + (32 * q + lr) * LDB + kk));
      }
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          accW[mt][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], w[q], accW[mt][q], 0, 0, 0);
          accZ[mt][q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mt], z[q], accZ[mt][q], 0, 0, 0);
        }
      }
    }
  }
}

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanh_(float x) { return 1.0f - 2.0f / (__expf(2.0f * x) + 1.0f); }

// Row (within the workgroup's 256) of accumulator element v of row tile mt
// for this lane: 32x32 MFMA output layout.
__device__ __forceinline__ int acc_row(int wave, int mt, int lg, int v) {
  return 64 * wave + 32 * mt + 8 * (v >> 2) + 4 * lg + (v & 3);
}

// ---------------------------------------------------------------------------
struct GateArgsB {
  const uint16_t* x;      // [M][El] bf16
  const uint16_t* hprev;  // [M][H]
  uint16_t* hout;         // [M][H]
  float* cst;             // [M][H] fp32
  const uint16_t* theta;
  uint64_t off_ih, off_hh, off_b;
  int El, H;
  const float* zb;  // [N][4H] eps z of the bias
  Key key;
  uint32_t i0;
  float eps;
  RowMap rm;
};

// Workgroup: 256 rows x 32 hidden units (the 4 gates' 32-column blocks).
template <int kind>
__global__ __launch_bounds__(256) void gate_bf16_kernel(GateArgsB g) {
  extern __shared__ __align__(16) uint16_t smem[];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int u0 = blockIdx.x * 32;
  const int64_t m0 = (int64_t)blockIdx.y * TM;
  const int pair = (int)(m0 / g.rm.pair_rows);
  const int H = g.H;
  auto colmap = [&](int rho, int& n) {
    n = (rho >> 5) * H + u0 + (rho & 31);
    return true;
  };
  f16v accW[2][4], accZ[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      accW[mt][q] = f16v{};
      accZ[mt][q] = f16v{};
    }
  const SegB s0{g.x + m0 * g.El, g.El, g.theta + g.off_ih, g.El, g.off_ih, g.El};
  const SegB s1{g.hprev + m0 * H, H, g.theta + g.off_hh, H, g.off_hh, H};
  mainloop_bf16<kind>(accW, accZ, s0, s1, 2, colmap, g.key, g.i0 + (uint32_t)pair, smem);

  const int u = u0 + lr;
  float bb[4], zz[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bb[q] = bf16_to_f32(g.theta[g.off_b + (uint64_t)(q * H + u)]);
    zz[q] = g.zb[(int64_t)pair * 4 * H + q * H + u];
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t r = m0 + acc_row(wave, mt, lg, v);
      const bool neg = (r - (int64_t)pair * g.rm.pair_rows) >= g.rm.Bp;
      const float se = neg ? -g.eps : g.eps;
      float pre[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        pre[q] = accW[mt][q][v] + se * accZ[mt][q][v] + (neg ? bb[q] - zz[q] : bb[q] + zz[q]);
      const float ig = sigm(pre[0]), fg = sigm(pre[1]), gg = tanh_(pre[2]), og = sigm(pre[3]);
      const int64_t o = r * H + u;
      const float c = fg * g.cst[o] + ig * gg;
      g.cst[o] = c;
      g.hout[o] = bf16_rne(og * tanh_(c));
    }
  }
}

// ---------------------------------------------------------------------------
struct HeadArgsB {
  const uint16_t* h;  // [rows][H] bf16
  const uint16_t* theta;
  uint64_t off_w, off_b;
  int H, V;
  const float* zbo;  // [N][V]
  Key key;
  uint32_t i0;
  float eps;
  RowMap rm;
  int64_t M, rows;
  const int32_t* tokens;
  int C, t0, B;
  float* pmax;
  float* psum;
  float* ptgt;
};

template <int kind>
__global__ __launch_bounds__(256) void head_bf16_kernel(HeadArgsB g) {
  extern __shared__ __align__(16) uint16_t smem[];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int vt = blockIdx.x;
  const int v0 = vt * TN;
  const int64_t rr0 = (int64_t)blockIdx.y * TM;
  const int tt = (int)(rr0 / g.M);
  const int64_t r0 = rr0 - (int64_t)tt * g.M;
  const int pair = (int)(r0 / g.rm.pair_rows);
  const int V = g.V;
  auto colmap = [&](int rho, int& n) {
    n = v0 + rho;
    const bool ok = n < V;
    if (!ok) n = 0;
    return ok;
  };
  f16v accW[2][4], accZ[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      accW[mt][q] = f16v{};
      accZ[mt][q] = f16v{};
    }
  const SegB s0{g.h + rr0 * g.H, g.H, g.theta + g.off_w, g.H, g.off_w, g.H};
  mainloop_bf16<kind>(accW, accZ, s0, s0, 1, colmap, g.key, g.i0 + (uint32_t)pair, smem);

  int col[4];
  bool cok[4];
  float bb[4], zz[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    col[q] = v0 + 32 * q + lr;
    cok[q] = col[q] < V;
    bb[q] = cok[q] ? bf16_to_f32(g.theta[g.off_b + (uint64_t)col[q]]) : 0.f;
    zz[q] = cok[q] ? g.zbo[(int64_t)pair * V + col[q]] : 0.f;
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int lrow = acc_row(wave, mt, lg, v);
      const int64_t r = r0 + lrow;
      const int loc = (int)(r - (int64_t)pair * g.rm.pair_rows);
      const bool neg = loc >= g.rm.Bp;
      const int b = neg ? loc - g.rm.Bp : loc;
      const float se = neg ? -g.eps : g.eps;
      float y[4];
      float mx = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        y[q] = cok[q] ? accW[mt][q][v] + se * accZ[mt][q][v] + (neg ? bb[q] - zz[q] : bb[q] + zz[q])
                      : -INFINITY;
        mx = fmaxf(mx, y[q]);
      }
      if (b < g.B) {
        const int tgt = g.tokens[(int64_t)b * (g.C + 1) + g.t0 + tt + 1];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (col[q] == tgt) g.ptgt[rr0 + lrow] = y[q];
      }
      // the row's 128 columns sit in the 32 lanes of this lane half
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      float se2 = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) se2 += cok[q] ? __expf(y[q] - mx) : 0.f;
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) se2 += __shfl_xor(se2, off, 64);
      if (lr == 0) {
        g.pmax[(int64_t)vt * g.rows + rr0 + lrow] = mx;
        g.psum[(int64_t)vt * g.rows + rr0 + lrow] = se2;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// x0[r][e] = bf16(EMB[tok][e] + s eps z_n[emb + tok E + e]); zeros for padding rows.
template <int kind>
__global__ __launch_bounds__(256) void embed_bf16_kernel(const uint16_t* theta, uint64_t emb_off, int E,
                                                         const int32_t* tokens, int C, int t, int B,
                                                         RowMap rm, int64_t M, Key key, uint32_t i0,
                                                         float eps, uint16_t* x0) {
  const int E4 = E >> 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= M * E4) return;
  const int64_t r = idx / E4;
  const int e = (int)(idx - r * E4) * 4;
  const int pair = (int)(r / rm.pair_rows);
  const int loc = (int)(r - pair * rm.pair_rows);
  const int sidx = loc >= rm.Bp;
  const int b = loc - sidx * rm.Bp;
  uint32_t lo = 0u, hi = 0u;
  if (b < B) {
    const int tok = tokens[(int64_t)b * (C + 1) + t];
    const uint64_t j = emb_off + (uint64_t)tok * E + e;
    const uint2 wv = *(const uint2*)(theta + j);
    float w[4] = {bf16_to_f32((uint16_t)wv.x), bf16_to_f32((uint16_t)(wv.x >> 16)),
                  bf16_to_f32((uint16_t)wv.y), bf16_to_f32((uint16_t)(wv.y >> 16))};
    float z[4];
    if constexpr (kind == ZO_RADEMACHER) {
      const uint32_t word = rademacher_word(key, i0 + pair, j >> 5) >> (uint32_t)(j & 31u);
#pragma unroll
      for (int q = 0; q < 4; ++q) z[q] = ((word >> q) & 1u) ? 1.0f : -1.0f;
    } else {
      gauss_block(key, i0 + pair, j >> 2, z);
    }
    const float se = sidx ? -eps : eps;
    lo = pack_bf16x2(w[0] + se * z[0], w[1] + se * z[1]);
    hi = pack_bf16x2(w[2] + se * z[2], w[3] + se * z[3]);
  }
  *(uint2*)(x0 + r * E + e) = uint2{lo, hi};
}

template <typename K>
hipError_t allow_smem(K kernel) {
  static bool done = false;  // set once per kernel instantiation (same value on every device)
  if (done) return hipSuccess;
  hipError_t e = hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)kSmemBytes);
  if (e == hipSuccess) done = true;
  return e;
}

}  // namespace

hipError_t launch_embed_bf16(const ForwardArgs& a, int t, void* x0, hipStream_t st) {
  const Rows& R = a.rows;
  const int E = a.cfg.embed;
  const RowMap rm{R.Bp, R.pair_rows};
  const int64_t n = R.M * (E / 4);
  const unsigned grid = (unsigned)((n + 255) / 256);
  const Key key = make_key(a.seed);
  ProfScope ps(kKEmbed, st);
  if (a.cfg.probe == ZO_RADEMACHER)
    embed_bf16_kernel<ZO_RADEMACHER><<<grid, 256, 0, st>>>((const uint16_t*)a.theta, a.lay.emb, E,
                                                           a.tokens, a.C, t, R.B, rm, R.M, key, a.i0,
                                                           a.eps, (uint16_t*)x0);
  else
    embed_bf16_kernel<ZO_GAUSSIAN><<<grid, 256, 0, st>>>((const uint16_t*)a.theta, a.lay.emb, E,
                                                         a.tokens, a.C, t, R.B, rm, R.M, key, a.i0,
                                                         a.eps, (uint16_t*)x0);
  return hipGetLastError();
}

hipError_t launch_gate_bf16(const ForwardArgs& a, int l, const void* x, const void* hprev, void* hout,
                            float* cst, const float* zb, hipStream_t st) {
  const Rows& R = a.rows;
  GateArgsB g;
  g.x = (const uint16_t*)x;
  g.hprev = (const uint16_t*)hprev;
  g.hout = (uint16_t*)hout;
  g.cst = cst;
  g.theta = (const uint16_t*)a.theta;
  g.off_ih = a.lay.w_ih[l];
  g.off_hh = a.lay.w_hh[l];
  g.off_b = a.lay.bias[l];
  g.El = l == 0 ? a.cfg.embed : a.cfg.hidden;
  g.H = a.cfg.hidden;
  g.zb = zb;
  g.key = make_key(a.seed);
  g.i0 = a.i0;
  g.eps = a.eps;
  g.rm = RowMap{R.Bp, R.pair_rows};
  const dim3 grid((unsigned)(g.H / 32), (unsigned)(R.M / TM));
  hipError_t e;
  if (a.cfg.probe == ZO_RADEMACHER) {
    if ((e = allow_smem(gate_bf16_kernel<ZO_RADEMACHER>)) != hipSuccess) return e;
    ProfScope ps(kKGate, st);
    gate_bf16_kernel<ZO_RADEMACHER><<<grid, 256, kSmemBytes, st>>>(g);
  } else {
    if ((e = allow_smem(gate_bf16_kernel<ZO_GAUSSIAN>)) != hipSuccess) return e;
    ProfScope ps(kKGate, st);
    gate_bf16_kernel<ZO_GAUSSIAN><<<grid, 256, kSmemBytes, st>>>(g);
  }
  return hipGetLastError();
}

hipError_t launch_head_bf16(const ForwardArgs& a, const void* hist, int t0, int Tc, const float* zbo,
                            float* pmax, float* psum, float* ptgt, hipStream_t st) {
  const Rows& R = a.rows;
  HeadArgsB h;
  h.h = (const uint16_t*)hist;
  h.theta = (const uint16_t*)a.theta;
  h.off_w = a.lay.w_out;
  h.off_b = a.lay.b_out;
  h.H = a.cfg.hidden;
  h.V = a.cfg.vocab;
  h.zbo = zbo;
  h.key = make_key(a.seed);
  h.i0 = a.i0;
  h.eps = a.eps;
  h.rm = RowMap{R.Bp, R.pair_rows};
  h.M = R.M;
  h.rows = (int64_t)Tc * R.M;
  h.tokens = a.tokens;
  h.C = a.C;
  h.t0 = t0;
  h.B = R.B;
  h.pmax = pmax;
  h.psum = psum;
  h.ptgt = ptgt;
  const dim3 grid((unsigned)a.ws.nvt, (unsigned)(h.rows / TM));
  hipError_t e;
  if (a.cfg.probe == ZO_RADEMACHER) {
    if ((e = allow_smem(head_bf16_kernel<ZO_RADEMACHER>)) != hipSuccess) return e;
    ProfScope ps(kKHead, st);
    head_bf16_kernel<ZO_RADEMACHER><<<grid, 256, kSmemBytes, st>>>(h);
  } else {
    if ((e = allow_smem(head_bf16_kernel<ZO_GAUSSIAN>)) != hipSuccess) return e;
    ProfScope ps(kKHead, st);
    head_bf16_kernel<ZO_GAUSSIAN><<<grid, 256, kSmemBytes, st>>>(h);
  }
  return hipGetLastError();
}

}  // namespace zo
