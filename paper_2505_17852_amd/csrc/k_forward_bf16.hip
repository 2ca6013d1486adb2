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
// Tiles: a workgroup of 8 waves computes TM = 256 rows x 128 columns with K
// tiles of 64; wave (wm, wn) owns rows 64 wm .. +63 and columns 64 wn .. +63
// as 2 x 2 tiles of v_mfma_f32_32x32x16_bf16 per stream (128 accumulator
// registers, under 256 VGPRs), so two waves share each SIMD and one wave's
// LDS reads, probe expansion and address work run under the other's matrix
// instructions. (Measured alternative: 128-row workgroups, two per CU, are
// 9% slower at the 1.2B shape and 2.5x slower with normal probes.)
// Lane l feeds row/column l % 32 and k block l / 32 of each 32x32x16 step.
//
// LDS (dynamic, double-buffered, one barrier per K tile): the activation tile
// [TM][72] and the weight tile [128][72] (bf16, rows padded to 144 B so that
// 16 lanes' 128-bit reads hit distinct banks), and the probe tile: Rademacher
// sign bits [128][2] words, expanded to bf16 +-1 by each wave, or normal
// values in bf16 [128][72]. The next K tile's global loads and probe
// generation are issued before the current tile's MFMAs.
#include <hip/hip_runtime.h>

#include "zo_kernels.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

typedef __bf16 bf8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int TN = 128;      // columns per workgroup
constexpr int TK = 64;       // K per tile
constexpr int LDB = TK + 8;  // LDS row stride in bf16 elements (144 B)
constexpr int TM = 256;              // rows per workgroup
constexpr int WAVES_M = TM / 64;     // waves along the rows
constexpr int NWAVES = 2 * WAVES_M;  // x 2 along the columns
constexpr int NT = 64 * NWAVES;      // threads per workgroup
constexpr int WCHUNKS = TN * 8 / NT; // 16-byte weight chunks per thread and K tile
constexpr int ZROW_T = NT / TN;      // threads per probe-tile row (normal probes)
constexpr int ZVALS = TK / ZROW_T;   // probe values per thread and K tile (normal probes)
static_assert(NT >= 256 && TM * 8 / NT == 4, "loader layout");

static_assert(2 * kRowGranuleBF16 % TM == 0, "a probe's rows must be a whole number of row tiles");
static_assert(TN == kVocabTile, "head vocabulary tile");

__device__ __forceinline__ bf8 as_bf8(u4 v) { return __builtin_bit_cast(bf8, v); }

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return (uint32_t)bf16_rne(lo) | ((uint32_t)bf16_rne(hi) << 16);
}

// Probe sign bits in LDS are kept in "unshuffled" order: the word of 32
// consecutive k holds the negative-sign flags (1 = -1) of the even elements
// 0, 2, .., 30 in bits 0..15 and of the odd elements 1, 3, .., 31 in bits
// 16..31. The two elements of one packed bf16 pair then sit 16 bits apart,
// so one shift and one mask-or turn them into the pair (+-1, +-1): the flag
// of the even element lands on bit 15 and that of the odd one on bit 31 over
// the constant 0x3F803F80 (= +1, +1).
__device__ __forceinline__ uint32_t unshuffle_bits(uint32_t x) {
  uint32_t t;
  t = (x ^ (x >> 1)) & 0x22222222u;
  x = x ^ t ^ (t << 1);
  t = (x ^ (x >> 2)) & 0x0C0C0C0Cu;
  x = x ^ t ^ (t << 2);
  t = (x ^ (x >> 4)) & 0x00F000F0u;
  x = x ^ t ^ (t << 4);
  t = (x ^ (x >> 8)) & 0x0000FF00u;
  x = x ^ t ^ (t << 8);
  return x;
}

struct SegB {
  const uint16_t* A;  // first row of this workgroup's activation tile; row r at A + r * lda
  int64_t lda;
  const uint16_t* W;  // weight row n at W + n * ldw (bf16, inside theta)
  int64_t ldw;
  uint64_t zoff;      // offset of W inside theta (probe coordinates)
  int K;
};

// LDS stage layout (bf16 element offsets): A tile, weight tile, probe tile.
constexpr int kATile = TM * LDB;
constexpr int kWTile = TN * LDB;
constexpr int kZTileGauss = TN * LDB;
constexpr int kZTileBits = TN * 2 * 2;  // TN rows x 2 words, in bf16 units
template <int kind>
constexpr int stage_elems() {
  return kATile + kWTile + (kind == ZO_RADEMACHER ? kZTileBits : kZTileGauss);
}
template <int kind>
constexpr size_t smem_bytes() {
  return (size_t)2 * stage_elems<kind>() * 2;
}

// accW / accZ: [2 row tiles][2 column tiles] of 32x32 fp32 for this wave.
// colmap(rho, &n) -> true if LDS column rho (0..127) maps to a real weight row n.
template <int kind, typename ColMap>
__device__ __forceinline__ void mainloop_bf16(f16v (&accW)[2][2], f16v (&accZ)[2][2], const SegB s0,
                                              const SegB s1, int nseg, ColMap colmap, Key key,
                                              uint32_t probe, uint16_t* sm) {
  constexpr int kStage = stage_elems<kind>();
  // plain offsets from the shared-memory base keep every access a DS instruction
  auto sa = [&](int b) { return sm + b * kStage; };
  auto sw = [&](int b) { return sm + b * kStage + kATile; };
  auto sz = [&](int b) { return sm + b * kStage + kATile + kWTile; };
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  const int ntiles = s0.K / TK + (nseg > 1 ? s1.K / TK : 0);

  // loader roles
  //   A: chunks idx = t + NT q (q < 4): row idx >> 3, 8 bf16 at 8 (idx & 7)
  //   W: chunks idx = t + NT q (q < WCHUNKS): row idx >> 3, 8 bf16 at 8 (idx & 7)
  //   probe: Rademacher, threads t < 256: row t >> 1, one 32-k word at 32 (t & 1);
  //          normal, all threads: row t / ZROW_T, ZVALS k at ZVALS (t % ZROW_T)
  int wrow[WCHUNKS];
  bool wok[WCHUNKS];
#pragma unroll
  for (int q = 0; q < WCHUNKS; ++q) wok[q] = colmap((t + NT * q) >> 3, wrow[q]);
  const int zr = kind == ZO_RADEMACHER ? (t >> 1) & 127 : t / ZROW_T;
  const int zpart = kind == ZO_RADEMACHER ? (t & 1) : (t % ZROW_T);
  int zn;
  const bool zok = colmap(zr, zn);
  const bool zthread = kind != ZO_RADEMACHER || t < 256;

  u4 ra[4], rw[WCHUNKS], rz[ZVALS / 8];
  uint32_t rbits = 0u;
  Words zcache{{0u, 0u, 0u, 0u}};
  int seg = 0, k0 = 0;

  auto fetch = [&]() {
    const SegB sg = seg == 0 ? s0 : s1;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + NT * q;
      ra[q] = *(const u4*)(sg.A + (int64_t)(idx >> 3) * sg.lda + k0 + 8 * (idx & 7));
    }
#pragma unroll
    for (int q = 0; q < WCHUNKS; ++q) {
      const int idx = t + NT * q;
      rw[q] = wok[q] ? *(const u4*)(sg.W + (int64_t)wrow[q] * sg.ldw + k0 + 8 * (idx & 7))
                     : u4{0u, 0u, 0u, 0u};
    }
    if constexpr (kind == ZO_RADEMACHER) {
      if (zthread) {
        const uint64_t j0 = sg.zoff + (uint64_t)zn * (uint64_t)sg.ldw + (uint64_t)k0 + 32 * zpart;
        uint32_t word;
        const bool aligned = (sg.zoff % 128u) == 0 && (sg.ldw % 128) == 0;
        if (aligned) {
          if ((k0 & 127) == 0) zcache = stream_block(key, j0 >> 7, probe, kTagRademacher);
          const int q = (int)((j0 >> 5) & 3u);
          word = q == 0 ? zcache.w[0] : q == 1 ? zcache.w[1] : q == 2 ? zcache.w[2] : zcache.w[3];
        } else {
          word = rademacher_word(key, probe, j0 >> 5);
        }
        // negative-sign flags in unshuffled order; padding columns: all -1
        // against zero weights, never scored
        rbits = zok ? unshuffle_bits(~word) : 0xFFFFFFFFu;
      }
    } else {
      const uint64_t j0 = sg.zoff + (uint64_t)zn * (uint64_t)sg.ldw + (uint64_t)k0 + ZVALS * zpart;
#pragma unroll
      for (int q = 0; q < ZVALS / 8; ++q) {
        float za[4], zb[4];
        gauss_block(key, probe, (j0 >> 2) + 2 * q, za);
        gauss_block(key, probe, (j0 >> 2) + 2 * q + 1, zb);
        rz[q] = zok ? u4{pack_bf16x2(za[0], za[1]), pack_bf16x2(za[2], za[3]),
                         pack_bf16x2(zb[0], zb[1]), pack_bf16x2(zb[2], zb[3])}
                    : u4{0u, 0u, 0u, 0u};
      }
    }
    k0 += TK;
    if (k0 == sg.K) {
      k0 = 0;
      ++seg;
    }
  };

  auto store = [&](int b) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int idx = t + NT * q;
      *(u4*)(sa(b) + (idx >> 3) * LDB + 8 * (idx & 7)) = ra[q];
    }
#pragma unroll
    for (int q = 0; q < WCHUNKS; ++q) {
      const int idx = t + NT * q;
      *(u4*)(sw(b) + (idx >> 3) * LDB + 8 * (idx & 7)) = rw[q];
    }
    if constexpr (kind == ZO_RADEMACHER) {
      if (zthread) ((uint32_t*)sz(b))[zr * 2 + zpart] = rbits;
    } else {
#pragma unroll
      for (int q = 0; q < ZVALS / 8; ++q) *(u4*)(sz(b) + zr * LDB + ZVALS * zpart + 8 * q) = rz[q];
    }
  };

  // Fragments of one 16-k step: activations (2 row tiles), weights and probe
  // values (2 column tiles). The next step's LDS reads and sign expansion are
  // issued between the current step's MFMAs (software pipelining within the
  // K tile), so the matrix pipe is fed while the VALU and LDS work proceeds.
  struct Frag {
    bf8 a[2], w[2], z[2];
  };
  auto compute = [&](int b) {
    const uint16_t* pa = sa(b) + (64 * wm + lr) * LDB + 8 * lg;
    const uint16_t* pw = sw(b) + (64 * wn + lr) * LDB + 8 * lg;
    // per lane, the flags of its k block pre-shifted so that a constant shift
    // per (k step, pair) brings them to bits 15 / 31 (see unshuffle_bits)
    uint32_t bits[2][2];
    if constexpr (kind == ZO_RADEMACHER) {
      const uint32_t pre = 4u * (uint32_t)(1 - lg);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const uint2 v = *(const uint2*)((const uint32_t*)sz(b) + (64 * wn + 32 * nt + lr) * 2);
        bits[nt][0] = v.x << pre;
        bits[nt][1] = v.y << pre;
      }
    }
    auto load = [&](int s, Frag& f) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) f.a[mt] = as_bf8(*(const u4*)(pa + 32 * mt * LDB + 16 * s));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        f.w[nt] = as_bf8(*(const u4*)(pw + 32 * nt * LDB + 16 * s));
        if constexpr (kind == ZO_RADEMACHER) {
          const uint32_t x = bits[nt][s >> 1];
          u4 v;
#pragma unroll
          for (int d = 0; d < 4; ++d) v[d] = ((x << (11 - 8 * (s & 1) - d)) & 0x80008000u) | 0x3F803F80u;
          f.z[nt] = as_bf8(v);
        } else {
          f.z[nt] = as_bf8(*(const u4*)(sz(b) + (64 * wn + 32 * nt + lr) * LDB + 16 * s + 8 * lg));
        }
      }
    };
    Frag f[2];
    load(0, f[0]);
#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      const Frag& c = f[s & 1];
      if (s + 1 < TK / 16) load(s + 1, f[(s + 1) & 1]);
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          accW[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c.a[mt], c.w[nt], accW[mt][nt], 0, 0, 0);
          accZ[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(c.a[mt], c.z[nt], accZ[mt][nt], 0, 0, 0);
        }
      }
      if (s + 1 < TK / 16) {
        // per step: the next step's LDS reads first, then each MFMA followed by
        // a few VALU instructions of the next step's sign expansion
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
        }
      }
    }
  };

  fetch();
  store(0);
  __syncthreads();
  if (ntiles > 1) fetch();
  for (int it = 0; it < ntiles; ++it) {
    compute(it & 1);
    if (it + 1 < ntiles) {
      store((it + 1) & 1);
      __syncthreads();
      if (it + 2 < ntiles) fetch();
    }
  }
}

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanh_(float x) { return 1.0f - 2.0f / (__expf(2.0f * x) + 1.0f); }

// Row (within the workgroup's TM) of accumulator element v of row tile mt
// for this lane: 32x32 MFMA output layout.
__device__ __forceinline__ int acc_row(int wm, int mt, int lg, int v) {
  return 64 * wm + 32 * mt + 8 * (v >> 2) + 4 * lg + (v & 3);
}

template <typename T>
__device__ __forceinline__ void zero_acc(T (&acc)[2][2]) {
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = T{};
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

// Workgroup: TM rows x 32 hidden units; LDS column rho = gate * 32 + unit.
// Waves wn = 0 hold gates i, f and waves wn = 1 gates g, o of the same units;
// after the main loop the wn = 1 waves pass their pre-activations through
// LDS and the wn = 0 waves update the cell.
template <int kind>
__global__ __launch_bounds__(NT, 512 / NT) void gate_bf16_kernel(GateArgsB g) {
  extern __shared__ __align__(16) uint16_t smem[];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  const int u0 = blockIdx.x * 32;
  const int64_t m0 = (int64_t)blockIdx.y * TM;
  const int pair = (int)(m0 / g.rm.pair_rows);
  const int H = g.H;
  auto colmap = [&](int rho, int& n) {
    n = (rho >> 5) * H + u0 + (rho & 31);
    return true;
  };
  f16v accW[2][2], accZ[2][2];
  zero_acc(accW);
  zero_acc(accZ);
  const SegB s0{g.x + m0 * g.El, g.El, g.theta + g.off_ih, g.El, g.off_ih, g.El};
  const SegB s1{g.hprev + m0 * H, H, g.theta + g.off_hh, H, g.off_hh, H};
  mainloop_bf16<kind>(accW, accZ, s0, s1, 2, colmap, g.key, g.i0 + (uint32_t)pair, smem);

  // pre-activations of this wave's two gates (2 wn, 2 wn + 1) for unit u
  const int u = u0 + lr;
  float bb[2], zz[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int gate = 2 * wn + nt;
    bb[nt] = bf16_to_f32(g.theta[g.off_b + (uint64_t)(gate * H + u)]);
    zz[nt] = g.zb[(int64_t)pair * 4 * H + gate * H + u];
  }
  __syncthreads();  // the main loop's LDS buffers are free from here on
  float* xg = (float*)smem;  // [TM rows][32 units][2]: pre-activations of gates g, o
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int lrow = acc_row(wm, mt, lg, v);
      const bool neg = (m0 + lrow - (int64_t)pair * g.rm.pair_rows) >= g.rm.Bp;
      const float se = neg ? -g.eps : g.eps;
      float pre[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
        pre[nt] = accW[mt][nt][v] + se * accZ[mt][nt][v] + (neg ? bb[nt] - zz[nt] : bb[nt] + zz[nt]);
      if (wn == 1) *(float2*)(xg + (lrow * 32 + lr) * 2) = float2{pre[0], pre[1]};
      accW[mt][0][v] = pre[0];  // keep i, f (wn == 0) for the cell update
      accW[mt][1][v] = pre[1];
    }
  }
  __syncthreads();
  if (wn == 0) {
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int lrow = acc_row(wm, mt, lg, v);
        const float2 go = *(const float2*)(xg + (lrow * 32 + lr) * 2);
        const float ig = sigm(accW[mt][0][v]), fg = sigm(accW[mt][1][v]);
        const float gg = tanh_(go.x), og = sigm(go.y);
        const int64_t o = (m0 + lrow) * H + u;
        const float c = fg * g.cst[o] + ig * gg;
        g.cst[o] = c;
        g.hout[o] = bf16_rne(og * tanh_(c));
      }
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
__global__ __launch_bounds__(NT, 512 / NT) void head_bf16_kernel(HeadArgsB g) {
  extern __shared__ __align__(16) uint16_t smem[];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % WAVES_M, wn = wave / WAVES_M;
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
  f16v accW[2][2], accZ[2][2];
  zero_acc(accW);
  zero_acc(accZ);
  const SegB s0{g.h + rr0 * g.H, g.H, g.theta + g.off_w, g.H, g.off_w, g.H};
  mainloop_bf16<kind>(accW, accZ, s0, s0, 1, colmap, g.key, g.i0 + (uint32_t)pair, smem);

  int col[2];
  bool cok[2];
  float bb[2], zz[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    col[nt] = v0 + 64 * wn + 32 * nt + lr;
    cok[nt] = col[nt] < V;
    bb[nt] = cok[nt] ? bf16_to_f32(g.theta[g.off_b + (uint64_t)col[nt]]) : 0.f;
    zz[nt] = cok[nt] ? g.zbo[(int64_t)pair * V + col[nt]] : 0.f;
  }
  __syncthreads();  // reuse the main loop's LDS for the cross-wave reduction
  float* red_m = (float*)smem;   // [2][TM]
  float* red_s = red_m + 2 * TM;  // [2][TM]
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int lrow = acc_row(wm, mt, lg, v);
      const int64_t r = r0 + lrow;
      const int loc = (int)(r - (int64_t)pair * g.rm.pair_rows);
      const bool neg = loc >= g.rm.Bp;
      const int b = neg ? loc - g.rm.Bp : loc;
      const float se = neg ? -g.eps : g.eps;
      float y[2];
      float mx = -INFINITY;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        y[nt] = cok[nt] ? accW[mt][nt][v] + se * accZ[mt][nt][v] + (neg ? bb[nt] - zz[nt] : bb[nt] + zz[nt])
                        : -INFINITY;
        mx = fmaxf(mx, y[nt]);
      }
      if (b < g.B) {
        const int tgt = g.tokens[(int64_t)b * (g.C + 1) + g.t0 + tt + 1];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
          if (col[nt] == tgt) g.ptgt[rr0 + lrow] = y[nt];
      }
      // the row's 64 columns of this wave sit in the 32 lanes of this lane half
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      float se2 = 0.f;
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) se2 += cok[nt] ? __expf(y[nt] - mx) : 0.f;
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) se2 += __shfl_xor(se2, off, 64);
      if (lr == 0) {
        red_m[wn * TM + lrow] = mx;
        red_s[wn * TM + lrow] = se2;
      }
    }
  }
  __syncthreads();
  if (t < TM) {
    const float m_a = red_m[t], m_b = red_m[TM + t];
    const float mx = fmaxf(m_a, m_b);
    const float sa = m_a == -INFINITY ? 0.f : red_s[t] * __expf(m_a - mx);
    const float sb = m_b == -INFINITY ? 0.f : red_s[TM + t] * __expf(m_b - mx);
    g.pmax[(int64_t)vt * g.rows + rr0 + t] = mx;
    g.psum[(int64_t)vt * g.rows + rr0 + t] = sa + sb;
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
hipError_t allow_smem(K kernel, size_t bytes) {
  static bool done = false;  // set once per kernel instantiation (same value on every device)
  if (done) return hipSuccess;
  hipError_t e = hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)bytes);
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
    constexpr size_t sb = smem_bytes<ZO_RADEMACHER>();
    if ((e = allow_smem(gate_bf16_kernel<ZO_RADEMACHER>, sb)) != hipSuccess) return e;
    ProfScope ps(kKGate, st);
    gate_bf16_kernel<ZO_RADEMACHER><<<grid, NT, sb, st>>>(g);
  } else {
    constexpr size_t sb = smem_bytes<ZO_GAUSSIAN>();
    if ((e = allow_smem(gate_bf16_kernel<ZO_GAUSSIAN>, sb)) != hipSuccess) return e;
    ProfScope ps(kKGate, st);
    gate_bf16_kernel<ZO_GAUSSIAN><<<grid, NT, sb, st>>>(g);
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
    constexpr size_t sb = smem_bytes<ZO_RADEMACHER>();
    if ((e = allow_smem(head_bf16_kernel<ZO_RADEMACHER>, sb)) != hipSuccess) return e;
    ProfScope ps(kKHead, st);
    head_bf16_kernel<ZO_RADEMACHER><<<grid, NT, sb, st>>>(h);
  } else {
    constexpr size_t sb = smem_bytes<ZO_GAUSSIAN>();
    if ((e = allow_smem(head_bf16_kernel<ZO_GAUSSIAN>, sb)) != hipSuccess) return e;
    ProfScope ps(kKHead, st);
    head_bf16_kernel<ZO_GAUSSIAN><<<grid, NT, sb, st>>>(h);
  }
  return hipGetLastError();
}

}  // namespace zo
