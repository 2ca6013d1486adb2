// The 2N perturbed forward passes of one CD-RGE step (Algorithm 1's probe
// loop; Eq. 2's two loss queries per probe), batched over all passes.
//
// Every pass (probe n, sign s) runs the same LSTM on the same B sequences
// with weights theta + s eps z_n. A matrix product of a timestep is computed
// for all 2N*B rows at once as
//     a[r] = sum_k A[r][k] W[c][k]  +  sum_k (s_r A[r][k]) (eps z_n[c][k])
// i.e. the shared weights times the state plus the probe times the signed
// state, accumulated in one MFMA accumulator. z_n is regenerated tile by
// tile in LDS from (seed, n, parameter offset); theta + s eps z_n is never
// formed in memory.
//
// Per timestep: embed (perturbed embedding rows) -> one gate kernel per
// layer (both input products, bias, gate nonlinearities and the cell update
// fused). Every kTimeChunk timesteps: one output-head kernel over the
// chunk's top-layer states (vocabulary-tiled, online logsumexp partials),
// then a combine kernel that adds each position's cross-entropy to its row.
// At the end a reduction turns row sums into the 2N losses.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <optional>
#include <type_traits>

#include "zo_kernels.hpp"
#include "zo_pack.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int BM = 64;    // rows per workgroup tile
constexpr int BNC = 128;  // columns per workgroup tile
constexpr int BK = 32;    // K per LDS tile
constexpr int LDK = BK + 4;

static_assert(2 * kRowGranuleF32 % BM == 0, "a probe's rows must be a whole number of row tiles");
static_assert(kRowGranuleF32 % 32 == 0, "a 32-row wave tile must lie inside one sign");
static_assert(BNC == kVocabTile, "head vocabulary tile");

// ---------------------------------------------------------------------------
// Bias probes: zb[l][n][c] = eps z_{i0+n}[bias_l + c], zbo[n][v] = eps z[b_out + v]
// (the biases' perturbation is the same for every timestep).
struct BiasOffsets {
  uint64_t layer[kMaxLayers];
};

__global__ __launch_bounds__(256) void prep_bias_kernel(int kind, Key key, uint32_t i0, float eps,
                                                        int N, int L, int H4, int V,
                                                        BiasOffsets bias_off, uint64_t bout_off,
                                                        float* zb, float* zbo) {
  const int64_t per_layer = (int64_t)N * H4;
  const int64_t total = per_layer * L + (int64_t)N * V;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    if (t < per_layer * L) {
      const int l = (int)(t / per_layer);
      const int64_t rem = t - l * per_layer;
      const int n = (int)(rem / H4);
      const int c = (int)(rem - (int64_t)n * H4);
      zb[t] = fmul(eps, probe_value(kind, key, i0 + n, bias_off.layer[l] + c));
    } else {
      const int64_t rem = t - per_layer * L;
      const int n = (int)(rem / V);
      const int v = (int)(rem - (int64_t)n * V);
      zbo[rem] = fmul(eps, probe_value(kind, key, i0 + n, bout_off + v));
    }
  }
}

// ---------------------------------------------------------------------------
// x0[tt][r][e] = EMB[tok][e] + s eps z_n[emb + tok E + e] for the input token
// of row r at time t0 + tt, tt < Tc; zeros for padding rows, NaN for a token
// outside [0, V) (never read). One thread per 4 elements; one launch per time
// chunk.
template <int kind>
__global__ __launch_bounds__(256) void embed_f32_kernel(const float* theta, uint64_t emb_off, int E, int V,
                                                        const int32_t* tokens, int C, int t0, int Tc, int B,
                                                        RowMap rm, int64_t M, Key key, uint32_t i0,
                                                        float eps, float* x0) {
  const int E4 = E >> 2;
  const int64_t total = (int64_t)Tc * M * E4;
  for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * blockDim.x) {
    const int64_t rr = idx / E4;  // row of the chunk: tt M + r
    const int e = (int)(idx - rr * E4) * 4;
    const int tt = (int)(rr / M);
    const int64_t r = rr - (int64_t)tt * M;
    const int t = t0 + tt;
    const PassOf ps = pass_of(rm, r);
    const int pair = ps.probe, b = ps.b;
    f4 out = {0.f, 0.f, 0.f, 0.f};
    const int tok = b < B ? tokens[(int64_t)b * (C + 1) + t] : 0;
    if (b < B && (uint32_t)tok >= (uint32_t)V) {
      out = f4{__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""), __builtin_nanf("")};
    } else if (b < B) {
      const uint64_t j = emb_off + (uint64_t)tok * E + e;
      const f4 w = *(const f4*)(theta + j);
      float z[4];
      if constexpr (kind == ZO_RADEMACHER) {
        const uint32_t word = rademacher_word(key, i0 + pair, j >> 5) >> (uint32_t)(j & 31u);
#pragma unroll
        for (int q = 0; q < 4; ++q) z[q] = ((word >> q) & 1u) ? 1.0f : -1.0f;
      } else {
        gauss_block(key, i0 + pair, j >> 2, z);
      }
      const float se = (float)ps.sign * eps;  // 0 for the clean pass: out = w
#pragma unroll
      for (int q = 0; q < 4; ++q) out[q] = w[q] + fmul(se, z[q]);
    }
    *(f4*)(x0 + rr * E + e) = out;
  }
}

// ---------------------------------------------------------------------------
// fp32 MFMA main loop shared by the gate and head kernels.
//
// Workgroup tile: 32 RM rows x BNC=128 columns (RM = 2: 64 rows, 4 waves;
// RM = 4: 128 rows, 8 waves, where a probe's rows come in blocks of 128, which
// loads a third fewer bytes per flop), waves in RM (rows) x 2 (columns); each
// wave owns 2 row tiles x 4 column tiles of 16x16 and runs
// v_mfma_f32_16x16x4_f32. Within a K tile of 32, lane group g (lane/16) feeds
// k = 8g + s at MFMA step s, so each lane reads 8 consecutive k with two
// 128-bit LDS loads (the order in which k is summed is free).
//
// Every 32-row wave tile lies inside one sign half of one probe's rows, so a
// wave needs a single weight operand: W + eps z (rows of the + pass) or
// W - eps z (rows of the - pass). The loader threads form both tiles in LDS
// from the weight tile and the regenerated probe tile (one fp32 rounding of
// w +- eps z), and each wave runs one MFMA stream over its own tile. The
// split variant (kSplit) keeps W and eps z apart and runs two MFMA streams,
// W.h and (s h).(eps z), into one accumulator (twice the MFMA work).
//
// Software pipeline: the next K tile's global loads and probe generation are
// issued before the current tile's MFMAs, so their latency overlaps the
// matrix work; LDS holds one tile (A [32 RM][36], two weight tiles [128][36]).
struct Seg {
  const float* A;  // row r of this tile at A + r * lda
  int64_t lda;
  const float* W;  // weight row n at W + n * ldw
  int64_t ldw;
  uint64_t zoff;   // offset of W inside theta (probe coordinates)
  int K;
  const float* Z;  // kGaussCached: eps z of this probe and matrix, laid out like W
};

template <int RM>
struct SmemT {
  float a[32 * RM * LDK];
  float p[BNC * LDK];  // W + eps z (split: W)
  float m[BNC * LDK];  // W - eps z (split: eps z)
};
using Smem = SmemT<BM / 32>;

// colmap(rho, &n) -> true if LDS column rho maps to a real weight row n.
// fd: forward differences: the second tile holds W itself (the clean pass)
// instead of W - eps z.
template <int kind, bool kSplit, int RM = 2, typename ColMap>
__device__ __forceinline__ void mainloop_f32(f4 (&acc)[2][4], const Seg s0, const Seg s1,
                                             int nseg, ColMap colmap, const int (&wrow)[4], int arow0,
                                             bool wave_neg, Key key, uint32_t probe, float eps,
                                             bool fd, SmemT<RM>& sm) {
  constexpr int NT = 128 * RM;     // threads
  constexpr int PPR = NT / BNC;    // loader threads per weight row
  constexpr int KPT = BK / PPR;    // consecutive k per loader thread
  constexpr int NW4 = KPT / 4;     // float4 weight loads per thread
  static_assert(PPR * KPT == BK && KPT % 4 == 0 && 32 * RM * 8 == 2 * NT, "loader roles");
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int g4 = lane >> 4;
  // loader roles: A rows (t + NT q) >> 3, float4 column t & 7; weight row
  // rho = t / PPR, KPT consecutive k starting at KPT * (t % PPR)
  const int rho = t / PPR, part = t % PPR;
  int wn;
  const bool wok = colmap(rho, wn);
  const int ntiles = s0.K / BK + (nseg > 1 ? s1.K / BK : 0);

  f4 ra[2], rw[NW4];
  float zv[KPT];
  Words zcache{{0u, 0u, 0u, 0u}};
  int seg = 0, k0 = 0;  // position of the tile being fetched

  auto fetch = [&]() {
    const Seg sg = seg == 0 ? s0 : s1;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = t + NT * q;
      ra[q] = *(const f4*)(sg.A + (int64_t)(idx >> 3) * sg.lda + k0 + 4 * (idx & 7));
    }
    const float* wp = sg.W + (int64_t)wn * sg.ldw + k0 + KPT * part;
#pragma unroll
    for (int q = 0; q < NW4; ++q) rw[q] = wok ? *(const f4*)(wp + 4 * q) : f4{0.f, 0.f, 0.f, 0.f};
    const uint64_t jrow = sg.zoff + (uint64_t)wn * (uint64_t)sg.ldw + (uint64_t)k0;
    if constexpr (kind == ZO_RADEMACHER) {
      uint32_t word;
      const bool aligned = (sg.zoff % 128u) == 0 && (sg.ldw % 128) == 0;
      if (aligned) {
        if ((k0 & 127) == 0) zcache = stream_block(key, jrow >> 7, probe, kTagRademacher);
        const int q = (k0 >> 5) & 3;
        word = q == 0 ? zcache.w[0] : q == 1 ? zcache.w[1] : q == 2 ? zcache.w[2] : zcache.w[3];
      } else {
        word = rademacher_word(key, probe, jrow >> 5);
      }
      word >>= KPT * part;
#pragma unroll
      for (int e = 0; e < KPT; ++e) zv[e] = ((word >> e) & 1u) ? eps : -eps;
    } else if constexpr (kind == kGaussCached) {
      const float* zp = sg.Z + (int64_t)wn * sg.ldw + k0 + KPT * part;
#pragma unroll
      for (int q = 0; q < NW4; ++q) {
        const f4 v = wok ? *(const f4*)(zp + 4 * q) : f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int e = 0; e < 4; ++e) zv[4 * q + e] = v[e];
      }
    } else {
      const uint64_t j0 = jrow + KPT * part;
#pragma unroll
      for (int b = 0; b < NW4; ++b) {
        float z4[4];
        gauss_block(key, probe, (j0 >> 2) + b, z4);
#pragma unroll
        for (int e = 0; e < 4; ++e) zv[4 * b + e] = fmul(eps, z4[e]);
      }
    }
    k0 += BK;
    if (k0 == sg.K) {
      k0 = 0;
      ++seg;
    }
  };

  fetch();
  for (int it = 0; it < ntiles; ++it) {
    __syncthreads();  // the previous tile's fragments have been read
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int idx = t + NT * q;
      *(f4*)(&sm.a[(idx >> 3) * LDK + 4 * (idx & 7)]) = ra[q];
    }
#pragma unroll
    for (int q = 0; q < NW4; ++q) {
      f4 vp, vm;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float w = rw[q][e], z = zv[4 * q + e];
        if constexpr (kSplit) {
          vp[e] = w;
          vm[e] = z;
        } else {
          vp[e] = fadd(w, z);
          vm[e] = fadd(w, fd ? 0.0f : -z);
        }
      }
      *(f4*)(&sm.p[rho * LDK + KPT * part + 4 * q]) = vp;
      *(f4*)(&sm.m[rho * LDK + KPT * part + 4 * q]) = vm;
    }
    __syncthreads();
    if (it + 1 < ntiles) fetch();  // next tile's loads and probe overlap this tile's MFMAs

    f4 a[2][2], b[4][2], z[4][2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const float* pa = &sm.a[(arow0 + 16 * mt + (lane & 15)) * LDK + 8 * g4];
      a[mt][0] = *(const f4*)pa;
      a[mt][1] = *(const f4*)(pa + 4);
    }
    const float* bsrc = (!kSplit && wave_neg) ? sm.m : sm.p;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float* pb = &bsrc[wrow[q] * LDK + 8 * g4];
      b[q][0] = *(const f4*)pb;
      b[q][1] = *(const f4*)(pb + 4);
      if constexpr (kSplit) {
        const float* pz = &sm.m[wrow[q] * LDK + 8 * g4];
        z[q][0] = *(const f4*)pz;
        z[q][1] = *(const f4*)(pz + 4);
      }
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const float av = a[mt][s >> 2][s & 3];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          acc[mt][q] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, b[q][s >> 2][s & 3], acc[mt][q], 0, 0, 0);
          if constexpr (kSplit) {
            const float sav = wave_neg ? -av : av;
            acc[mt][q] = __builtin_amdgcn_mfma_f32_16x16x4f32(sav, z[q][s >> 2][s & 3], acc[mt][q], 0, 0, 0);
          }
        }
      }
    }
  }
}

__device__ __forceinline__ float sigmoidf_(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanhf_(float x) { return 1.0f - 2.0f / (__expf(2.0f * x) + 1.0f); }

// ---------------------------------------------------------------------------
// One LSTM layer at one timestep for all rows:
//   a = W_ih x + W_hh h + b  (+ s eps (Z_ih x + Z_hh h + z_b))
//   i, f, o = sigmoid, g = tanh; c <- f c + i g; h <- o tanh(c)
// Workgroup: 32 RM rows x 32 hidden units (4 gates x 32 = 128 columns); LDS
// column rho = gate * 32 + unit. One launch runs up to kLaunchLayers layers,
// each at its own timestep (blockIdx.z picks the layer): the step is a
// wavefront over (layer, timestep) in which layer l at time t and layer l + 1
// at time t - 1 are independent.
constexpr int kLaunchLayers = 8;
struct GateLayer {
  const float* x;      // [M][El]
  const float* hprev;  // [M][H]
  float* hout;         // [M][H]
  float* cst;          // [M][H]
  uint64_t off_ih, off_hh, off_b;
  int El;
  const float* zb;     // [N][4H] eps z of this layer's bias
  const float* zc_ih;  // probe cache: W_ih's and W_hh's values of probe 0; probe n at + n * zc_stride
  const float* zc_hh;
};
struct GateArgs {
  GateLayer layer[kLaunchLayers];
  const float* theta;
  int H;
  Key key;
  uint32_t i0;
  float eps;
  RowMap rm;
  uint64_t zc_stride;
};

// 128-row workgroups are held to 128 VGPRs (four waves per SIMD), so that two
// of them share a CU and each hides the other's tile loads.
template <int kind, bool kSplit, int RM>
__global__ __launch_bounds__(128 * RM, RM == 4 ? 4 : 2) void gate_f32_kernel(GateArgs g) {
  __shared__ SmemT<RM> sm;
  const GateLayer& gl = g.layer[blockIdx.z];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % RM, wn = wave / RM;
  const int u0 = blockIdx.x * 32;
  const int64_t m0 = (int64_t)blockIdx.y * (32 * RM);
  const int pair = pass_of(g.rm, m0).probe;
  const int H = g.H;
  auto colmap = [&](int rho, int& n) {
    n = (rho >> 5) * H + u0 + (rho & 31);
    return true;
  };
  int wrow[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) wrow[q] = q * 32 + 16 * wn + (lane & 15);
  // a 32-row wave tile lies inside one pass: one sign (+1, -1, or 0 clean)
  const int ws = pass_of(g.rm, m0 + 32 * wm).sign;
  const bool wave_neg = ws <= 0;  // tile W - eps z, or W for the clean pass
  f4 acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[mt][q] = f4{0.f, 0.f, 0.f, 0.f};

  const uint32_t probe = g.i0 + (uint32_t)pair;
  const uint64_t zpos = (uint64_t)pair * g.zc_stride;
  const Seg s0{gl.x + m0 * gl.El, gl.El, g.theta + gl.off_ih, gl.El, gl.off_ih, gl.El,
               kind == kGaussCached ? gl.zc_ih + zpos : nullptr};
  const Seg s1{gl.hprev + m0 * H, H, g.theta + gl.off_hh, H, gl.off_hh, H,
               kind == kGaussCached ? gl.zc_hh + zpos : nullptr};
  mainloop_f32<kind, kSplit, RM>(acc, s0, s1, 2, colmap, wrow, 32 * wm, wave_neg, g.key, probe, g.eps,
                                 g.rm.fd != 0, sm);

  // epilogue: lane holds rows 4*(lane/16)+v of each row tile, unit u
  const int u = u0 + 16 * wn + (lane & 15);
  const float* bias = g.theta + gl.off_b;
  const float* zb = gl.zb + (int64_t)pair * 4 * H;
  float bs[4];  // bias + eps z_b, bias - eps z_b, or the bias (clean pass)
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float bb = bias[q * H + u], zz = zb[q * H + u];
    bs[q] = ws > 0 ? bb + zz : ws < 0 ? bb - zz : bb;
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t r = m0 + 32 * wm + 16 * mt + 4 * (lane >> 4) + v;
      const float ai = acc[mt][0][v] + bs[0];
      const float af = acc[mt][1][v] + bs[1];
      const float ag = acc[mt][2][v] + bs[2];
      const float ao = acc[mt][3][v] + bs[3];
      const float ig = sigmoidf_(ai), fg = sigmoidf_(af), gg = tanhf_(ag), og = sigmoidf_(ao);
      const int64_t o = r * H + u;
      const float c = fg * gl.cst[o] + ig * gg;
      gl.cst[o] = c;
      gl.hout[o] = og * tanhf_(c);
    }
  }
}

// ---------------------------------------------------------------------------
// Output head over a chunk of timesteps: rows rr = tt*M + r of the chunk's
// top-layer states. Logits y = W_out h + b_out (+ s eps (Z_out h + z_bout))
// for a 128-wide vocabulary tile; the tile's running max and sum of
// exp(y - max) per row go to pmax/psum, and the logit of the target token is
// written by the tile that holds it.
struct HeadArgs {
  const float* h;  // [Tc*M][H]
  const float* theta;
  uint64_t off_w, off_b;
  int H, V;
  const float* zbo;  // [N][V]
  Key key;
  uint32_t i0;
  float eps;
  RowMap rm;
  int64_t M;
  int64_t rows;  // Tc * M
  const int32_t* tokens;
  int C, t0, B;
  float* pmax;  // [nvt][rows]
  float* psum;
  float* ptgt;  // [rows]
  const float* zc_out;  // probe cache: W_out's values of probe 0; probe n at + n * zc_stride
  uint64_t zc_stride;
};

template <int kind, bool kSplit>
__global__ __launch_bounds__(256) void head_f32_kernel(HeadArgs g) {
  __shared__ Smem sm;
  __shared__ float red_m[2][BM], red_s[2][BM];
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int vt = blockIdx.x;
  const int v0 = vt * BNC;
  const int64_t rr0 = (int64_t)blockIdx.y * BM;
  const int tt = (int)(rr0 / g.M);
  const int64_t r0 = rr0 - (int64_t)tt * g.M;
  const int pair = pass_of(g.rm, r0).probe;
  const int V = g.V;
  auto colmap = [&](int rho, int& n) {
    n = v0 + rho;
    const bool ok = n < V;
    if (!ok) n = 0;
    return ok;
  };
  int wrow[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) wrow[q] = 64 * wn + 16 * q + (lane & 15);
  // a 32-row wave tile lies inside one pass: one sign (+1, -1, or 0 clean)
  const int ws = pass_of(g.rm, r0 + 32 * wm).sign;
  const bool wave_neg = ws <= 0;
  f4 acc[2][4];
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[mt][q] = f4{0.f, 0.f, 0.f, 0.f};
  const uint32_t probe = g.i0 + (uint32_t)pair;
  const Seg s0{g.h + rr0 * g.H, g.H, g.theta + g.off_w, g.H, g.off_w, g.H,
               kind == kGaussCached ? g.zc_out + (uint64_t)pair * g.zc_stride : nullptr};
  mainloop_f32<kind, kSplit>(acc, s0, s0, 1, colmap, wrow, 32 * wm, wave_neg, g.key, probe, g.eps,
                             g.rm.fd != 0, sm);

  const float* bout = g.theta + g.off_b;
  const float* zbo = g.zbo + (int64_t)pair * V;
  float bs[4];  // bias + eps z_b, bias - eps z_b, or the bias (clean pass)
  bool cok[4];
  int col[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    col[q] = v0 + 64 * wn + 16 * q + (lane & 15);
    cok[q] = col[q] < V;
    const float bb = cok[q] ? bout[col[q]] : 0.f, zz = cok[q] ? zbo[col[q]] : 0.f;
    bs[q] = ws > 0 ? bb + zz : ws < 0 ? bb - zz : bb;
  }
#pragma unroll
  for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int lrow = 32 * wm + 16 * mt + 4 * (lane >> 4) + v;
      const int b = pass_of(g.rm, r0 + lrow).b;
      float y[4];
      float mx = -INFINITY;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        y[q] = cok[q] ? acc[mt][q][v] + bs[q] : -INFINITY;
        mx = fmaxf(mx, y[q]);
      }
      if (b < g.B) {
        const int tgt = g.tokens[(int64_t)b * (g.C + 1) + g.t0 + tt + 1];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (col[q] == tgt) g.ptgt[rr0 + lrow] = y[q];
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      float se = 0.f;
#pragma unroll
      for (int q = 0; q < 4; ++q) se += cok[q] ? __expf(y[q] - mx) : 0.f;
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) se += __shfl_xor(se, off, 64);
      if ((lane & 15) == 0) {
        red_m[wn][lrow] = mx;
        red_s[wn][lrow] = se;
      }
    }
  }
  __syncthreads();
  if (t < BM) {
    const float m_a = red_m[0][t], m_b = red_m[1][t];
    const float mx = fmaxf(m_a, m_b);
    const float sa = m_a == -INFINITY ? 0.f : red_s[0][t] * __expf(m_a - mx);
    const float sb = m_b == -INFINITY ? 0.f : red_s[1][t] * __expf(m_b - mx);
    g.pmax[(int64_t)vt * g.rows + rr0 + t] = mx;
    g.psum[(int64_t)vt * g.rows + rr0 + t] = sa + sb;
  }
}

// ---------------------------------------------------------------------------
// Cross-entropy of every position of the chunk: logsumexp over the
// vocabulary tiles' (max, sum of exp) partials, merged online in tile order,
// minus the target logit. One thread per (timestep, row); the loss replaces
// the target logit in ptgt (0 for unscored positions and padding rows, NaN
// for a scored position whose target token lies outside [0, V)).
__global__ __launch_bounds__(256) void combine_kernel(const float* pmax, const float* psum,
                                                      float* ptgt, int nvt, int64_t rows,
                                                      int64_t M, int t0, int C, int B, RowMap rm,
                                                      const uint8_t* mask, const int32_t* tokens, int V) {
  const int64_t rr = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (rr >= rows) return;
  const int tt = (int)(rr / M);
  const int64_t r = rr - (int64_t)tt * M;
  const int b = pass_of(rm, r).b;
  if (b >= B || (mask && !mask[(int64_t)b * C + t0 + tt])) {
    ptgt[rr] = 0.f;
    return;
  }
  if ((uint32_t)tokens[(int64_t)b * (C + 1) + t0 + tt + 1] >= (uint32_t)V) {
    ptgt[rr] = __builtin_nanf("");
    return;
  }
  float mx = -INFINITY, s = 0.f;
  for (int v = 0; v < nvt; ++v) {
    const float m = pmax[(int64_t)v * rows + rr];
    const float e = psum[(int64_t)v * rows + rr];
    if (m == -INFINITY) continue;
    if (m > mx) {
      s = s * expf(mx - m) + e;
      mx = m;
    } else {
      s += e * expf(m - mx);
    }
  }
  ptgt[rr] = mx + logf(s) - ptgt[rr];
}

// Adds the chunk's per-position losses to each row's running sum, in time
// order (a fixed summation order: the result does not depend on scheduling).
__global__ __launch_bounds__(256) void accumulate_kernel(const float* ell, int64_t M, int Tc,
                                                         double* row_loss) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= M) return;
  double acc = row_loss[r];
  for (int tt = 0; tt < Tc; ++tt) acc += (double)ell[(int64_t)tt * M + r];
  row_loss[r] = acc;
}

// Loss of each pass = (sum over the pass's sequences of their row sums) /
// (scored positions). Central differences: pass 2n -> Lp[n], 2n+1 -> Lm[n];
// forward differences: pass p < N -> Lp[p], the clean pass N -> Lm[0].
__global__ __launch_bounds__(256) void reduce_kernel(const double* row_loss, int N, int B, int C,
                                                     RowMap rm, const uint8_t* mask, float* Lp,
                                                     float* Lm) {
  __shared__ double part[256];
  double cnt = 0.0;
  if (mask) {
    for (int64_t k = threadIdx.x; k < (int64_t)B * C; k += blockDim.x) cnt += mask[k] ? 1.0 : 0.0;
  } else if (threadIdx.x == 0) {
    cnt = (double)B * (double)C;
  }
  part[threadIdx.x] = cnt;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) part[threadIdx.x] += part[threadIdx.x + s];
    __syncthreads();
  }
  const double total = part[0];
  const int npass = rm.fd ? N + 1 : 2 * N;
  for (int p = threadIdx.x; p < npass; p += blockDim.x) {
    double s = 0.0;
    const double* rl = row_loss + (int64_t)p * rm.Bp;
    for (int b = 0; b < B; ++b) s += rl[b];
    const float L = total > 0.0 ? (float)(s / total) : 0.0f;
    if (rm.fd) {
      if (p < N) Lp[p] = L;
      else Lm[0] = L;
    } else if (p & 1) {
      Lm[p >> 1] = L;
    } else {
      Lp[p >> 1] = L;
    }
  }
}

// Zero n16 16-byte words. A kernel rather than a memset, so that a caller can
// capture the forward into a graph and replay it.
__global__ __launch_bounds__(256) void zero_kernel(uint4* p, uint64_t n16) {
  const uint64_t stride = (uint64_t)gridDim.x * 256u;
  for (uint64_t i = (uint64_t)blockIdx.x * 256u + threadIdx.x; i < n16; i += stride) p[i] = uint4{0u, 0u, 0u, 0u};
}

// bytes: a multiple of 16 at a 16-byte aligned address (every workspace buffer is).
hipError_t zero_async(void* p, size_t bytes, hipStream_t st) {
  if (bytes == 0) return hipSuccess;
  if ((bytes & 15u) || ((uintptr_t)p & 15u)) return hipErrorInvalidValue;
  const uint64_t n16 = bytes / 16;
  uint64_t grid = (n16 + 255) / 256;
  if (grid > 8192) grid = 8192;
  zero_kernel<<<dim3((unsigned)grid), dim3(256), 0, st>>>((uint4*)p, n16);
  return hipGetLastError();
}

// Probe cache fill of the fp32 path: eps z of every weight matrix for probes
// i0 .. i0+N-1 (layout: ZCacheMap, row-major matrices). The values are the
// ones the forward kernels compute when they regenerate the probe,
// fp32(eps * z) of the same normal value z. One thread per Philox block (4
// values); the matrices are listed by their start in a probe's block and in
// theta.
struct ZSegs {
  int n;
  uint64_t cstart[2 * kMaxLayers + 2];  // start of matrix m in a probe's block; cstart[n] = P_g
  uint64_t toff[2 * kMaxLayers + 1];    // offset of matrix m in theta
};

__global__ __launch_bounds__(256) void zcache_fill_kernel(float* zc, ZSegs segs, Key key, uint32_t i0, int N,
                                                          float eps) {
  const uint64_t pg = segs.cstart[segs.n];
  const uint64_t nb = pg >> 2;
  for (int n = blockIdx.y; n < N; n += gridDim.y) {
    float* zp = zc + (uint64_t)n * pg;
    for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < nb;
         b += (uint64_t)gridDim.x * blockDim.x) {
      const uint64_t u = b << 2;
      int m = 0;
      while (m + 1 < segs.n && u >= segs.cstart[m + 1]) ++m;
      const uint64_t j = segs.toff[m] + (u - segs.cstart[m]);
      float z[4];
      gauss_block(key, i0 + (uint32_t)n, j >> 2, z);
      *(f4*)(zp + u) = f4{fmul(eps, z[0]), fmul(eps, z[1]), fmul(eps, z[2]), fmul(eps, z[3])};
    }
  }
}

// The bf16 path's product matrices in fragment-packed order (zo_pack.hpp):
// their packed start (ZCacheMap offsets, in values), their offset in theta,
// K, and whether the matrix is the head (vocabulary rows, zero-padded) or a
// gate matrix (4H rows in the gate column order).
struct PackSegs {
  int n;
  int64_t H, V;
  uint64_t cstart[2 * kMaxLayers + 2];  // cstart[n] = P_g (padded)
  uint64_t toff[2 * kMaxLayers + 1];
  int64_t K[2 * kMaxLayers + 1];
  int head[2 * kMaxLayers + 1];
};

// Theta row of packed chunk u (16 bytes) of matrix m and its first k;
// row < 0 for the head's padding rows.
__device__ __forceinline__ void packed_source(const PackSegs& segs, uint64_t chunk, int& m, int64_t& row,
                                              int64_t& k) {
  const uint64_t u = chunk << 3;
  m = 0;
  while (m + 1 < segs.n && u >= segs.cstart[m + 1]) ++m;
  const PackedChunk pc = packed_chunk((u - segs.cstart[m]) >> 3, segs.K[m]);
  row = segs.head[m] ? (pc.col < segs.V ? pc.col : -1) : gate_row_of_column(pc.col, segs.H);
  k = pc.k;
}

// fp16 copy of the bf16 weight matrices, fragment-packed, read by the bf16
// path's products in place of theta: bf16 -> fp32 is exact and fp32 -> fp16
// rounds to nearest even, exact for every bf16 weight in [2^-14, 65504)
// (smaller ones keep an absolute error below 2^-25). One thread per packed
// 16-byte chunk (8 consecutive k of one row, 16 bytes of theta).
__global__ __launch_bounds__(256) void w16_pack_kernel(const uint16_t* theta, uint16_t* w16, PackSegs segs) {
  const uint64_t nchunks = segs.cstart[segs.n] >> 3;
  for (uint64_t q = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nchunks;
       q += (uint64_t)gridDim.x * blockDim.x) {
    int m;
    int64_t row, k;
    packed_source(segs, q, m, row, k);
    uint32_t o[4] = {0u, 0u, 0u, 0u};
    if (row >= 0) {
      const uint4 v = *(const uint4*)(theta + segs.toff[m] + (uint64_t)row * (uint64_t)segs.K[m] + (uint64_t)k);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int d = 0; d < 4; ++d)
        o[d] = pack_f16x2(bf16_to_f32((uint16_t)w[d]), bf16_to_f32((uint16_t)(w[d] >> 16)));
    }
    *(uint4*)(w16 + (q << 3)) = uint4{o[0], o[1], o[2], o[3]};
  }
}

// Probe cache of the bf16 path: fp16(eps z) of every product matrix,
// fragment-packed like the weight copy, for probes i0 .. i0 + N - 1. One
// thread per packed chunk: 8 consecutive elements j (a multiple of 8), two
// Philox blocks; zeros for the head's padding rows. The values are those the
// kernels compute when they regenerate the probe.
// w +- z for two packed fp16 pairs, each rounded once to nearest even (the
// value the products' fused form computes in registers from w and z).
__device__ __forceinline__ uint32_t add_f16x2(uint32_t w, uint32_t z, bool minus) {
  typedef _Float16 h2 __attribute__((ext_vector_type(2)));
  const h2 a = __builtin_bit_cast(h2, w), b = __builtin_bit_cast(h2, z);
  return __builtin_bit_cast(uint32_t, minus ? a - b : a + b);
}

// bf16 weights: the probe cache in the packed order of the fp16 weight copy.
// perturbed = false: probe n's fp16(eps z) at n pg. perturbed = true: probe
// n's perturbed weights fp16(w + fp16(eps z)) at 2n pg and fp16(w - fp16(eps
// z)) at (2n + 1) pg, from the packed fp16 weights w16 (written before).
__global__ __launch_bounds__(256) void zcache_pack_kernel(uint16_t* zc, const uint16_t* w16, PackSegs segs, Key key,
                                                          uint32_t i0, int N, float eps, bool perturbed) {
  const uint64_t pg = segs.cstart[segs.n];
  const uint64_t nchunks = pg >> 3;
  for (int n = blockIdx.y; n < N; n += gridDim.y) {
    for (uint64_t q = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; q < nchunks;
         q += (uint64_t)gridDim.x * blockDim.x) {
      int m;
      int64_t row, k;
      packed_source(segs, q, m, row, k);
      uint32_t o[4] = {0u, 0u, 0u, 0u};
      if (row >= 0) {
        const uint64_t j = segs.toff[m] + (uint64_t)row * (uint64_t)segs.K[m] + (uint64_t)k;
        float za[4], zb[4];
        gauss_block(key, i0 + (uint32_t)n, j >> 2, za);
        gauss_block(key, i0 + (uint32_t)n, (j >> 2) + 1, zb);
        o[0] = pack_f16x2(fmul(eps, za[0]), fmul(eps, za[1]));
        o[1] = pack_f16x2(fmul(eps, za[2]), fmul(eps, za[3]));
        o[2] = pack_f16x2(fmul(eps, zb[0]), fmul(eps, zb[1]));
        o[3] = pack_f16x2(fmul(eps, zb[2]), fmul(eps, zb[3]));
      }
      if (!perturbed) {
        *(uint4*)(zc + (uint64_t)n * pg + (q << 3)) = uint4{o[0], o[1], o[2], o[3]};
      } else {
        // padding rows: w = 0 and z = 0
        const uint4 w = *(const uint4*)(w16 + (q << 3));
        *(uint4*)(zc + (uint64_t)(2 * n) * pg + (q << 3)) =
            uint4{add_f16x2(w.x, o[0], false), add_f16x2(w.y, o[1], false), add_f16x2(w.z, o[2], false),
                  add_f16x2(w.w, o[3], false)};
        *(uint4*)(zc + (uint64_t)(2 * n + 1) * pg + (q << 3)) =
            uint4{add_f16x2(w.x, o[0], true), add_f16x2(w.y, o[1], true), add_f16x2(w.z, o[2], true),
                  add_f16x2(w.w, o[3], true)};
      }
    }
  }
}

}  // namespace

namespace {

// The product matrices in theta order: their start in a probe-cache block
// (fp32 path) and in theta.
ZSegs matrix_segments(const ForwardArgs& a) {
  const zo_config& c = a.cfg;
  ZSegs segs{};
  int m = 0;
  for (int l = 0; l < c.n_layers; ++l) {
    segs.cstart[m] = a.zmap.ih[l];
    segs.toff[m++] = a.lay.w_ih[l];
    segs.cstart[m] = a.zmap.hh[l];
    segs.toff[m++] = a.lay.w_hh[l];
  }
  segs.cstart[m] = a.zmap.out;
  segs.toff[m++] = a.lay.w_out;
  segs.n = m;
  segs.cstart[m] = a.zmap.pg;
  return segs;
}

// The same matrices for the bf16 path's packed fp16 weight copy and probe
// cache.
PackSegs packed_segments(const ForwardArgs& a) {
  const zo_config& c = a.cfg;
  PackSegs segs{};
  segs.H = c.hidden;
  segs.V = c.vocab;
  int m = 0;
  for (int l = 0; l < c.n_layers; ++l) {
    segs.cstart[m] = a.zmap.ih[l];
    segs.toff[m] = a.lay.w_ih[l];
    segs.K[m] = l == 0 ? c.embed : c.hidden;
    segs.head[m++] = 0;
    segs.cstart[m] = a.zmap.hh[l];
    segs.toff[m] = a.lay.w_hh[l];
    segs.K[m] = c.hidden;
    segs.head[m++] = 0;
  }
  segs.cstart[m] = a.zmap.out;
  segs.toff[m] = a.lay.w_out;
  segs.K[m] = c.hidden;
  segs.head[m++] = 1;
  segs.n = m;
  segs.cstart[m] = a.zmap.pg;
  return segs;
}

hipError_t launch_w16_fill(const ForwardArgs& a, hipStream_t st) {
  const PackSegs segs = packed_segments(a);
  uint64_t grid = (a.zmap.pg / 8 + 255) / 256;
  if (grid > 16384) grid = 16384;
  ProfScope ps(kKWeights16, st);
  w16_pack_kernel<<<dim3((unsigned)grid), 256, 0, st>>>((const uint16_t*)a.theta, (uint16_t*)a.w16, segs);
  return hipGetLastError();
}

hipError_t launch_zcache_fill(const ForwardArgs& a, hipStream_t st) {
  const zo_config& c = a.cfg;
  const unsigned gy = (unsigned)(a.rows.N < 65535 ? a.rows.N : 65535);
  const Key key = make_key(a.seed);
  ProfScope ps(kKProbeCache, st);
  if (c.wdtype == ZO_WBF16) {
    const PackSegs segs = packed_segments(a);
    uint64_t gx = (a.zmap.pg / 8 + 255) / 256;
    if (gx > 4096) gx = 4096;
    // fused products read the perturbed weights; two-stream ones fp16(eps z)
    zcache_pack_kernel<<<dim3((unsigned)gx, gy), 256, 0, st>>>((uint16_t*)a.zc, (const uint16_t*)a.w16, segs, key,
                                                                a.i0, a.rows.N, a.eps, !a.split);
  } else {
    const ZSegs segs = matrix_segments(a);
    uint64_t gx = (a.zmap.pg / 4 + 255) / 256;
    if (gx > 4096) gx = 4096;
    zcache_fill_kernel<<<dim3((unsigned)gx, gy), 256, 0, st>>>((float*)a.zc, segs, key, a.i0, a.rows.N, a.eps);
  }
  return hipGetLastError();
}

// Perturbed embeddings of timesteps t0 .. t0 + Tc - 1 into x0 [Tc][M][E].
hipError_t launch_embed_f32(const ForwardArgs& a, int t0, int Tc, void* x0, hipStream_t st) {
  const Rows& R = a.rows;
  const int E = a.cfg.embed;
  const RowMap rm = row_map(R);
  const int64_t n = (int64_t)Tc * R.M * (E / 4);
  const unsigned grid = (unsigned)std::min<int64_t>((n + 255) / 256, (int64_t)1 << 20);
  const Key key = make_key(a.seed);
  ProfScope ps(kKEmbed, st);
  if (a.cfg.probe == ZO_RADEMACHER)
    embed_f32_kernel<ZO_RADEMACHER><<<grid, 256, 0, st>>>((const float*)a.theta, a.lay.emb, E,
                                                          a.cfg.vocab, a.tokens, a.C, t0, Tc, R.B, rm, R.M, key, a.i0,
                                                          a.eps, (float*)x0);
  else
    embed_f32_kernel<ZO_GAUSSIAN><<<grid, 256, 0, st>>>((const float*)a.theta, a.lay.emb, E,
                                                        a.cfg.vocab, a.tokens, a.C, t0, Tc, R.B, rm, R.M, key, a.i0,
                                                        a.eps, (float*)x0);
  return hipGetLastError();
}

// One fp32 gate launch over n (<= kLaunchLayers) layer-timesteps.
hipError_t launch_gates_f32(const ForwardArgs& a, const GateLayer* ls, int n, hipStream_t st) {
  if (n < 1 || n > kLaunchLayers) return hipErrorInvalidValue;
  const Rows& R = a.rows;
  GateArgs g{};
  for (int i = 0; i < n; ++i) g.layer[i] = ls[i];
  g.theta = (const float*)a.theta;
  g.H = a.cfg.hidden;
  g.key = make_key(a.seed);
  g.i0 = a.i0;
  g.eps = a.eps;
  g.rm = row_map(R);
  g.zc_stride = a.zmap.pg;
  const bool split = a.split;
  // 128-row workgroups where every block of 128 rows lies inside one probe's rows
  const bool wide = R.pair_rows % 128 == 0;
  auto go = [&](auto rm_tag) {
    constexpr int RM = decltype(rm_tag)::value;
    const dim3 grid((unsigned)(g.H / 32), (unsigned)(R.M / (32 * RM)), (unsigned)n);
    ProfScope ps(kKGate, st);
    if (a.cfg.probe == ZO_RADEMACHER) {
      if (split) gate_f32_kernel<ZO_RADEMACHER, true, RM><<<grid, 128 * RM, 0, st>>>(g);
      else gate_f32_kernel<ZO_RADEMACHER, false, RM><<<grid, 128 * RM, 0, st>>>(g);
    } else if (a.zc) {
      if (split) gate_f32_kernel<kGaussCached, true, RM><<<grid, 128 * RM, 0, st>>>(g);
      else gate_f32_kernel<kGaussCached, false, RM><<<grid, 128 * RM, 0, st>>>(g);
    } else {
      if (split) gate_f32_kernel<ZO_GAUSSIAN, true, RM><<<grid, 128 * RM, 0, st>>>(g);
      else gate_f32_kernel<ZO_GAUSSIAN, false, RM><<<grid, 128 * RM, 0, st>>>(g);
    }
  };
  if (wide) go(std::integral_constant<int, 4>{});
  else go(std::integral_constant<int, 2>{});
  return hipGetLastError();
}

hipError_t launch_head_f32(const ForwardArgs& a, const void* hist, int t0, int Tc, const float* zbo,
                           float* pmax, float* psum, float* ptgt, hipStream_t st) {
  const Rows& R = a.rows;
  HeadArgs h;
  h.h = (const float*)hist;
  h.theta = (const float*)a.theta;
  h.off_w = a.lay.w_out;
  h.off_b = a.lay.b_out;
  h.H = a.cfg.hidden;
  h.V = a.cfg.vocab;
  h.zbo = zbo;
  h.key = make_key(a.seed);
  h.i0 = a.i0;
  h.eps = a.eps;
  h.rm = row_map(R);
  h.M = R.M;
  h.rows = (int64_t)Tc * R.M;
  h.tokens = a.tokens;
  h.C = a.C;
  h.t0 = t0;
  h.B = R.B;
  h.pmax = pmax;
  h.psum = psum;
  h.ptgt = ptgt;
  h.zc_out = a.zc ? (const float*)a.zc + a.zmap.out : nullptr;
  h.zc_stride = a.zmap.pg;
  const dim3 grid((unsigned)a.ws.nvt, (unsigned)(h.rows / BM));
  const bool split = a.split;
  ProfScope ps(kKHead, st);
  if (a.cfg.probe == ZO_RADEMACHER) {
    if (split) head_f32_kernel<ZO_RADEMACHER, true><<<grid, 256, 0, st>>>(h);
    else head_f32_kernel<ZO_RADEMACHER, false><<<grid, 256, 0, st>>>(h);
  } else if (a.zc) {
    if (split) head_f32_kernel<kGaussCached, true><<<grid, 256, 0, st>>>(h);
    else head_f32_kernel<kGaussCached, false><<<grid, 256, 0, st>>>(h);
  } else {
    if (split) head_f32_kernel<ZO_GAUSSIAN, true><<<grid, 256, 0, st>>>(h);
    else head_f32_kernel<ZO_GAUSSIAN, false><<<grid, 256, 0, st>>>(h);
  }
  return hipGetLastError();
}

}  // namespace

// The step driver: per timestep the perturbed embedding and one gate launch
// per layer; per time chunk one head launch and one combine; then the
// per-pass reduction. The fp32 and bf16 paths differ only in their embed,
// gate and head kernels.
hipError_t launch_forward(const ForwardArgs& a, hipStream_t st) {
  const zo_config& c = a.cfg;
  const bool bf16 = c.wdtype == ZO_WBF16;
  const int L = c.n_layers, H = c.hidden, V = c.vocab;
  const Rows& R = a.rows;
  const WsPlan& W = a.ws;
  const int64_t M = R.M;
  const size_t el = bf16 ? 2 : 4;  // activation element size
  const size_t state = (size_t)M * H * el;
  const RowMap rm = row_map(R);
  char* ws = a.work;
  char* x0 = ws + W.x0;
  char* hbuf = ws + W.hbuf;
  char* hist = ws + W.hist;
  float* cbuf = (float*)(ws + W.cbuf);
  float* zb = (float*)(ws + W.zb);
  float* zbo = (float*)(ws + W.zbo);
  float* pmax = (float*)(ws + W.pmax);
  float* psum = (float*)(ws + W.psum);
  float* ptgt = (float*)(ws + W.ptgt);
  double* row_loss = (double*)(ws + W.row_loss);
  auto head = bf16 ? launch_head_bf16 : launch_head_f32;
  hipError_t e;
#define ZO_TRY(x)                          \
  do {                                     \
    if ((e = (x)) != hipSuccess) return e; \
  } while (0)

  const int T = W.T;
  std::optional<PhaseRange> phase;
  phase.emplace("forward: prepare");
  // every pass starts from h = c = 0: zero what is read before it is written
  // (the state slots that timestep 0 reads, the cell states) and the row sums
  for (int l = 0; l + 1 < L; ++l) ZO_TRY(zero_async(hbuf + (size_t)(2 * l + 1) * state, state, st));
  ZO_TRY(zero_async(hist + (size_t)(T - 1) * state, state, st));
  ZO_TRY(zero_async(cbuf, (size_t)L * M * H * 4, st));
  ZO_TRY(zero_async(row_loss, (size_t)M * 8, st));

  // bf16 weights: the fp16 copy of the product matrices; probe cache (normal
  // probes, when the workspace holds it)
  if (bf16) ZO_TRY(launch_w16_fill(a, st));
  if (a.zc) ZO_TRY(launch_zcache_fill(a, st));
  if (a.bits) ZO_TRY(launch_bits_fill(a.bits, a.lay.total, a.seed, a.i0, R.N, st));

  // bias probes
  {
    BiasOffsets boff{};
    for (int l = 0; l < L; ++l) boff.layer[l] = a.lay.bias[l];
    const int64_t total = (int64_t)R.N * 4 * H * L + (int64_t)R.N * V;
    int64_t grid = (total + 255) / 256;
    if (grid > 65536) grid = 65536;
    prep_bias_kernel<<<dim3((unsigned)grid), dim3(256), 0, st>>>(c.probe, make_key(a.seed), a.i0,
                                                                a.eps, R.N, L, 4 * H, V, boff,
                                                                a.lay.b_out, zb, zbo);
    ZO_TRY(hipGetLastError());
  }

  // states of layer l at time t: lower layers alternate between two slots
  // (time t in slot t & 1), the top layer writes the time-chunk ring
  auto state_in = [&](int l, int t) -> char* {  // h of layer l at time t - 1
    if (l < L - 1) return hbuf + (size_t)l * 2 * state + (size_t)((t + 1) & 1) * state;
    return hist + (size_t)((t + T - 1) % T) * state;
  };
  auto state_out = [&](int l, int t) -> char* {  // h of layer l at time t
    if (l < L - 1) return hbuf + (size_t)l * 2 * state + (size_t)(t & 1) * state;
    return hist + (size_t)(t % T) * state;
  };
  // Launch order. bf16: per timestep the embedding and one gate launch per
  // layer. fp32: a wavefront, launch d running layer l at time d - l for every
  // layer with 0 <= d - l < C, in one launch (layer l reads layer l - 1's state
  // of time d - l, written by launch d - 1, while layer l - 1 writes its other
  // slot); the embeddings of a whole time chunk [d, d + T) are written in one
  // launch before launch d, after launch d - 1 read the last of the previous
  // chunk's.
  const int ndiag = bf16 ? a.C : a.C + L - 1;
  const size_t x0_step = (size_t)M * c.embed * el;  // one timestep of embeddings
  phase.reset();
  for (int d = 0; d < ndiag; ++d) {
    PhaseRange step_range("forward: layer steps of one timestep");
    if (bf16) ZO_TRY(launch_embed_bf16(a, d, x0, st));
    else if (d < a.C && d % T == 0) ZO_TRY(launch_embed_f32(a, d, std::min(T, a.C - d), x0, st));
    if (bf16) {
      for (int l = 0; l < L; ++l) {
        const char* xin = l == 0 ? x0 : state_out(l - 1, d);
        ZO_TRY(launch_gate_bf16(a, l, xin, state_in(l, d), state_out(l, d), cbuf + (size_t)l * M * H,
                                zb + (size_t)l * R.N * 4 * H, st));
      }
    } else {
      GateLayer ls[kLaunchLayers];
      int n = 0;
      for (int l = 0; l < L; ++l) {
        const int t = d - l;
        if (t < 0 || t >= a.C) continue;
        GateLayer& g = ls[n++];
        g.x = (const float*)(l == 0 ? x0 + (size_t)(t % T) * x0_step : state_out(l - 1, t));
        g.hprev = (const float*)state_in(l, t);
        g.hout = (float*)state_out(l, t);
        g.cst = cbuf + (size_t)l * M * H;
        g.off_ih = a.lay.w_ih[l];
        g.off_hh = a.lay.w_hh[l];
        g.off_b = a.lay.bias[l];
        g.El = l == 0 ? c.embed : c.hidden;
        g.zb = zb + (size_t)l * R.N * 4 * H;
        g.zc_ih = a.zc ? (const float*)a.zc + a.zmap.ih[l] : nullptr;
        g.zc_hh = a.zc ? (const float*)a.zc + a.zmap.hh[l] : nullptr;
        if (n == kLaunchLayers) {
          ZO_TRY(launch_gates_f32(a, ls, n, st));
          n = 0;
        }
      }
      if (n) ZO_TRY(launch_gates_f32(a, ls, n, st));
    }
    // the top layer has finished time t: the head runs over each completed time chunk
    const int t = bf16 ? d : d - (L - 1);
    if (t >= 0 && (t % T == T - 1 || t == a.C - 1)) {
      const int t0 = t - t % T;
      const int Tc = t - t0 + 1;
      PhaseRange head_range("forward: head and cross entropy of a time chunk");
      ZO_TRY(head(a, hist, t0, Tc, zbo, pmax, psum, ptgt, st));
      ProfScope ps(kKCombine, st);
      const int64_t rows = (int64_t)Tc * M;
      combine_kernel<<<dim3((unsigned)((rows + 255) / 256)), 256, 0, st>>>(
          pmax, psum, ptgt, W.nvt, rows, M, t0, a.C, R.B, rm, a.mask, a.tokens, a.cfg.vocab);
      ZO_TRY(hipGetLastError());
      accumulate_kernel<<<dim3((unsigned)((M + 255) / 256)), 256, 0, st>>>(ptgt, M, Tc, row_loss);
      ZO_TRY(hipGetLastError());
    }
  }
  PhaseRange reduce_range("forward: loss reduction");
  reduce_kernel<<<1, 256, 0, st>>>(row_loss, R.N, R.B, a.C, rm, a.mask, a.Lplus, a.Lminus);
  ZO_TRY(hipGetLastError());
#undef ZO_TRY
  return hipSuccess;
}

}  // namespace zo
