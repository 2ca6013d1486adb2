// Kernels of the batched perturbed forward for bf16 weights (fp16 MFMA
// operands, fp32 accumulation and fp32 cell state).
//
// A bf16 weight cannot carry a perturbation of eps = 1e-3: its spacing near
// |w| = 1/64 is 1.2e-4, so a rounded w + eps z would lose about 6% of eps z
// per element. fp16 can: its spacing there is 1.5e-5, so fp16(w + eps z) keeps
// eps z to within 0.8% per element, and over a K-long product the rounding
// errors average to a few tenths of a percent of the probe term. So the call
// first writes an fp16 copy of every weight matrix (exact: bf16 values lie on
// the fp16 grid in [2^-14, 65504)), activations are stored in fp16, and every
// product is ONE v_mfma_f32_32x32x16_f16 stream
//     acc += A . fp16(W + s eps z)
// whose B fragment each wave forms in registers from the fp16 weight fragment
// and the probe fragment with one packed fp16 add per pair (+-fp16(eps) for
// sign probes, expanded from bits; fp16(eps z), sign-flipped for -eps rows,
// for normal probes). theta +- eps z is never formed in memory.
//
// Tiles: a workgroup of 8 waves computes TM = 256 rows x TN = 256 columns
// (waves 2 x 4, wave tiles 128 x 64 = 4 x 2 tiles of 32x32 MFMA output); two
// waves share each SIMD, so one wave's LDS reads, probe expansion and address
// work run under the other's matrix instructions. Lane l feeds row/column
// l % 32 and k block l / 32.
//
// LDS (static, one barrier per K tile): per stage the activation tile
// [TM][TK] and the weight tile [TN][TK] (fp16 rows of 2 TK bytes whose
// 16-byte chunks are XOR-swizzled by row), copied from global memory straight
// into LDS without passing through registers, and the probe tile. Sign
// probes: K tiles of 64 in two stages, the probe tile as sign bits [TN][2]
// words expanded to fp16 +-eps by each wave. Normal probes: the probe tile is
// fp16(eps z) [TN][TK], copied from the probe cache like the weights or
// generated in registers, which takes a third of the stage; K tiles of 32 in
// three stages (3 x 48 KB) keep the 256 x 256 tile and so copy 48 KB per 16.8
// MFLOP of matrix work instead of 64 KB with 256 x 128 tiles of 64. K tile
// it + STAGES - 1 (copies and probe tile) is issued during the MFMAs of tile it.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "zo_kernels.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));

constexpr int TM = 256;         // rows per workgroup
constexpr int NWAVES = 8;
constexpr int NT = 64 * NWAVES;  // threads per workgroup
// Global->LDS copies: each copy instruction moves 1 KB (64 lanes x 16 B).
// kCopyWaves of the 8 waves issue them, spread over the first kCopySteps k
// steps of the previous K tile.
constexpr int kCopyWaves = 4;
constexpr int kCopySteps = 2;

// Sign probes: K per tile and LDS stages.
constexpr int kSignTK = 64;
constexpr int kSignStages = 2;

// Per probe kind: K tile, stages, LDS layout, copy split, probe roles.
template <int kind>
struct Tiles {
  static constexpr bool kSigns = kind == ZO_RADEMACHER;
  static constexpr int TK = kSigns ? kSignTK : 32;           // K per tile
  static constexpr int STAGES = kSigns ? kSignStages : 3;    // LDS stages
  static constexpr int SW = TK / 32;                         // sign words per row and tile
  static constexpr int RowBytes = TK * 2;           // one LDS row: TK fp16
  static constexpr int CPR = RowBytes / 16;         // 16-byte chunks per row
  static constexpr int RPB = 256 / RowBytes;        // rows per 256 bytes (every LDS bank once)
  static constexpr int RPC = 1024 / RowBytes;       // rows per 1 KB copy
  static constexpr int ABytes = TM * RowBytes;
  static constexpr int TN = kVocabTileWide;
  static constexpr int WAVES_N = TN / 64;  // wave tiles are 64 columns wide
  static constexpr int WAVES_M = NWAVES / WAVES_N;
  static constexpr int WROWS = TM / WAVES_M;  // rows per wave tile
  static constexpr int MT = WROWS / 32;
  static constexpr int WBytes = TN * RowBytes;
  static constexpr int ZBytes = kSigns ? TN * 4 * SW : TN * RowBytes;
  static constexpr int StageBytes = ABytes + WBytes + (kSigns ? 0 : ZBytes);  // sign bits: own arrays
  static constexpr int ACopies = ABytes / 1024 / kCopyWaves;  // activation copies per copying wave
  static constexpr int WCopies = WBytes / 1024 / kCopyWaves;  // weight copies per copying wave
  // cached normal probes: the probe tile is copied like the weight tile
  static constexpr int ZCopies = kind == kGaussCached ? WCopies : 0;
  static constexpr int Copies = ACopies + WCopies + ZCopies;
  static constexpr int ZROW_T = NT / TN;     // threads per probe-tile row (normal probes)
  static constexpr int ZVALS = TK / ZROW_T;  // probe values per thread and K tile (normal probes)
  // 16-byte slot of chunk c in LDS row r: c ^ swz(r). Any RPB consecutive rows
  // cover the 64 banks once per chunk, and swz gives the CPR groups of RPB rows
  // among 16 consecutive rows distinct chunks, so the 16 rows of one 128-bit
  // fragment read (same chunk) hit every bank exactly once.
  __device__ static __forceinline__ int swz(int r) { return (r / RPB) & (CPR - 1); }
  static_assert(RPB * CPR == 16, "swizzle period of 16 rows");
  static_assert(WAVES_M * WAVES_N == NWAVES && WROWS % 32 == 0, "wave grid");
  static_assert(WCopies * kCopyWaves * 1024 == WBytes && ACopies * kCopyWaves * 1024 == ABytes,
                "copy split");
  static_assert(Copies < 64, "outstanding copies fit the vmcnt counter");
  static_assert(!kSigns || TN * SW <= NT, "at most one sign word per thread");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert(kSigns || (ZVALS % 8 == 0 && ZROW_T * TN == NT), "probe roles");
  static_assert(kRowGranuleBF16 % WROWS == 0, "a wave tile lies inside one sign's rows");
  static_assert(TK % 16 == 0 && (TK / 16 == 4 || TK / 16 == 2), "k steps per tile");
};
static_assert(2 * kRowGranuleBF16 % TM == 0, "a probe's rows must be a whole number of row tiles");
static_assert(Tiles<kGaussCached>::StageBytes == Tiles<ZO_GAUSSIAN>::StageBytes, "normal-probe stages");

// LDS stages per probe kind (static, so that every offset is a constant).
__shared__ __align__(16) uint8_t lds_r0[Tiles<ZO_RADEMACHER>::StageBytes];
__shared__ __align__(16) uint8_t lds_r1[Tiles<ZO_RADEMACHER>::StageBytes];
__shared__ __align__(16) uint8_t lds_r2[Tiles<ZO_RADEMACHER>::StageBytes];
__shared__ __align__(16) uint8_t lds_r3[Tiles<ZO_RADEMACHER>::StageBytes];
__shared__ __align__(16) uint32_t lds_b0[Tiles<ZO_RADEMACHER>::ZBytes / 4];
__shared__ __align__(16) uint32_t lds_b1[Tiles<ZO_RADEMACHER>::ZBytes / 4];
__shared__ __align__(16) uint32_t lds_b2[Tiles<ZO_RADEMACHER>::ZBytes / 4];
__shared__ __align__(16) uint32_t lds_b3[Tiles<ZO_RADEMACHER>::ZBytes / 4];
__shared__ __align__(16) uint8_t lds_g0[Tiles<ZO_GAUSSIAN>::StageBytes];
__shared__ __align__(16) uint8_t lds_g1[Tiles<ZO_GAUSSIAN>::StageBytes];
__shared__ __align__(16) uint8_t lds_g2[Tiles<ZO_GAUSSIAN>::StageBytes];
static_assert(Tiles<ZO_RADEMACHER>::STAGES * (sizeof(lds_r0) + sizeof(lds_b0)) <= 160 * 1024, "LDS");
static_assert(Tiles<ZO_GAUSSIAN>::STAGES * sizeof(lds_g0) <= 160 * 1024, "LDS");

template <int kind, int S>
__device__ __forceinline__ uint8_t* stage() {
  static_assert(S >= 0 && S < Tiles<kind>::STAGES, "stage index");
  if constexpr (kind == ZO_RADEMACHER)
    return S == 0 ? lds_r0 : S == 1 ? lds_r1 : S == 2 ? lds_r2 : lds_r3;
  else
    return S == 0 ? lds_g0 : S == 1 ? lds_g1 : lds_g2;
}
template <int S>
__device__ __forceinline__ uint32_t* sign_bits() {
  static_assert(S >= 0 && S < Tiles<ZO_RADEMACHER>::STAGES, "stage index");
  return S == 0 ? lds_b0 : S == 1 ? lds_b1 : S == 2 ? lds_b2 : lds_b3;
}

__device__ __forceinline__ h8 as_h8(u4 v) { return __builtin_bit_cast(h8, v); }

// Probe sign bits in LDS are kept in "unshuffled" order: the word of 32
// consecutive k holds the negative-sign flags (1 = -1) of the even elements
// 0, 2, .., 30 in bits 0..15 and of the odd elements 1, 3, .., 31 in bits
// 16..31. The two elements of one packed fp16 pair then sit 16 bits apart,
// so one shift, one mask and one xor turn them into the pair (+-e, +-e): the
// flag of the even element lands on bit 15 and that of the odd one on bit
// 31, and flip the sign bits of the constant pair (e, e).
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

// 16 bytes per lane from global memory straight into LDS: the wave's 64
// lanes fill the 1 KB at lds (wave-uniform), lane L at lds + 16 L. Written as
// an asm statement, so the compiler inserts no waits of its own for these
// copies; the K-tile loop waits for them explicitly (vmcnt) before each barrier.
__device__ __forceinline__ void copy_to_lds(const void* src, uint8_t* lds) {
  const uint32_t m0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) uint8_t*)lds;
  asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(src), "{m0}"(m0) : "memory");
}

// Wait until at most VM of this thread's global->LDS copies are outstanding
// and its LDS accesses are complete (s_waitcnt vmcnt(VM) lgkmcnt(0); the gfx9
// encoding splits vmcnt into bits 3:0 and 15:14, expcnt 7 = no wait), then a
// workgroup barrier without a memory fence. The empty asm statements keep the
// compiler from moving memory accesses across either.
template <int VM>
__device__ __forceinline__ void wait_and_barrier() {
  static_assert(VM >= 0 && VM < 64, "vmcnt");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | 0x70);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

struct SegB {
  const uint16_t* A;  // first row of this workgroup's activation tile; row r at A + r * lda
  int64_t lda;
  const uint16_t* W;  // weight row n at W + n * ldw (the fp16 copy of the matrix)
  int64_t ldw;
  uint64_t zoff;      // offset of the matrix inside theta (probe coordinates)
  int K;
  const uint16_t* Z;  // kGaussCached: fp16(eps z) of this probe and matrix, laid out like W
};

// acc: [MT row tiles][2 column tiles] of 32x32 fp32 for this wave.
// colmap(rho, &n) maps LDS column rho (0..TN-1) to a weight row n inside the
// matrix (columns beyond the matrix map to a valid row; they are never
// scored). sgn: the sign of eps for this wave's rows (+1, -1, or 0 for the
// clean pass of forward differences, kFD only); eps_b: fp16 bits of eps.
// kTrans: accumulate the transposed product (weight columns on the rows of
// each 32x32 tile, activation rows on its columns): both operands of
// v_mfma_f32_32x32x16_f16 have the same fragment layout, so only their order
// changes. Lane (lr, lg) then holds, for activation row lr of a tile, the 16
// columns 8 (v >> 2) + 4 lg + (v & 3), v < 16.
// kSplit: the two-stream form for small eps, acc += A.W then acc += A.(s eps z)
// (the probe fragment as an operand of its own, twice the matrix work),
// instead of acc += A.fp16(W + s eps z): a weight fragment rounded with the
// probe added loses up to half an fp16 ulp of w per element, which is a
// large share of eps z once eps is small against |w|.
template <int kind, bool kTrans = false, bool kFD = false, bool kSplit = false, typename ColMap>
__device__ __forceinline__ void mainloop_bf16(f16v (&acc)[Tiles<kind>::MT][2], const SegB s0, const SegB s1,
                                              int nseg, ColMap colmap, Key key, uint32_t probe, int sgn,
                                              float eps, uint16_t eps_b) {
  using T = Tiles<kind>;
  constexpr int MT = T::MT;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  constexpr int TK = T::TK;
  const int ntiles = s0.K / TK + (nseg > 1 ? s1.K / TK : 0);

  // copy roles: copy q of copying wave w fills rows RPC (q kCopyWaves + w) .. +RPC-1
  // of the activation (q < ACopies) or weight tile, 1 KB lane-linear in LDS:
  // lane L writes row + L / CPR, slot L % CPR, which holds chunk (L % CPR) ^ swz(row)
  const int crow = lane / T::CPR;
  int arow[T::ACopies], wrow[T::WCopies];
  uint32_t aoff[T::ACopies], woff[T::WCopies];  // element offsets of the chunk inside the row
#pragma unroll
  for (int q = 0; q < T::ACopies; ++q) {
    const int r = T::RPC * (q * kCopyWaves + wave % kCopyWaves) + crow;
    arow[q] = r;
    aoff[q] = 8u * (uint32_t)((lane % T::CPR) ^ T::swz(r));
  }
#pragma unroll
  for (int q = 0; q < T::WCopies; ++q) {
    const int r = T::RPC * (q * kCopyWaves + wave % kCopyWaves) + crow;
    colmap(r, wrow[q]);
    woff[q] = 8u * (uint32_t)((lane % T::CPR) ^ T::swz(r));
  }
  // probe roles: signs, threads t < TN SW: row t / SW, one 32-k word at 32 (t % SW);
  //              normal, every thread: row t / ZROW_T, ZVALS k at ZVALS (t % ZROW_T)
  const int zr = kind == ZO_RADEMACHER ? t / T::SW : t / T::ZROW_T;
  const int zpart = kind == ZO_RADEMACHER ? (t % T::SW) : (t % T::ZROW_T);
  int zn;
  colmap(zr, zn);

  Words zcache{{0u, 0u, 0u, 0u}};
  int seg = 0, k0 = 0;

  // Issue the next K tile into stage S, in four parts spread over the
  // current tile's k steps (so that no wave stalls on a burst of copies):
  // parts 0 and 1 the global->LDS copies of the activation and weight rows,
  // half each; part 2 the probe tile, computed in registers and written to
  // LDS; part 3 advances to the following tile.
  auto issue = [&](auto stage_tag, auto part_tag) {
    constexpr int S = decltype(stage_tag)::value;
    constexpr int P = decltype(part_tag)::value;
    uint8_t* base = stage<kind, S>();
    const SegB sg = seg == 0 ? s0 : s1;
    if (wave < kCopyWaves) {
#pragma unroll
      for (int c = P * T::Copies / kCopySteps; c < (P < kCopySteps ? (P + 1) * T::Copies / kCopySteps : 0); ++c) {
        if (c < T::ACopies) {
          copy_to_lds(sg.A + (int64_t)arow[c] * sg.lda + k0 + aoff[c], base + (c * kCopyWaves + wave) * 1024);
        } else if (c < T::ACopies + T::WCopies) {
          const int q = c - T::ACopies;
          copy_to_lds(sg.W + (int64_t)wrow[q] * sg.ldw + k0 + woff[q],
                      base + T::ABytes + (q * kCopyWaves + wave) * 1024);
        } else {  // cached probe rows: the same rows and chunk order as the weight copy q
          const int q = c - T::ACopies - T::WCopies;
          copy_to_lds(sg.Z + (int64_t)wrow[q] * sg.ldw + k0 + woff[q],
                      base + T::ABytes + T::WBytes + (q * kCopyWaves + wave) * 1024);
        }
      }
    }
    if constexpr (P == 2 && kind == ZO_RADEMACHER) {
      if (T::TN * T::SW == NT || t < T::TN * T::SW) {
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
      // negative-sign flags in unshuffled order
      sign_bits<S>()[zr * T::SW + zpart] = unshuffle_bits(~word);
      }
    } else if constexpr (P == 2 && kind == ZO_GAUSSIAN) {
      const uint64_t j0 = sg.zoff + (uint64_t)zn * (uint64_t)sg.ldw + (uint64_t)k0 + T::ZVALS * zpart;
      uint8_t* zrow = base + T::ABytes + T::WBytes + zr * T::RowBytes;
#pragma unroll
      for (int q = 0; q < T::ZVALS / 8; ++q) {
        float za[4], zb[4];
        gauss_block(key, probe, (j0 >> 2) + 2 * q, za);
        gauss_block(key, probe, (j0 >> 2) + 2 * q + 1, zb);
        const int chunk = (T::ZVALS / 8) * zpart + q;
        *(u4*)(zrow + 16 * (chunk ^ T::swz(zr))) =
            u4{pack_f16x2(eps * za[0], eps * za[1]), pack_f16x2(eps * za[2], eps * za[3]),
               pack_f16x2(eps * zb[0], eps * zb[1]), pack_f16x2(eps * zb[2], eps * zb[3])};
      }
    }
    if constexpr (P == 3) {
      k0 += TK;
      if (k0 == sg.K) {
        k0 = 0;
        ++seg;
      }
    }
  };
  auto issue_all = [&](auto stage_tag) {
    issue(stage_tag, std::integral_constant<int, 0>{});
    issue(stage_tag, std::integral_constant<int, 1>{});
    issue(stage_tag, std::integral_constant<int, 2>{});
    issue(stage_tag, std::integral_constant<int, 3>{});
  };

  // Fragments of one 16-k step: activations (MT row tiles), weights and
  // probe values (2 column tiles). The next step's LDS reads and sign
  // expansion are issued between the current step's MFMAs (software
  // pipelining within the K tile). Lane (lr, lg) reads chunk 2 s + lg of its
  // rows, in slot (2 s) ^ y with y = lg ^ swz(lr) (every row offset below is
  // a multiple of 16, the swizzle period).
  const uint32_t y = (uint32_t)(lg ^ T::swz(lr));
  const uint32_t a_lane = (uint32_t)(T::WROWS * wm + lr) * T::RowBytes;
  const uint32_t w_lane = (uint32_t)(64 * wn + lr) * T::RowBytes;
  // the pair (s eps, s eps) in fp16 (signs), or the sign flip of -eps rows (normal)
  const uint32_t ebits = (uint32_t)eps_b | ((uint32_t)eps_b << 16);
  const bool neg = sgn < 0;
  const uint32_t zc = kind == ZO_RADEMACHER ? (neg ? ebits ^ 0x80008000u : ebits) : (neg ? 0x80008000u : 0u);
  // forward differences: the clean pass multiplies its probe fragments by 0
  const uint32_t zmask = sgn == 0 ? 0u : 0xFFFFFFFFu;
  struct Frag {
    h8 a[MT], w[2], z[2];
  };
  auto compute = [&](auto stage_tag, bool more) {
    constexpr int S = decltype(stage_tag)::value;
    const uint8_t* base = stage<kind, S>();
    const uint8_t* pa = base + a_lane;
    const uint8_t* pw = base + T::ABytes + w_lane;
    // per lane, the flags of its k block pre-shifted so that a constant shift
    // per (k step, pair) brings them to bits 15 / 31 (see unshuffle_bits)
    uint32_t bits[2][2];
    if constexpr (kind == ZO_RADEMACHER) {
      const uint32_t pre = 4u * (uint32_t)(1 - lg);
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        if constexpr (T::SW == 2) {
          const uint2 v = *(const uint2*)(sign_bits<S>() + (64 * wn + 32 * nt + lr) * 2);
          bits[nt][0] = v.x << pre;
          bits[nt][1] = v.y << pre;
        } else {
          bits[nt][0] = sign_bits<S>()[64 * wn + 32 * nt + lr] << pre;
          bits[nt][1] = 0u;
        }
      }
    }
    auto load = [&](int s, Frag& f) {
      const uint32_t so = 16u * ((uint32_t)(2 * s) ^ y);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) f.a[mt] = as_h8(*(const u4*)(pa + 32 * mt * T::RowBytes + so));
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        f.w[nt] = as_h8(*(const u4*)(pw + 32 * nt * T::RowBytes + so));
        u4 v;
        if constexpr (kind == ZO_RADEMACHER) {
          const uint32_t x = bits[nt][s >> 1];
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            v[d] = ((x << (11 - 8 * (s & 1) - d)) & 0x80008000u) ^ zc;
            if constexpr (kFD) v[d] &= zmask;
          }
        } else {
          v = *(const u4*)(pw + T::WBytes + 32 * nt * T::RowBytes + so);
#pragma unroll
          for (int d = 0; d < 4; ++d) {
            v[d] ^= zc;
            if constexpr (kFD) v[d] &= zmask;
          }
        }
        f.z[nt] = as_h8(v);
      }
    };
    Frag f[2];
    load(0, f[0]);
#pragma unroll
    for (int s = 0; s < TK / 16; ++s) {
      const Frag& c = f[s & 1];
      if (s + 1 < TK / 16) load(s + 1, f[(s + 1) & 1]);
      auto mma = [&](const h8(&b)[2]) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int nt = 0; nt < 2; ++nt)
            acc[mt][nt] = kTrans ? __builtin_amdgcn_mfma_f32_32x32x16_f16(b[nt], c.a[mt], acc[mt][nt], 0, 0, 0)
                                 : __builtin_amdgcn_mfma_f32_32x32x16_f16(c.a[mt], b[nt], acc[mt][nt], 0, 0, 0);
      };
      if constexpr (kSplit) {
        // A.W for every accumulator, then A.(s eps z): the two products into
        // one accumulator are MT x 2 instructions apart
        mma(c.w);
        mma(c.z);
      } else {
        // B = fp16(W + s eps z): one packed fp16 add per pair (round to
        // nearest even), then one MFMA per accumulator
        h8 wz[2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) wz[nt] = c.w[nt] + c.z[nt];
        mma(wz);
      }
      if (more) {
        // tile it + STAGES - 1 goes to the stage tile it - 1 used
        constexpr std::integral_constant<int, (S + T::STAGES - 1) % T::STAGES> next{};
        if constexpr (TK / 16 == 4) {
          if (s == 0) issue(next, std::integral_constant<int, 0>{});
          if (s == 1) issue(next, std::integral_constant<int, 1>{});
          if (s == 2) issue(next, std::integral_constant<int, 2>{});
          if (s == 3) issue(next, std::integral_constant<int, 3>{});
        } else {
          if (s == 0) {
            issue(next, std::integral_constant<int, 0>{});
            issue(next, std::integral_constant<int, 1>{});
          }
          if (s == 1) {
            issue(next, std::integral_constant<int, 2>{});
            issue(next, std::integral_constant<int, 3>{});
          }
        }
      }
      if (s + 1 < TK / 16) {
        // per step: the next step's LDS reads first, then each MFMA followed by
        // a few VALU instructions of the next step's probe fragments
        __builtin_amdgcn_sched_group_barrier(0x100, MT + 2 + (kind == ZO_RADEMACHER ? 0 : 2), 0);
#pragma unroll
        for (int i = 0; i < (kSplit ? 4 : 2) * MT; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);
        }
      }
    }
  };

  // K tile it lives in stage it % STAGES. Per tile: wait for this thread's
  // copies of tile it (with three stages those of tile it + 1, issued later,
  // may stay in flight) and its LDS writes; barrier (tile it complete for
  // every wave, and the stage computed at it - 1 free); compute it while
  // issuing tile it + STAGES - 1 into that stage.
  auto step = [&](auto stage_tag, int it) {
    // the copies of tiles it + 1 .. it + STAGES - 2 (those issued) may stay in flight
    if constexpr (T::STAGES == 4) {
      if (it + 2 < ntiles) wait_and_barrier<2 * T::Copies>();
      else if (it + 1 < ntiles) wait_and_barrier<T::Copies>();
      else wait_and_barrier<0>();
    } else if constexpr (T::STAGES == 3) {
      if (it + 1 < ntiles) wait_and_barrier<T::Copies>();
      else wait_and_barrier<0>();
    } else {
      wait_and_barrier<0>();
    }
    compute(stage_tag, it + T::STAGES - 1 < ntiles);
  };
  issue_all(std::integral_constant<int, 0>{});
  if constexpr (T::STAGES >= 3) {
    if (ntiles > 1) issue_all(std::integral_constant<int, 1>{});
  }
  if constexpr (T::STAGES >= 4) {
    if (ntiles > 2) issue_all(std::integral_constant<int, 2>{});
  }
  for (int it = 0; it < ntiles; it += T::STAGES) {
    step(std::integral_constant<int, 0>{}, it);
    if (it + 1 < ntiles) step(std::integral_constant<int, 1>{}, it + 1);
    if constexpr (T::STAGES >= 3) {
      if (it + 2 < ntiles) step(std::integral_constant<int, 2 % T::STAGES>{}, it + 2);
    }
    if constexpr (T::STAGES >= 4) {
      if (it + 3 < ntiles) step(std::integral_constant<int, 3 % T::STAGES>{}, it + 3);
    }
  }
  __syncthreads();  // every wave done with the stages before they are reused
}

// Tile (row block m, column block n) of workgroup L of a 1-D grid of nm x nn
// tiles. Workgroups are dispatched to the 8 XCDs in turn (L % 8), each XCD
// with its own L2: XCD x takes the row blocks [x nm/8, (x+1) nm/8) and sweeps
// the column blocks in groups of R row blocks, so that the 32 workgroups an
// XCD runs at a time share R activation and 32 / R weight tiles, and all
// XCDs read the same weight columns at the same time. Shapes with nm not a
// multiple of 8 take the plain row-major order. Any order is correct.
__device__ __forceinline__ void tile_of(int L, int nm, int nn, int& m, int& n) {
  if (nm % 8 != 0) {
    m = L / nn;
    n = L - m * nn;
    return;
  }
  const int x = L & 7, j = L >> 3, per = nm >> 3;
  const int R = per % 4 == 0 ? 4 : per % 2 == 0 ? 2 : 1;
  const int g = j / (R * nn), rem = j - g * (R * nn);
  n = rem / R;
  m = x * per + g * R + (rem - n * R);
}

__device__ __forceinline__ float sigm(float x) { return 1.0f / (1.0f + __expf(-x)); }
__device__ __forceinline__ float tanh_(float x) { return 1.0f - 2.0f / (__expf(2.0f * x) + 1.0f); }

// Row (within the workgroup's TM) of accumulator element v of row tile mt
// for this lane: 32x32 MFMA output layout.
template <int kind>
__device__ __forceinline__ int acc_row(int wm, int mt, int lg, int v) {
  return Tiles<kind>::WROWS * wm + 32 * mt + 8 * (v >> 2) + 4 * lg + (v & 3);
}

template <int MT>
__device__ __forceinline__ void zero_acc(f16v (&acc)[MT][2]) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) acc[mt][nt] = f16v{};
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
  uint16_t eps_b;
  RowMap rm;
  int n_row_blocks;  // M / TM
  const uint16_t* zc_ih;  // probe cache: W_ih's and W_hh's values of probe 0; probe n at + n * zc_stride
  const uint16_t* zc_hh;
  uint64_t zc_stride;
  const uint16_t* w_ih16;  // fp16 copies of W_ih and W_hh
  const uint16_t* w_hh16;
};

// Workgroup: TM rows x TN / 4 hidden units. Wave column c (0..63) of wave wn
// is gate c / 16 of unit 16 wn + c % 16, so lane lr holds gates i, g (lr < 16)
// or f, o (lr >= 16) of unit lr % 16 in its two column tiles, and one
// exchange with lane lr ^ 16 brings all four gates of a (row, unit) together.
template <int kind, bool kFD, bool kSplit>
__global__ __launch_bounds__(NT, 1) void gate_bf16_kernel(GateArgsB g) {
  using T = Tiles<kind>;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  int mb, nb;
  tile_of(blockIdx.x, g.n_row_blocks, g.H / (T::TN / 4), mb, nb);
  const int u0 = nb * (T::TN / 4);
  const int64_t m0 = (int64_t)mb * TM;
  const int pair = pass_of(g.rm, m0).probe;
  const int sgn = pass_of(g.rm, m0 + T::WROWS * wm).sign;  // a wave tile lies inside one pass
  const int H = g.H;
  auto colmap = [&](int rho, int& n) {
    const int c = rho & 63;
    n = (c >> 4) * H + u0 + 16 * (rho >> 6) + (c & 15);
  };
  f16v acc[T::MT][2];
  zero_acc(acc);
  const uint64_t zpos = (uint64_t)pair * g.zc_stride;
  const SegB s0{g.x + m0 * g.El, g.El, g.w_ih16, g.El, g.off_ih, g.El,
                kind == kGaussCached ? g.zc_ih + zpos : nullptr};
  const SegB s1{g.hprev + m0 * H, H, g.w_hh16, H, g.off_hh, H,
                kind == kGaussCached ? g.zc_hh + zpos : nullptr};
  mainloop_bf16<kind, false, kFD, kSplit>(acc, s0, s1, 2, colmap, g.key, g.i0 + (uint32_t)pair, sgn, g.eps,
                                          g.eps_b);

  const int hi = lr >> 4;  // 0: gates i, g; 1: gates f, o
  const int u = u0 + 16 * wn + (lr & 15);
  float bias[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
    const int gate = 2 * nt + hi;
    const float b = bf16_to_f32(g.theta[g.off_b + (uint64_t)(gate * H + u)]);
    const float z = g.zb[(int64_t)pair * 4 * H + gate * H + u];
    bias[nt] = b + (float)sgn * z;
  }
#pragma unroll
  for (int mt = 0; mt < T::MT; ++mt) {
#pragma unroll
    for (int v = 0; v < 16; v += 2) {
      // lanes lr < 16 update row element v, lanes lr >= 16 element v + 1
      float mine[2], send[2], got[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const float p0 = acc[mt][nt][v] + bias[nt], p1 = acc[mt][nt][v + 1] + bias[nt];
        mine[nt] = hi ? p1 : p0;
        send[nt] = hi ? p0 : p1;
        got[nt] = __shfl_xor(send[nt], 16, 64);
      }
      const float ip = hi ? got[0] : mine[0], fp = hi ? mine[0] : got[0];
      const float gp = hi ? got[1] : mine[1], op = hi ? mine[1] : got[1];
      const int lrow = acc_row<kind>(wm, mt, lg, v + hi);
      const int64_t o = (m0 + lrow) * H + u;
      const float c = sigm(fp) * g.cst[o] + sigm(ip) * tanh_(gp);
      g.cst[o] = c;
      g.hout[o] = f16_bits(sigm(op) * tanh_(c));
    }
  }
}

// ---------------------------------------------------------------------------
struct HeadArgsB {
  const uint16_t* h;  // [rows][H] fp16
  const uint16_t* theta;
  uint64_t off_w, off_b;
  int H, V;
  const float* zbo;  // [N][V]
  Key key;
  uint32_t i0;
  float eps;
  uint16_t eps_b;
  RowMap rm;
  int64_t M, rows;
  const int32_t* tokens;
  int C, t0, B;
  float* pmax;
  float* psum;
  float* ptgt;
  int nvt;  // vocabulary tiles
  const uint16_t* zc_out;  // probe cache: W_out's values of probe 0; probe n at + n * zc_stride
  uint64_t zc_stride;
  const uint16_t* w_out16;  // fp16 copy of W_out
};

template <int kind, bool kFD, bool kSplit>
__global__ __launch_bounds__(NT, 1) void head_bf16_kernel(HeadArgsB g) {
  using T = Tiles<kind>;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  int mb, vt;
  tile_of(blockIdx.x, (int)(g.rows / TM), g.nvt, mb, vt);
  const int v0 = vt * T::TN;
  const int64_t rr0 = (int64_t)mb * TM;
  const int tt = (int)(rr0 / g.M);
  const int64_t r0 = rr0 - (int64_t)tt * g.M;
  const int pair = pass_of(g.rm, r0).probe;
  const int sgn = pass_of(g.rm, r0 + T::WROWS * wm).sign;  // a wave tile lies inside one pass
  const int V = g.V;
  auto colmap = [&](int rho, int& n) { n = min(v0 + rho, V - 1); };
  f16v acc[T::MT][2];
  zero_acc(acc);
  const SegB s0{g.h + rr0 * g.H, g.H, g.w_out16, g.H, g.off_w, g.H,
                kind == kGaussCached ? g.zc_out + (uint64_t)pair * g.zc_stride : nullptr};
  mainloop_bf16<kind, true, kFD, kSplit>(acc, s0, s0, 1, colmap, g.key, g.i0 + (uint32_t)pair, sgn, g.eps,
                                         g.eps_b);

  // transposed tiles: acc[mt][nt][v] is the logit of activation row
  // WROWS wm + 32 mt + lr and vocabulary column cbase + 32 nt + vcol(v)
  const int cbase = v0 + 64 * wn;
  auto vcol = [&](int v) { return 8 * (v >> 2) + 4 * lg + (v & 3); };
  // bias and bias probe of each column held (-inf past the vocabulary)
  float add[2][16];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int col = cbase + 32 * nt + vcol(v);
      float a = -INFINITY;
      if (col < V) {
        const float b = bf16_to_f32(g.theta[g.off_b + (uint64_t)col]);
        const float z = g.zbo[(int64_t)pair * V + col];
        a = b + (float)sgn * z;
      }
      add[nt][v] = a;
    }
  }
  // cross-wave reduction in the first stage buffer (free after the loop)
  float* red_m = (float*)stage<kind, 0>();         // [WAVES_N][TM]
  float* red_s = red_m + T::WAVES_N * TM;          // [WAVES_N][TM]
#pragma unroll
  for (int mt = 0; mt < T::MT; ++mt) {
    const int lrow = T::WROWS * wm + 32 * mt + lr;
    const int b = pass_of(g.rm, r0 + lrow).b;
    const int tgt = b < g.B ? g.tokens[(int64_t)b * (g.C + 1) + g.t0 + tt + 1] - cbase : -1;
    float mx = -INFINITY, yt = 0.f;
    bool has_t = false;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float y = acc[mt][nt][v] + add[nt][v];
        acc[mt][nt][v] = y;
        mx = fmaxf(mx, y);
        const bool hit = tgt == 32 * nt + vcol(v);
        yt = hit ? y : yt;
        has_t = has_t || hit;
      }
    }
    if (has_t) g.ptgt[rr0 + lrow] = yt;
    // the row's 64 columns of this wave: 32 here, 32 in lane lr + 32
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float se = 0.f;
    if (mx != -INFINITY) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int v = 0; v < 16; ++v) se += __expf(acc[mt][nt][v] - mx);
    }
    se += __shfl_xor(se, 32, 64);
    if (lg == 0) {
      red_m[wn * TM + lrow] = mx;
      red_s[wn * TM + lrow] = se;
    }
  }
  __syncthreads();
  if (t < TM) {
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < T::WAVES_N; ++w) mx = fmaxf(mx, red_m[w * TM + t]);
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < T::WAVES_N; ++w) {
      const float m = red_m[w * TM + t];
      sum += m == -INFINITY ? 0.f : red_s[w * TM + t] * __expf(m - mx);
    }
    g.pmax[(int64_t)vt * g.rows + rr0 + t] = mx;
    g.psum[(int64_t)vt * g.rows + rr0 + t] = sum;
  }
}

// ---------------------------------------------------------------------------
// x0[r][e] = fp16(EMB[tok][e] + s eps z_n[emb + tok E + e]); zeros for padding
// rows, NaN for a token outside [0, V) (never read).
constexpr uint32_t kNaNf16x2 = 0x7E007E00u;
template <int kind>
__global__ __launch_bounds__(256) void embed_bf16_kernel(const uint16_t* theta, uint64_t emb_off, int E, int V,
                                                         const int32_t* tokens, int C, int t, int B,
                                                         RowMap rm, int64_t M, Key key, uint32_t i0,
                                                         float eps, uint16_t* x0) {
  const int E4 = E >> 2;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= M * E4) return;
  const int64_t r = idx / E4;
  const int e = (int)(idx - r * E4) * 4;
  const PassOf ps = pass_of(rm, r);
  const int pair = ps.probe, b = ps.b;
  uint32_t lo = 0u, hi = 0u;
  const int tok = b < B ? tokens[(int64_t)b * (C + 1) + t] : 0;
  if (b < B && (uint32_t)tok >= (uint32_t)V) {
    lo = hi = kNaNf16x2;
  } else if (b < B) {
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
    const float se = (float)ps.sign * eps;  // 0 for the clean pass
    lo = pack_f16x2(w[0] + se * z[0], w[1] + se * z[1]);
    hi = pack_f16x2(w[2] + se * z[2], w[3] + se * z[3]);
  }
  *(uint2*)(x0 + r * E + e) = uint2{lo, hi};
}

// Sign probes: one thread per 32 consecutive elements of a row, which share
// one Philox word (bit k of the word for element k), so a row costs E / 128
// Philox blocks instead of E / 4.
__global__ __launch_bounds__(256) void embed_bf16_rad_kernel(const uint16_t* theta, uint64_t emb_off, int E, int V,
                                                             const int32_t* tokens, int C, int t, int B,
                                                             RowMap rm, int64_t M, Key key, uint32_t i0,
                                                             float eps, uint16_t* x0) {
  const int E32 = E >> 5;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= M * E32) return;
  const int64_t r = idx / E32;
  const int e = (int)(idx - r * E32) * 32;
  const PassOf ps = pass_of(rm, r);
  const int pair = ps.probe, b = ps.b;
  u4 out[4] = {u4{0u, 0u, 0u, 0u}, u4{0u, 0u, 0u, 0u}, u4{0u, 0u, 0u, 0u}, u4{0u, 0u, 0u, 0u}};
  const int tok = b < B ? tokens[(int64_t)b * (C + 1) + t] : 0;
  if (b < B && (uint32_t)tok >= (uint32_t)V) {
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = u4{kNaNf16x2, kNaNf16x2, kNaNf16x2, kNaNf16x2};
  } else if (b < B) {
    const uint64_t j = emb_off + (uint64_t)tok * E + e;  // a multiple of 32: one whole word
    const uint32_t word = rademacher_word(key, i0 + pair, j >> 5);
    const float se = (float)ps.sign * eps;  // 0 for the clean pass
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u4 wv = *(const u4*)(theta + j + 8 * q);
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const int k = 8 * q + 2 * d;
        const float w0 = bf16_to_f32((uint16_t)wv[d]), w1 = bf16_to_f32((uint16_t)(wv[d] >> 16));
        const float z0 = ((word >> k) & 1u) ? 1.0f : -1.0f, z1 = ((word >> (k + 1)) & 1u) ? 1.0f : -1.0f;
        out[q][d] = pack_f16x2(w0 + se * z0, w1 + se * z1);
      }
    }
  }
  u4* dst = (u4*)(x0 + r * E + e);
#pragma unroll
  for (int q = 0; q < 4; ++q) dst[q] = out[q];
}

// Calls go(kind, fd, split) with the compile-time variant of this call: the
// probe kind (sign probes; normal probes read from the probe cache or
// regenerated), central or forward differences, fused or two-stream products.
template <typename Go>
void dispatch_bf16(const ForwardArgs& a, Go&& go) {
  using std::integral_constant;
  auto by_split = [&](auto kind_tag, auto fd_tag) {
    if (a.split) go(kind_tag, fd_tag, integral_constant<bool, true>{});
    else go(kind_tag, fd_tag, integral_constant<bool, false>{});
  };
  auto by_fd = [&](auto kind_tag) {
    if (a.rows.fd) by_split(kind_tag, integral_constant<bool, true>{});
    else by_split(kind_tag, integral_constant<bool, false>{});
  };
  if (a.cfg.probe == ZO_RADEMACHER) by_fd(integral_constant<int, ZO_RADEMACHER>{});
  else if (a.zc) by_fd(integral_constant<int, kGaussCached>{});
  else by_fd(integral_constant<int, ZO_GAUSSIAN>{});
}

}  // namespace

hipError_t launch_embed_bf16(const ForwardArgs& a, int t, void* x0, hipStream_t st) {
  const Rows& R = a.rows;
  const int E = a.cfg.embed;
  const RowMap rm = row_map(R);
  const Key key = make_key(a.seed);
  ProfScope ps(kKEmbed, st);
  if (a.cfg.probe == ZO_RADEMACHER) {
    const int64_t n = R.M * (E / 32);
    const unsigned grid = (unsigned)((n + 255) / 256);
    embed_bf16_rad_kernel<<<grid, 256, 0, st>>>((const uint16_t*)a.theta, a.lay.emb, E, a.cfg.vocab, a.tokens, a.C, t, R.B,
                                                rm, R.M, key, a.i0, a.eps, (uint16_t*)x0);
  } else {
    const int64_t n = R.M * (E / 4);
    const unsigned grid = (unsigned)((n + 255) / 256);
    embed_bf16_kernel<ZO_GAUSSIAN><<<grid, 256, 0, st>>>((const uint16_t*)a.theta, a.lay.emb, E,
                                                         a.cfg.vocab, a.tokens, a.C, t, R.B, rm, R.M, key, a.i0,
                                                         a.eps, (uint16_t*)x0);
  }
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
  g.eps_b = f16_rne(a.eps);
  g.rm = row_map(R);
  g.n_row_blocks = (int)(R.M / TM);
  g.w_ih16 = (const uint16_t*)a.w16 + a.zmap.ih[l];
  g.w_hh16 = (const uint16_t*)a.w16 + a.zmap.hh[l];
  g.zc_ih = a.zc ? (const uint16_t*)a.zc + a.zmap.ih[l] : nullptr;
  g.zc_hh = a.zc ? (const uint16_t*)a.zc + a.zmap.hh[l] : nullptr;
  g.zc_stride = a.zmap.pg;
  auto go = [&](auto kind_tag, auto fd_tag, auto split_tag) {
    constexpr int kind = decltype(kind_tag)::value;
    constexpr bool fd = decltype(fd_tag)::value;
    constexpr bool split = decltype(split_tag)::value;
    const dim3 grid((unsigned)(g.n_row_blocks * (g.H / (Tiles<kind>::TN / 4))));
    ProfScope ps(kKGate, st);
    gate_bf16_kernel<kind, fd, split><<<grid, NT, 0, st>>>(g);
  };
  dispatch_bf16(a, go);
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
  h.eps_b = f16_rne(a.eps);
  h.w_out16 = (const uint16_t*)a.w16 + a.zmap.out;
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
  h.nvt = a.ws.nvt;
  h.zc_out = a.zc ? (const uint16_t*)a.zc + a.zmap.out : nullptr;
  h.zc_stride = a.zmap.pg;
  const dim3 grid((unsigned)((int64_t)a.ws.nvt * (h.rows / TM)));
  auto go = [&](auto kind_tag, auto fd_tag, auto split_tag) {
    constexpr int kind = decltype(kind_tag)::value;
    constexpr bool fd = decltype(fd_tag)::value;
    constexpr bool split = decltype(split_tag)::value;
    ProfScope ps(kKHead, st);
    head_bf16_kernel<kind, fd, split><<<grid, NT, 0, st>>>(h);
  };
  dispatch_bf16(a, go);
  return hipGetLastError();
}

}  // namespace zo
