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
// sign probes, expanded from bits), or loads ready-formed (normal probes: the
// probe cache's perturbed weights, the same values). The parameter vector
// theta +- eps z is never formed. For small eps the two-stream form
// acc += A . W; acc += A . (s eps z) is used instead (kSplit).
//
// Tiles: a workgroup of 8 waves computes TM rows x TN columns, TM x TN =
// 65536 (TN = kVocabTileWide, 256: 256 x 256); its waves split the
// columns into TN / 64 wave columns and the rows into 8 / (TN / 64) wave
// rows, each wave computing 128 rows x 64 columns (4 x 2 tiles of 32x32 MFMA
// output). Two waves share each SIMD, so one wave's loads, probe expansion
// and address work run under the other's matrix instructions. Lane l feeds
// row/column l % 32 and k block l / 32.
//
// Operands. The activations (A) pass through LDS: each K tile of the TM rows
// is copied from global memory straight into LDS (buffer loads with the LDS
// destination, 1 KB per wave instruction), one tile ahead, into one of two
// stages, and read by every wave of its rows. The B operand (the fp16 weight
// copy, and the cached fp16(eps z) of normal probes) is loaded by each wave
// straight into registers, a few k steps ahead, from the fragment-packed
// copies the call writes (zo_pack.hpp): one contiguous 1 KB per wave
// instruction. Every global access is a buffer access against a resource
// sized to its matrix (or to the workgroup's activation rows), so an offset
// outside it reads zeros rather than faulting. The probe term: sign probes as
// two words of sign flags per column and K tile (regenerated, one Philox word
// per 32 k, or read from the sign-probe cache, one 8-byte load per thread
// for both words of a tile, into a ring of tile buffers) in a small LDS
// array of their own, which every lane expands into +-fp16(eps) fragments in
// registers;
// normal probes regenerated into an LDS tile per K tile, or read from the
// probe cache: with the fused form as the pass's perturbed weights
// fp16(W + s eps z), written once per call and loaded as the only B operand,
// with the two-stream form as fp16(eps z) loaded beside the weights.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "zo_kernels.hpp"
#include "zo_pack.hpp"
#include "zo_profile.hpp"
#include "zo_rng.hpp"

namespace zo {
namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f16v __attribute__((ext_vector_type(16)));
typedef uint32_t u4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

constexpr int TM = 65536 / kVocabTileWide;  // rows per workgroup (kVocabTileWide columns)
constexpr int NWAVES = 8;
constexpr int NT = 64 * NWAVES;  // threads per workgroup

// Per probe kind: K tile, LDS layout, copy roles, B-operand prefetch depth.
template <int kind>
struct Tiles {
  static constexpr bool kSigns = kind == ZO_RADEMACHER || kind == kSignsCached;
  static constexpr bool kBits = kind == kSignsCached;      // sign words read from the sign-probe cache
  static constexpr bool kZDirect = kind == kGaussCached;  // probe fragments loaded like the weights
  static constexpr bool kZTile = kind == ZO_GAUSSIAN;     // probe tile of regenerated normals formed in LDS
  static constexpr int TK = 64;                            // K per tile
  static constexpr int KSTEPS = TK / 16;                   // MFMA k steps per tile
  static constexpr int SW = TK / 32;                       // sign words per column and tile
  static constexpr int RowBytes = TK * 2;                  // one LDS row: TK fp16
  static constexpr int ABytes = TM * RowBytes;
  static constexpr int TN = kVocabTileWide;
  static constexpr int WAVES_N = TN / 64;  // wave tiles are 64 columns wide
  static constexpr int WAVES_M = NWAVES / WAVES_N;
  static constexpr int WROWS = TM / WAVES_M;  // rows per wave tile
  static constexpr int MT = WROWS / 32;
  static constexpr int ZTileBytes = TN * RowBytes;
  static constexpr int StageBytes = ABytes + (kZTile ? ZTileBytes : 0);
  static constexpr int ACopies = ABytes / 1024 / NWAVES;  // activation copies per wave and tile
  // B fragments for k step s + DIST are loaded at step s, into SLOTS rotating
  // register sets, as far ahead as the registers of two waves per SIMD allow
  // without spilling (fp16(eps z) as a second stream doubles the loads;
  // regenerated probes hold the generator's state): cached sign probes and
  // the perturbed-weight cache 7 k steps (c4 gate 2.25 -> 2.18 ms against 3),
  // the others 3 (c3 gate with fp16(eps z) streamed 0.90 -> 0.74 ms against 1).
  static constexpr bool kPerturbed = kind == kGaussPerturbed;  // B is the cached fp16(W + s eps z) itself
  static constexpr int DIST = kBits || kPerturbed ? 7 : 3;
  static constexpr int SLOTS = DIST < 4 ? 4 : 8;  // a divisor of the two K tiles the loop body spans
  static constexpr int LoadsPerStep = kZDirect ? 4 : 2;
  // probe-tile roles: thread t forms ZVALS consecutive k of column t / ZROW_T
  static constexpr int ZROW_T = NT / TN;
  static constexpr int ZVALS = TK / ZROW_T;
  static constexpr int WPT = ZVALS / 32;  // sign words (or blocks of 32 normals) per thread and tile
  static_assert(WAVES_M * WAVES_N == NWAVES && WROWS % 32 == 0, "wave grid");
  static_assert(ACopies * NWAVES * 1024 == ABytes, "copy split");
  static_assert((2 * KSTEPS) % SLOTS == 0 && SLOTS <= 8, "the B slots repeat every two tiles");
  static_assert(ZVALS % 32 == 0 && ZROW_T * TN == NT, "probe roles: whole 32-k sign words per thread");
  static_assert(kRowGranuleBF16 % WROWS == 0, "a wave tile lies inside one sign's rows");
  static_assert(RowBytes == 128, "swizzle of 128-byte rows (act_swizzle)");
};
static_assert(2 * kRowGranuleBF16 % TM == 0, "a probe's rows must be a whole number of row tiles");
static_assert(TM % 128 == 0 && TM * kVocabTileWide == 65536, "workgroup tile");

// LDS stages (static, so that every offset is a constant): activation tile
// and probe tile (regenerated normal probes), or the activation tile alone
// (sign probes, whose words have arrays of their own, and cached normal
// probes).
__shared__ __align__(16) uint8_t lds_s0[Tiles<ZO_GAUSSIAN>::StageBytes];
__shared__ __align__(16) uint8_t lds_s1[Tiles<ZO_GAUSSIAN>::StageBytes];
__shared__ __align__(16) uint8_t lds_c0[Tiles<kGaussCached>::StageBytes];
__shared__ __align__(16) uint8_t lds_c1[Tiles<kGaussCached>::StageBytes];
static_assert(Tiles<ZO_RADEMACHER>::StageBytes == Tiles<kGaussCached>::StageBytes, "activation-only stages");
static_assert(Tiles<kSignsCached>::StageBytes == Tiles<kGaussCached>::StageBytes, "activation-only stages");
static_assert(2 * sizeof(lds_s0) <= 160 * 1024, "LDS");
// Sign words of a K tile (two per workgroup column, unshuffled), per stage,
// in arrays of their own: the compiler orders an LDS store after every copy
// in flight into the same array.
constexpr int kWordBytes = kVocabTileWide * 2 * 4;
__shared__ __align__(16) uint8_t lds_words0[kWordBytes];
__shared__ __align__(16) uint8_t lds_words1[kWordBytes];
// Cached sign words: a ring of four tiles' words (tile t in buffer t % 4).
__shared__ __align__(16) uint8_t lds_wring[4 * kWordBytes];

// The gate's cell states c of its tile (TM rows x the TN / 4 hidden units of
// its columns, row-major), fetched before the main loop so that the cell
// update reads them from LDS; kinds whose stages leave room for it (not the
// regenerated normal probes' activation + probe stages).
constexpr int kCellCols = kVocabTileWide / 4;
__shared__ __align__(16) float lds_gc[TM * kCellCols];
static_assert(2 * sizeof(lds_c0) + 2 * kWordBytes + sizeof(lds_gc) <= 160 * 1024, "LDS");

// The head's bias values of its vocabulary tile, fetched before the main
// loop so that the epilogue finds them in LDS: 256 words of theta from the
// 4-byte boundary at or below the tile's first bias element (raw bf16), and
// the 256 bias-probe values eps z of the tile's columns.
__shared__ __align__(16) uint8_t lds_hbias[1024];
__shared__ __align__(16) float lds_hzbo[kVocabTileWide];
// bias + s eps z of each column for the rows of each sign (-inf past V)
__shared__ __align__(16) float lds_hadd[2][kVocabTileWide];
// the target token of each row of the head's tile (-1 for padding rows)
__shared__ __align__(16) int lds_htgt[TM];

template <int kind, int S>
__device__ __forceinline__ uint8_t* stage() {
  static_assert(S == 0 || S == 1, "stage index");
  if constexpr (!Tiles<kind>::kZTile)
    return S == 0 ? lds_c0 : lds_c1;
  else
    return S == 0 ? lds_s0 : lds_s1;
}
template <int S>
__device__ __forceinline__ uint8_t* words4() {
  static_assert(S == 0 || S == 1, "stage index");
  return S == 0 ? lds_words0 : lds_words1;
}

// The workgroup geometry of the loop, as the gate and head epilogues use it:
// 8 waves, 2 row halves x 4 column quarters, wave tiles of 128 rows x 64
// columns (4 x 2 tiles of 32x32).
struct Geo {
  static constexpr int WAVES_M = Tiles<ZO_GAUSSIAN>::WAVES_M, WAVES_N = Tiles<ZO_GAUSSIAN>::WAVES_N;
  static constexpr int WROWS = Tiles<ZO_GAUSSIAN>::WROWS, WCOLS = 64;
  static constexpr int MT = Tiles<ZO_GAUSSIAN>::MT, NTW = 2;
};

__device__ __forceinline__ h8 as_h8(u4 v) { return __builtin_bit_cast(h8, v); }

// Calls f(integral_constant<int, i>) for a slot index i < N <= 8 known only
// after unrolling (register arrays need compile-time indices).
template <int N, typename F>
__device__ __forceinline__ void with_slot(int i, F&& f) {
  static_assert(N >= 1 && N <= 8, "slots");
  auto call = [&](auto tag) {
    if constexpr (decltype(tag)::value < N) f(tag);
  };
  using std::integral_constant;
  switch (i) {
    case 0: call(integral_constant<int, 0>{}); break;
    case 1: call(integral_constant<int, 1>{}); break;
    case 2: call(integral_constant<int, 2>{}); break;
    case 3: call(integral_constant<int, 3>{}); break;
    case 4: call(integral_constant<int, 4>{}); break;
    case 5: call(integral_constant<int, 5>{}); break;
    case 6: call(integral_constant<int, 6>{}); break;
    default: call(integral_constant<int, 7>{}); break;
  }
}

// A raw buffer resource over [base, base + bytes), bytes < 2^31.
__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// 4 bytes per lane from global memory straight into LDS: lane L's word at
// lds + 4 L (lds wave-uniform); reads past the resource give zeros.
__device__ __forceinline__ void copy4_to_lds(Rsrc r, uint32_t voff, uint8_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 4, voff, 0, 0, 0);
}

// 16 bytes per lane from global memory straight into LDS: the wave's 64
// lanes fill the 1 KB at lds (wave-uniform), lane L at lds + 16 L; the
// address is the resource base + voff (per lane) + soff (wave-uniform).
__device__ __forceinline__ void copy_to_lds(Rsrc r, uint32_t voff, uint32_t soff, uint8_t* lds) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds, 16, voff, soff, 0, 0);
}

// One 16-byte B fragment piece per lane, straight into registers.
__device__ __forceinline__ h8 load_frag(Rsrc r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(h8, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Wait until at most VM of this thread's vector memory loads are outstanding
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

// Keeps the compiler from moving memory accesses or scheduling instructions
// across this point (the load counts of wait_and_barrier depend on the order
// in which the tile's loads are issued).
__device__ __forceinline__ void issue_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// One K segment of a product: the activations (A, rows of the workgroup's
// tile), the packed fp16 weight copy (B) and, for cached normal probes, this
// probe's packed fp16(eps z) of the same matrix.
struct SegB {
  const uint16_t* A;  // first row of this workgroup's activation tile; row r at A + r * lda
  int64_t lda;
  const uint16_t* W;  // packed fp16 weights of the matrix (cols x K)
  uint32_t wbytes;    // bytes of the packed matrix
  uint64_t zoff;      // offset of the matrix inside theta (probe coordinates)
  int64_t ldw;        // row stride of the matrix in theta (= K)
  int K;
  const uint16_t* Z;  // kGaussCached: fp16(eps z) of this probe and matrix, packed like W
};

// The sign-probe cache of this workgroup's probe (kSignsCached): bit_words(P)
// words, word w holding the signs of parameters 32 w .. 32 w + 31.
struct BitsB {
  const uint32_t* words;
  uint32_t bytes;
};

// acc: [MT row tiles][2 column tiles] of 32x32 fp32 for this wave. cb0: the
// packed column block of the workgroup's first column (8 per 256 columns).
// colmap(rho, &n) maps workgroup column rho (0..TN-1) to the weight row n in
// theta that carries its probe coordinates (columns beyond the matrix map to
// a valid row; they are never scored). sgn: the sign of eps for this wave's
// rows (+1, -1, or 0 for the clean pass of forward differences); eps_b: fp16
// bits of eps.
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
template <int kind, bool kTrans = false, bool kSplit = false, typename ColMap>
__device__ __forceinline__ void mainloop_bf16(f16v (&acc)[Tiles<kind>::MT][2], const SegB s0, const SegB s1,
                                              int nseg, int64_t cb0, ColMap colmap, Key key, uint32_t probe,
                                              int sgn, float eps, uint16_t eps_b, const BitsB bits) {
  using T = Tiles<kind>;
  static_assert(!(kSplit && T::kPerturbed), "the perturbed-weight cache holds the fused form only");
  constexpr int MT = T::MT;
  constexpr int TK = T::TK;
  constexpr int KSTEPS = T::KSTEPS;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wm = wave % T::WAVES_M, wn = wave / T::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  const int ntiles = s0.K / TK + (nseg > 1 ? s1.K / TK : 0);

  // Buffer resources: the workgroup's activation rows and the packed matrices
  // of each segment (the probe cache per probe).
  const Rsrc ra0 = make_rsrc(s0.A, (uint32_t)(TM * s0.lda * 2));
  const Rsrc ra1 = make_rsrc(s1.A, (uint32_t)(TM * s1.lda * 2));
  const Rsrc rw0 = make_rsrc(s0.W, s0.wbytes), rw1 = make_rsrc(s1.W, s1.wbytes);
  Rsrc rz0 = rw0, rz1 = rw1;
  if constexpr (T::kZDirect) {
    rz0 = make_rsrc(s0.Z, s0.wbytes);
    rz1 = make_rsrc(s1.Z, s1.wbytes);
  }
  // activation copies: copy q of this wave fills LDS rows act_row_of_copy(q,
  // wave, lane); its per-lane offset is row * lda * 2 + chunk * 16, the K
  // tile adds 2 k0 bytes (wave-uniform)
  uint32_t arow2[T::ACopies], achunk[T::ACopies];
#pragma unroll
  for (int q = 0; q < T::ACopies; ++q) {
    const int r = act_row_of_copy(q, wave, lane, NWAVES);
    arow2[q] = (uint32_t)r;
    achunk[q] = 16u * (uint32_t)((lane % 8) ^ act_swizzle(r));
  }
  const uint32_t lda2_0 = (uint32_t)(2 * s0.lda), lda2_1 = (uint32_t)(2 * s1.lda);
  // B fragments: lane part of the packed offset (the block and k step parts
  // are wave-uniform and go in the scalar offset)
  const uint32_t blane = (uint32_t)lane * 16u;
  const int64_t cbw = cb0 + 2 * wn;
  // probe-tile roles: column zr, 32 k at 32 zpart
  const int zr = t / T::ZROW_T, zpart = t % T::ZROW_T;
  int zn;
  colmap(zr, zn);

  // B fragments in flight: slot j holds the (weight, probe) fragments of the
  // k steps j, j + SLOTS, ... Every load below is issued unconditionally
  // (past the last k step it repeats the last one, and past the last tile
  // the copies repeat the last tile into the idle stage), so that the number
  // of loads between any two points of the loop is fixed: the compiler then
  // waits for each fragment with an exact count, and wait_and_barrier's counts
  // hold.
  h8 wfr[T::SLOTS][2], zfr[T::kZDirect ? T::SLOTS : 1][2];
  // The B loads of K tile ti: the segment's resources and the scalar offsets
  // of the tile's first k step in the wave's two column blocks, worked out
  // once per tile (k step p of the tile adds p kPackBlockBytes). Past the
  // last tile the loads repeat
  // the last tile (their values are never used).
  struct TileB {
    Rsrc rw, rz;
    uint32_t off[2];
  };
  const int ntiles0 = s0.K / TK;
  auto tile_b = [&](int ti) {
    ti = ti < ntiles ? ti : ntiles - 1;
    const bool second = ti >= ntiles0;
    const uint32_t kt = (uint32_t)(second ? ti - ntiles0 : ti);
    const uint32_t KS = (uint32_t)(second ? s1.K : s0.K) / 16u;
    TileB b;
    b.rw = second ? rw1 : rw0;
    b.rz = second ? rz1 : rz0;
    b.off[0] = ((uint32_t)cbw * KS + kt * (uint32_t)KSTEPS) * (uint32_t)kPackBlockBytes;
    b.off[1] = b.off[0] + KS * (uint32_t)kPackBlockBytes;
    return b;
  };
  // k step P of the tile b into slot SL
  auto load_b = [&](auto slot_tag, auto step_tag, const TileB& b) {
    constexpr int SL = decltype(slot_tag)::value;
    constexpr uint32_t P = decltype(step_tag)::value;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
      const uint32_t soff = b.off[nt] + P * (uint32_t)kPackBlockBytes;
      wfr[SL][nt] = load_frag(b.rw, blane, soff);
      if constexpr (T::kZDirect) zfr[SL][nt] = load_frag(b.rz, blane, soff);
    }
  };

  Words zcache{{0u, 0u, 0u, 0u}};
  int seg = 0, k0 = 0;  // the next tile to be copied (stays on the last tile once past it)
  // advance (seg, k0) by one K tile, staying on the last tile once past it
  auto next_tile = [&](int& sg_, int& k_) {
    const int K = sg_ == 0 ? s0.K : s1.K;
    k_ += TK;
    if (k_ == K) {
      if (sg_ + 1 < nseg) {
        k_ = 0;
        ++sg_;
      } else {
        k_ -= TK;
      }
    }
  };
  // cached sign words: every thread reads the two words (64 k) of its column
  // zn for one tile with one 8-byte load, two tiles per round: at each even
  // tile it, thread (zn, zpart) loads tile it + 2 + zpart's words; at the
  // following odd tile both tiles' words (stored unshuffled in the cache) go
  // into the ring of four LDS buffers (tile t in buffer t % 4, rewritten two
  // barriers after its tile was read)
  Rsrc rbits = rw0;
  if constexpr (T::kBits) rbits = make_rsrc(bits.words, bits.bytes);
  uint2 wq = {0u, 0u};
  auto tile_words = [&](int ti) {
    ti = ti < ntiles ? ti : ntiles - 1;  // past the last tile: its words again (never read)
    const bool second = ti >= ntiles0;
    const SegB& sg = second ? s1 : s0;
    const uint64_t kt = (uint64_t)(second ? ti - ntiles0 : ti) * TK;
    const uint64_t j0 = sg.zoff + (uint64_t)zn * (uint64_t)sg.ldw + kt;
    return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rbits, sign_word_offset(j0), 0, 0));
  };
  auto put_words = [&](int ti, uint2 w) { *(uint2*)(lds_wring + (ti & 3) * kWordBytes + zr * 8) = w; };

  // The next K tile's activation copies into stage S (the last loads of a
  // tile before its B loads: the count wait_and_barrier leaves in flight).
  auto issue_copies = [&](auto stage_tag) {
    constexpr int S = decltype(stage_tag)::value;
    uint8_t* base = stage<kind, S>();
    const bool second = seg != 0;
    const uint32_t lda2 = second ? lda2_1 : lda2_0;
#pragma unroll
    for (int q = 0; q < T::ACopies; ++q)
      copy_to_lds(second ? ra1 : ra0, arow2[q] * lda2 + achunk[q], 2u * (uint32_t)k0,
                  base + (q * NWAVES + wave) * 1024);
  };
  // The next K tile's probe part into stage S, then advance to the
  // following tile: the sign words of the tile's TN columns (WPT words per
  // thread: regenerated, or read from the sign-probe cache), or the tile of
  // fp16(eps z) of regenerated normal probes (eight Box-Muller blocks per 32
  // k). Cached normal probes have no probe part.
  auto issue_probe = [&](auto stage_tag) {
    constexpr int S = decltype(stage_tag)::value;
    const SegB& sg = seg == 0 ? s0 : s1;
    const uint64_t j0 = sg.zoff + (uint64_t)zn * (uint64_t)sg.ldw + (uint64_t)k0 + T::ZVALS * zpart;
    if constexpr (T::kSigns && !T::kBits) {
      const bool aligned = (sg.zoff % 128u) == 0 && (sg.ldw % 128) == 0;
#pragma unroll
      for (int i = 0; i < T::WPT; ++i) {
        const uint64_t j = j0 + 32u * (uint64_t)i;
        uint32_t word;
        if (aligned) {
          // one Philox block holds the words of 128 k
          if ((j & 127u) == 0 || i == 0) zcache = stream_block(key, j >> 7, probe, kTagRademacher);
          const int q = (int)((j >> 5) & 3u);
          word = q == 0 ? zcache.w[0] : q == 1 ? zcache.w[1] : q == 2 ? zcache.w[2] : zcache.w[3];
        } else {
          word = rademacher_word(key, probe, j >> 5);
        }
        // the word of column zr's 32 k at 32 (WPT zpart + i), unshuffled
        *(uint32_t*)(words4<S>() + zr * 8 + (T::WPT * zpart + i) * 4) = sign_word_unshuffle(word);
      }
    } else if constexpr (T::kZTile) {
      uint8_t* zrow = stage<kind, S>() + T::ABytes + zr * T::RowBytes;
#pragma unroll 2
      for (int c = 0; c < 4 * T::WPT; ++c) {
        float za[4], zb[4];
        gauss_block(key, probe, (j0 >> 2) + 2 * c, za);
        gauss_block(key, probe, (j0 >> 2) + 2 * c + 1, zb);
        *(u4*)(zrow + 16 * ((4 * T::WPT * zpart + c) ^ act_swizzle(zr))) =
            u4{pack_f16x2(eps * za[0], eps * za[1]), pack_f16x2(eps * za[2], eps * za[3]),
               pack_f16x2(eps * zb[0], eps * zb[1]), pack_f16x2(eps * zb[2], eps * zb[3])};
      }
    }
    next_tile(seg, k0);
  };

  // Fragments of one 16-k step: activations (MT row tiles) and probe values
  // (2 column tiles) from LDS, the next step's read while the current one
  // computes. Lane (lr, lg) reads chunk 2 s + lg of its rows, in slot
  // (2 s) ^ y with y = lg ^ swz(lr) (every row offset below is a multiple of
  // 16, the swizzle period).
  const uint32_t y = (uint32_t)(lg ^ act_swizzle(lr));
  const uint32_t a_lane = (uint32_t)(T::WROWS * wm + lr) * T::RowBytes;
  const uint32_t z_lane = (uint32_t)(64 * wn + lr) * T::RowBytes;
  // the sign of eps of this wave's rows as a packed fp16 pair (+-1, or 0 for
  // the clean pass): B = fp16(W + s eps z) is one packed fp16 fma per pair
  const _Float16 sh = (_Float16)(float)sgn;
  const h8 s8 = {sh, sh, sh, sh, sh, sh, sh, sh};
  // sign probes: the fragment of lane (lr, lg) at k step s holds k = 16 s +
  // 8 lg + e of the tile, i.e. flags 8 (s % 2) + 4 lg + d (d = e / 2) of the
  // unshuffled word s / 2 of its column; the pre-shift by 4 lg leaves
  // 8 (s % 2) + d. A set flag means z = +1; the pass sign flips them all
  // (the clean pass of forward differences gives +-0).
  const uint32_t flip = sgn < 0 ? 0u : 0xFFFFFFFFu;
  const uint32_t lshift = 4u * (uint32_t)lg;
  const uint32_t ebits = sgn == 0 ? 0u : ((uint32_t)eps_b | ((uint32_t)eps_b << 16));
  const uint32_t w_lane = (uint32_t)((64 * wn + lr) * 8);
  struct Frag {
    h8 a[MT], z[2];
  };
  constexpr int kQ0 = T::DIST / KSTEPS, kQ1 = (KSTEPS - 1 + T::DIST) / KSTEPS;
  auto compute = [&](auto stage_tag, int it) {
    constexpr int S = decltype(stage_tag)::value;
    constexpr std::integral_constant<int, 1 - S> next{};
    const uint8_t* base = stage<kind, S>();
    const uint8_t* pa = base + a_lane;
    const uint8_t* pz = base + T::ABytes + z_lane;
    // the B tiles this tile's steps load from: it + kQ0 .. it + kQ1
    TileB tb[kQ1 - kQ0 + 1];
#pragma unroll
    for (int q = 0; q <= kQ1 - kQ0; ++q) tb[q] = tile_b(it + kQ0 + q);
    uint32_t us[2][2] = {};
    if constexpr (T::kSigns) {
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        const uint8_t* wsrc;
        if constexpr (T::kBits)
          wsrc = lds_wring + (it & 3) * kWordBytes;
        else
          wsrc = words4<S>();
        const uint2 wd = *(const uint2*)(wsrc + w_lane + 32 * 8 * nt);
        us[nt][0] = (wd.x ^ flip) >> lshift;
        us[nt][1] = (wd.y ^ flip) >> lshift;
      }
    }
    auto load = [&](int s, Frag& f) {
      const uint32_t so = 16u * ((uint32_t)(2 * s) ^ y);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) f.a[mt] = as_h8(*(const u4*)(pa + 32 * mt * T::RowBytes + so));
      if constexpr (T::kZTile) {
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) f.z[nt] = as_h8(*(const u4*)(pz + 32 * nt * T::RowBytes + so));
      }
    };
    Frag f[2];
    load(0, f[0]);
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      const Frag& c = f[s & 1];
      if (s == 0) {
        // the sign words of the next round's two tiles (cached, even tiles),
        // then the next tile's activation copies, then this step's B loads
        if constexpr (T::kBits && S == 0) {
          wq = tile_words(it + 2 + zpart);
          issue_fence();
        }
        issue_copies(next);
        issue_fence();
      }
      // B fragments DIST steps ahead: k step (s + DIST) % KSTEPS of tile
      // it + (s + DIST) / KSTEPS
      with_slot<T::SLOTS>((S * KSTEPS + s + T::DIST) % T::SLOTS, [&](auto slot_tag) {
        with_slot<KSTEPS>((s + T::DIST) % KSTEPS, [&](auto step_tag) {
          load_b(slot_tag, step_tag, tb[(s + T::DIST) / KSTEPS - kQ0]);
        });
      });
      if (s + 1 < KSTEPS) load(s + 1, f[(s + 1) & 1]);
      // this step's weight fragments (slot s % SLOTS) and probe fragments
      h8 w[2], z[2];
#pragma unroll
      for (int nt = 0; nt < 2; ++nt) {
        with_slot<T::SLOTS>((S * KSTEPS + s) % T::SLOTS, [&](auto slot_tag) {
          constexpr int SL = decltype(slot_tag)::value;
          w[nt] = wfr[SL][nt];
          if constexpr (T::kZDirect) z[nt] = zfr[SL][nt];
        });
        if constexpr (T::kZTile) z[nt] = c.z[nt];
        if constexpr (T::kSigns) {
          const uint32_t u = us[nt][s >> 1];
          u4 v;
#pragma unroll
          for (int d = 0; d < 4; ++d) v[d] = ((u << (15 - 8 * (s & 1) - d)) & 0x80008000u) | ebits;
          z[nt] = as_h8(v);  // s eps z, the pass sign included
        }
      }
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
        h8 sz[2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) sz[nt] = T::kSigns ? z[nt] : z[nt] * s8;
        mma(w);
        mma(sz);
      } else {
        // B = fp16(W + s eps z): one packed fp16 fma per pair (s z exact,
        // one rounding to nearest even), then one MFMA per accumulator
        h8 wz[2];
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          if constexpr (T::kPerturbed)
            wz[nt] = w[nt];  // formed once per call by the cache fill, the same value bit for bit
          else
            wz[nt] = T::kSigns ? w[nt] + z[nt] : __builtin_elementwise_fma(z[nt], s8, w[nt]);
        }
        mma(wz);
      }
      if (s == 2) {
        if constexpr (T::kBits && S == 1) put_words(it + 1 + zpart, wq);
        issue_probe(next);
      }
    }
  };

  // K tile it lives in stage it % 2. Before tile it: wait for this thread's
  // copies of tile it (the B loads issued after them may stay in flight) and
  // its LDS writes; barrier (tile it complete for every wave, and the stage
  // computed at it - 1 free); compute it while issuing tile it + 1 into the
  // other stage. Prologue: the sign words of tiles 0 and 1 (cached, put into
  // the ring after the B loads are issued), tile 0's copies and probe part,
  // the first DIST steps' B loads.
  if constexpr (T::kBits) {
    wq = tile_words(zpart);
    issue_fence();
  }
  issue_copies(std::integral_constant<int, 0>{});
  issue_fence();
  {
    TileB tb0[(T::DIST - 1) / KSTEPS + 1];
#pragma unroll
    for (int q = 0; q <= (T::DIST - 1) / KSTEPS; ++q) tb0[q] = tile_b(q);
#pragma unroll
    for (int g = 0; g < T::DIST; ++g)
      with_slot<T::SLOTS>(g, [&](auto slot_tag) {
        with_slot<KSTEPS>(g % KSTEPS, [&](auto step_tag) { load_b(slot_tag, step_tag, tb0[g / KSTEPS]); });
      });
  }
  if constexpr (T::kBits) put_words(zpart, wq);
  issue_probe(std::integral_constant<int, 0>{});
  // loads issued after the copies of the tile a barrier waits for: the first
  // DIST steps' B loads (prologue), then a whole tile's B loads (every later
  // tile); the cached sign words are issued before the copies
  constexpr int kAfter0 = T::DIST * T::LoadsPerStep;
  constexpr int kAfter = KSTEPS * T::LoadsPerStep;
  wait_and_barrier<kAfter0>();
  int it = 0;
  for (; it + 1 < ntiles; it += 2) {
    compute(std::integral_constant<int, 0>{}, it);
    wait_and_barrier<kAfter>();
    compute(std::integral_constant<int, 1>{}, it + 1);
    wait_and_barrier<kAfter>();
  }
  if (it < ntiles) compute(std::integral_constant<int, 0>{}, it);
  __syncthreads();  // every wave done with the stages (and every copy landed) before they are reused
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
__device__ __forceinline__ int acc_row(int wm, int mt, int lg, int v) {
  return Geo::WROWS * wm + 32 * mt + 8 * (v >> 2) + 4 * lg + (v & 3);
}

template <int MT, int NTW>
__device__ __forceinline__ void zero_acc(f16v (&acc)[MT][NTW]) {
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) acc[mt][nt] = f16v{};
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
  const uint32_t* bits;    // sign-probe cache (kSignsCached): probe 0's words; probe n at + n * bits_stride
  uint64_t bits_stride;
};

// Workgroup: TM rows x TN / 4 hidden units (TN gate columns). Column rho = 64 ug
// + c of the workgroup is gate c / 16 of unit 16 ug + c % 16; a wave's
// column tiles come in pairs (2 p, 2 p + 1) covering one group ug of 16
// units, so lane lr holds gates i, g (lr < 16) or f, o (lr >= 16) of unit
// lr % 16 in the pair, and one exchange with lane lr ^ 16 brings all four
// gates of a (row, unit) together.
template <int kind, bool kFD, bool kSplit>
__global__ __launch_bounds__(NT, 1) void gate_bf16_kernel(GateArgsB g) {
  using G = Geo;
  constexpr int TN = kVocabTileWide;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % G::WAVES_M, wn = wave / G::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  int mb, nb;
  tile_of(blockIdx.x, g.n_row_blocks, (4 * g.H + TN - 1) / TN, mb, nb);
  const int u0 = nb * (TN / 4);
  const int64_t m0 = (int64_t)mb * TM;
  const int pair = pass_of(g.rm, m0).probe;
  const int sgn = pass_of(g.rm, m0 + G::WROWS * wm).sign;  // a wave tile lies inside one pass
  const int H = g.H;
  // (columns past the 4H of the matrix, in a last workgroup column block
  // that 4H does not fill, map to its last row; they are never scored)
  auto colmap = [&](int rho, int& n) {
    const int c = rho & 63;
    n = min((c >> 4) * H + u0 + 16 * (rho >> 6) + (c & 15), 4 * H - 1);
  };
  f16v acc[G::MT][G::NTW];
  zero_acc(acc);
  const uint64_t zpos = (uint64_t)pair * g.zc_stride;
  // kGaussPerturbed: this wave's B operand is its pass's perturbed weights
  // (block 2 pair for +eps, 2 pair + 1 for -eps), or the plain weights for the
  // clean pass of forward differences
  const uint64_t ppos = (uint64_t)(2 * pair + (sgn < 0 ? 1 : 0)) * g.zc_stride;
  const bool pert = kind == kGaussPerturbed && sgn != 0;
  const SegB s0{g.x + m0 * g.El, g.El, pert ? g.zc_ih + ppos : g.w_ih16, (uint32_t)((uint64_t)4 * H * g.El * 2),
                g.off_ih, g.El, g.El, kind == kGaussCached ? g.zc_ih + zpos : nullptr};
  const SegB s1{g.hprev + m0 * H, H, pert ? g.zc_hh + ppos : g.w_hh16, (uint32_t)((uint64_t)4 * H * H * 2), g.off_hh,
                H, H, kind == kGaussCached ? g.zc_hh + zpos : nullptr};
  const BitsB bits{kind == kSignsCached ? g.bits + (uint64_t)pair * g.bits_stride : nullptr,
                   (uint32_t)(g.bits_stride * 4)};
  constexpr bool kCellLds = !Tiles<kind>::kZTile;
  if constexpr (kCellLds) {
    // the tile's cell states into LDS: 1 KB copies of 4 rows (16 lanes of 16
    // bytes per row), copy j of wave w is copy 8 j + w of the 64; issued
    // before the loop's first loads, so its first barrier waits for them
    static_assert(TM * kCellCols * 4 == 64 * 1024 && kCellCols == 64, "cell tile copies");
    const Rsrc rc = make_rsrc(g.cst + m0 * H, (uint32_t)TM * (uint32_t)H * 4u);
    const int w = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int cp = 8 * j + w;
      copy_to_lds(rc, cell_copy_offset(cp, lane, H, u0), 0u, (uint8_t*)lds_gc + 1024 * cp);
    }
  }
  mainloop_bf16<kind, false, kSplit>(acc, s0, s1, 2, (TN / kPackBlockCols) * (int64_t)nb, colmap, g.key,
                                     g.i0 + (uint32_t)pair, sgn, g.eps, g.eps_b, bits);

  constexpr int NP = G::NTW / 2;  // unit groups per wave
  if (u0 + 16 * NP * wn >= H) return;  // a wave past the hidden units (wave-uniform)
  const int hi = lr >> 4;         // 0: gates i, g; 1: gates f, o
  int u[NP];
  float bias[NP][2];
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    u[p] = u0 + 16 * (NP * wn + p) + (lr & 15);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int gate = 2 * q + hi;
      const float b = bf16_to_f32(g.theta[g.off_b + (uint64_t)(gate * H + u[p])]);
      const float z = g.zb[(int64_t)pair * 4 * H + gate * H + u[p]];
      bias[p][q] = b + (float)sgn * z;
    }
  }
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt) {
#pragma unroll
    for (int p = 0; p < NP; ++p) {
#pragma unroll
      for (int v = 0; v < 16; v += 2) {
        // lanes lr < 16 update row element v, lanes lr >= 16 element v + 1
        float mine[2], send[2], got[2];
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const f16v& a = acc[mt][2 * p + q];
          const float p0 = a[v] + bias[p][q], p1 = a[v + 1] + bias[p][q];
          mine[q] = hi ? p1 : p0;
          send[q] = hi ? p0 : p1;
          got[q] = __shfl_xor(send[q], 16, 64);
        }
        const float ip = hi ? got[0] : mine[0], fp = hi ? mine[0] : got[0];
        const float gp = hi ? got[1] : mine[1], op = hi ? mine[1] : got[1];
        const int lrow = acc_row(wm, mt, lg, v + hi);
        const int64_t o = (m0 + lrow) * H + u[p];
        const float cprev = kCellLds ? lds_gc[lrow * kCellCols + (u[p] - u0)] : g.cst[o];
        const float c = sigm(fp) * cprev + sigm(ip) * tanh_(gp);
        g.cst[o] = c;
        g.hout[o] = f16_bits(sigm(op) * tanh_(c));
      }
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
  const uint32_t* bits;     // sign-probe cache (kSignsCached), as in GateArgsB
  uint64_t bits_stride;
};

template <int kind, bool kFD, bool kSplit>
__global__ __launch_bounds__(NT, 1) void head_bf16_kernel(HeadArgsB g) {
  using G = Geo;
  constexpr int TN = kVocabTileWide;
  constexpr int NTW = G::NTW;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave % G::WAVES_M, wn = wave / G::WAVES_M;
  const int lr = lane & 31, lg = lane >> 5;
  int mb, vt;
  tile_of(blockIdx.x, (int)(g.rows / TM), g.nvt, mb, vt);
  if constexpr (kind == kGaussPerturbed || kind == kGaussCached) {
    // Normal-probe caches: the weight operand differs per pass (or probe),
    // so the row blocks tile_of groups on one XCD are taken as one pass
    // block's consecutive timesteps (the order's block mb is timestep
    // mb % Tc of pass block mb / Tc), which then share each cached W_out
    // tile instead of each reading its own. Any order is correct.
    const int per_t = (int)(g.M / TM), Tc = (int)(g.rows / g.M);
    const int pb = mb / Tc, ts = mb - pb * Tc;
    mb = ts * per_t + pb;
  }
  const int v0 = vt * TN;
  const int64_t rr0 = (int64_t)mb * TM;
  const int tt = (int)(rr0 / g.M);
  const int64_t r0 = rr0 - (int64_t)tt * g.M;
  const int pair = pass_of(g.rm, r0).probe;
  const int sgn = pass_of(g.rm, r0 + G::WROWS * wm).sign;  // a wave tile lies inside one pass
  const int V = g.V;
  auto colmap = [&](int rho, int& n) { n = min(v0 + rho, V - 1); };
  f16v acc[G::MT][NTW];
  zero_acc(acc);
  const bool pert = kind == kGaussPerturbed && sgn != 0;  // as in the gate kernel
  const uint64_t ppos = (uint64_t)(2 * pair + (sgn < 0 ? 1 : 0)) * g.zc_stride;
  const SegB s0{g.h + rr0 * g.H, g.H, pert ? g.zc_out + ppos : g.w_out16,
                (uint32_t)((uint64_t)g.nvt * TN * g.H * 2), g.off_w, g.H, g.H,
                kind == kGaussCached ? g.zc_out + (uint64_t)pair * g.zc_stride : nullptr};
  const BitsB bits{kind == kSignsCached ? g.bits + (uint64_t)pair * g.bits_stride : nullptr,
                   (uint32_t)(g.bits_stride * 4)};
  // the tile's bias values into LDS (waves 0-3: eps z of the bias, one column
  // per lane; waves 4-7: the bf16 bias as 4-byte words from the aligned
  // boundary; columns past V read zeros). Issued before the loop's first
  // loads: its first barrier waits for them. The word resource spans the
  // 4-byte words that hold the V bias values: at most 2 bytes before the
  // first and 2 after the last, inside those aligned words, so inside the
  // pages that hold theta.
  const uintptr_t bias_at = (uintptr_t)(g.theta + g.off_b);
  const uint32_t bias_lead = (uint32_t)(bias_at & 3u);  // 0 or 2 bytes before the first element
  {
    const int q = __builtin_amdgcn_readfirstlane(wave);
    if (q < 4) {
      const Rsrc rz = make_rsrc(g.zbo + (int64_t)pair * V, (uint32_t)V * 4u);
      copy4_to_lds(rz, head_probe_offset(v0, q, lane), (uint8_t*)lds_hzbo + 256 * q);
    } else {
      const Rsrc rb = make_rsrc((const void*)(bias_at - bias_lead), head_bias_bytes(bias_lead, V));
      copy4_to_lds(rb, head_bias_word_offset(v0, 64 * (q - 4) + lane), lds_hbias + 256 * (q - 4));
    }
  }
  // the target token of tile row t (threads t < TM), read before the loop
  // and held in a register through it
  int tgt_tok = -1;
  if (t < TM) {
    const int b = pass_of(g.rm, r0 + t).b;
    if (b < g.B) tgt_tok = g.tokens[(int64_t)b * (g.C + 1) + g.t0 + tt + 1];
  }
  mainloop_bf16<kind, true, kSplit>(acc, s0, s0, 1, (TN / kPackBlockCols) * (int64_t)vt, colmap, g.key,
                                    g.i0 + (uint32_t)pair, sgn, g.eps, g.eps_b, bits);

  // transposed tiles: acc[mt][nt][v] is the logit of activation row
  // WROWS wm + 32 mt + lr and vocabulary column cbase + 32 nt + vcol(v)
  const int cbase = v0 + G::WCOLS * wn;
  auto vcol = [&](int v) { return 8 * (v >> 2) + 4 * lg + (v & 3); };
  // bias + s eps z of the tile's columns for the rows of each wave row
  // (thread t: wave row t / TN, column t % TN), then per lane the columns it
  // holds, four consecutive ones per read (-inf past the vocabulary)
  static_assert(NT == G::WAVES_M * TN && G::WAVES_M == 2, "one thread per wave row and column");
  {
    const int c = t % TN, half = t / TN;
    const int sg = pass_of(g.rm, r0 + G::WROWS * half).sign;
    const float b = bf16_to_f32(*(const uint16_t*)(lds_hbias + bias_lead + 2 * c));
    lds_hadd[half][c] = v0 + c < V ? b + (float)sg * lds_hzbo[c] : -INFINITY;
    if (t < TM) lds_htgt[t] = tgt_tok;
  }
  __syncthreads();
  float add[NTW][16];
#pragma unroll
  for (int nt = 0; nt < NTW; ++nt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 a4 = *(const float4*)&lds_hadd[wm][G::WCOLS * wn + 32 * nt + vcol(4 * j)];
      add[nt][4 * j] = a4.x;
      add[nt][4 * j + 1] = a4.y;
      add[nt][4 * j + 2] = a4.z;
      add[nt][4 * j + 3] = a4.w;
    }
  }
  // cross-wave reduction in the first stage buffer (free after the loop)
  float* red_m = (float*)stage<kind, 0>();  // [WAVES_N][TM]
  float* red_s = red_m + G::WAVES_N * TM;   // [WAVES_N][TM]
#pragma unroll
  for (int mt = 0; mt < G::MT; ++mt) {
    const int lrow = G::WROWS * wm + 32 * mt + lr;
    const int tgt = lds_htgt[lrow] - cbase;  // negative (never a held column) for padding rows
    float mx = -INFINITY;
#pragma unroll
    for (int nt = 0; nt < NTW; ++nt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float y = acc[mt][nt][v] + add[nt][v];
        acc[mt][nt][v] = y;
        mx = fmaxf(mx, y);
      }
    }
    // the target logit, where a lane of the wave holds its row's target
    // column (lane group lg holds the columns with bit 2 equal to lg); the
    // rest of the time the wave skips the search
    const bool holds_t = (unsigned)tgt < (unsigned)G::WCOLS && ((tgt >> 2) & 1) == lg;
    if (__builtin_amdgcn_ballot_w64(holds_t) != 0) {
      float yt = 0.f;
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
        for (int v = 0; v < 16; ++v) yt = tgt == 32 * nt + vcol(v) ? acc[mt][nt][v] : yt;
      if (holds_t) g.ptgt[rr0 + lrow] = yt;
    }
    // the row's WCOLS columns of this wave: half here, half in lane lr + 32
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    // sum of exp(y - mx) as 2^(y log2(e) - mx log2(e)) (one fma and one
    // v_exp_f32 per column)
    constexpr float kLog2e = 1.4426950408889634f;
    float se = 0.f;
    if (mx != -INFINITY) {
      const float mxl = mx * kLog2e;
#pragma unroll
      for (int nt = 0; nt < NTW; ++nt)
#pragma unroll
        for (int v = 0; v < 16; ++v) se += __builtin_amdgcn_exp2f(fmaf(acc[mt][nt][v], kLog2e, -mxl));
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
    for (int w = 0; w < G::WAVES_N; ++w) mx = fmaxf(mx, red_m[w * TM + t]);
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < G::WAVES_N; ++w) {
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
  if (a.cfg.probe == ZO_RADEMACHER && a.bits) by_fd(integral_constant<int, kSignsCached>{});
  else if (a.cfg.probe == ZO_RADEMACHER) by_fd(integral_constant<int, ZO_RADEMACHER>{});
  else if (a.zc && !a.split) {
    // perturbed weights hold the fused form only
    if (a.rows.fd) go(integral_constant<int, kGaussPerturbed>{}, integral_constant<bool, true>{}, integral_constant<bool, false>{});
    else go(integral_constant<int, kGaussPerturbed>{}, integral_constant<bool, false>{}, integral_constant<bool, false>{});
  }
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
  g.bits = a.bits;
  g.bits_stride = bit_words(a.lay.total);
  auto go = [&](auto kind_tag, auto fd_tag, auto split_tag) {
    constexpr int kind = decltype(kind_tag)::value;
    constexpr bool fd = decltype(fd_tag)::value;
    constexpr bool split = decltype(split_tag)::value;
    const dim3 grid((unsigned)(g.n_row_blocks * ((4 * g.H + kVocabTileWide - 1) / kVocabTileWide)));
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
  h.bits = a.bits;
  h.bits_stride = bit_words(a.lay.total);
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
