// Shapes, parameter layout, pass/row numbering and workspace plan of the
// CD-RGE step, shared by the host launchers and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/zo.h"

namespace zo {

constexpr int kMaxLayers = 64;

// Flat parameter layout (the model as one vector, every element perturbed):
// EMB[V][E]; per layer W_ih[4H][E_l], W_hh[4H][H], b[4H]; W_out[V][H]; b_out[V].
struct Layout {
  uint64_t emb;
  uint64_t w_ih[kMaxLayers];
  uint64_t w_hh[kMaxLayers];
  uint64_t bias[kMaxLayers];
  uint64_t w_out;
  uint64_t b_out;
  uint64_t total;
};

inline bool config_valid(const zo_config* c) {
  return c && c->n_layers >= 1 && c->n_layers <= kMaxLayers && c->vocab >= 1 && c->embed >= 1 &&
         c->hidden >= 1 && (c->wdtype == ZO_WFP32 || c->wdtype == ZO_WBF16) &&
         (c->probe == ZO_RADEMACHER || c->probe == ZO_GAUSSIAN);
}

inline Layout make_layout(const zo_config& c) {
  Layout L{};
  const uint64_t V = (uint64_t)c.vocab, E = (uint64_t)c.embed, H = (uint64_t)c.hidden;
  uint64_t p = 0;
  L.emb = p;
  p += V * E;
  for (int l = 0; l < c.n_layers; ++l) {
    const uint64_t El = l == 0 ? E : H;
    L.w_ih[l] = p;
    p += 4 * H * El;
    L.w_hh[l] = p;
    p += 4 * H * H;
    L.bias[l] = p;
    p += 4 * H;
  }
  L.w_out = p;
  p += V * H;
  L.b_out = p;
  p += V;
  L.total = p;
  return L;
}

// Rows of the batched forward. The passes each run the B sequences; every
// matrix product of a timestep covers all of them at once. B is padded to Bp
// (a multiple of the path's row granule) so that every row tile of a kernel
// lies inside one pass (and, for central differences, one probe). Padded
// rows (b >= B) carry zeros in, are computed like the others and never
// scored.
//   central differences (2N passes): row r = (2 n + sidx) Bp + b with sidx 0
//     for theta + eps z_n and 1 for theta - eps z_n;
//   forward differences (N + 1 passes): row r = p Bp + b, pass p < N at
//     theta + eps z_p, pass N at theta itself (the clean pass).
constexpr int kRowGranuleF32 = 32;   // fp32 path: 64-row tiles, 32-row wave tiles
constexpr int kRowGranuleBF16 = 128; // bf16 path: 256-row tiles

inline int row_granule(const zo_config& c, bool fd = false) {
  // forward differences: a whole row tile (64 or 256 rows) inside one pass
  if (fd) return c.wdtype == ZO_WBF16 ? 2 * kRowGranuleBF16 : 2 * kRowGranuleF32;
  return c.wdtype == ZO_WBF16 ? kRowGranuleBF16 : kRowGranuleF32;
}

struct Rows {
  int32_t B, Bp, N;
  int64_t pair_rows;  // rows of one probe: 2 Bp (central) or Bp (forward)
  int64_t M;          // all rows: 2 N Bp (central) or (N + 1) Bp (forward)
  int fd;
};

struct RowMap {
  int Bp;
  int64_t pair_rows;
  int fd;  // forward differences
  int N;
};

inline Rows make_rows(int32_t N, int32_t B, int granule, bool fd = false) {
  Rows r;
  r.B = B;
  r.N = N;
  r.fd = fd ? 1 : 0;
  r.Bp = (B + granule - 1) / granule * granule;
  r.pair_rows = fd ? (int64_t)r.Bp : 2 * (int64_t)r.Bp;
  r.M = fd ? (int64_t)(N + 1) * r.Bp : (int64_t)N * r.pair_rows;
  return r;
}

inline RowMap row_map(const Rows& r) { return RowMap{r.Bp, r.pair_rows, r.fd, r.N}; }

// The pass of row r: its probe (relative index; the clean pass reports
// probe N - 1, whose values it multiplies by 0), the sign of eps (+1, -1, or
// 0 for the clean pass) and its sequence b.
struct PassOf {
  int probe;
  int sign;
  int b;
};
__host__ __device__ inline PassOf pass_of(const RowMap& m, int64_t r) {
  const int64_t p = r / m.pair_rows;
  const int loc = (int)(r - p * m.pair_rows);
  if (m.fd) return PassOf{p < m.N ? (int)p : m.N - 1, p < m.N ? 1 : 0, loc};
  return loc >= m.Bp ? PassOf{(int)p, -1, loc - m.Bp} : PassOf{(int)p, 1, loc};
}

// Time steps whose top-layer states are kept for one batched output-head pass.
constexpr int kTimeChunk = 16;

// Output-head vocabulary tile (columns per workgroup): 256 on the bf16 path,
// 128 on the fp32 path.
constexpr int kVocabTile = 128;
// Columns per workgroup of the bf16 products (gate columns or vocabulary
// rows); its rows are 65536 / kVocabTileWide. (128 x 512 workgroups, which
// load each weight fragment once, measured slower than 256 x 256.)
constexpr int kVocabTileWide = 256;
inline int vocab_tile(const zo_config& c) { return c.wdtype == ZO_WBF16 ? kVocabTileWide : kVocabTile; }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Probe cache (normal probes only): the 2N forward passes read the probe
// terms of every weight matrix (W_ih, W_hh of each layer and W_out) at every
// timestep and row tile, while each value is the same for the whole call.
// With a large enough workspace the call first writes, once, the values the
// kernels would otherwise regenerate: eps z in fp32 (fp32 weights) or
// fp16(eps z) (bf16 weights), for probes i0 .. i0+N-1. Layout: probe n's
// block of P_g values (the matrices in theta order) at n * P_g; each matrix
// row-major like the matrix itself (fp32 weights) or fragment-packed like the
// fp16 weight copy (bf16 weights, zo_pack.hpp). Sign probes are cheap to
// regenerate and are never cached. The same map places the matrices of the
// bf16 path's fp16 weight copy; there the head matrix is padded with zero
// rows to a whole number of 256-wide vocabulary tiles.
struct ZCacheMap {
  uint64_t pg;              // values per probe: the matrices' total size
  uint64_t ih[kMaxLayers];  // offsets of each matrix inside a probe's block
  uint64_t hh[kMaxLayers];
  uint64_t out;
  uint64_t out_rows;        // rows of the head matrix as stored (V, or padded on the bf16 path)
};

inline ZCacheMap make_zcache_map(const zo_config& c) {
  ZCacheMap m{};
  const uint64_t E = (uint64_t)c.embed, H = (uint64_t)c.hidden, V = (uint64_t)c.vocab;
  uint64_t p = 0;
  for (int l = 0; l < c.n_layers; ++l) {
    m.ih[l] = p;
    p += 4 * H * (l == 0 ? E : H);
    m.hh[l] = p;
    p += 4 * H * H;
  }
  m.out = p;
  m.out_rows = c.wdtype == ZO_WBF16 ? (V + kVocabTileWide - 1) / kVocabTileWide * kVocabTileWide : V;
  p += m.out_rows * H;
  m.pg = p;
  return m;
}

inline bool probe_cache_kind(const zo_config& c) { return c.probe == ZO_GAUSSIAN; }

// Bit-packed sign-probe cache (bf16 weights with sign probes): the sign words
// of probes i0 .. i0+N-1 over the whole parameter vector, written once per call
// (one Philox block per 128 parameters and probe) and read by the forward
// kernels in place of regenerating them in every K tile: probe n's word w, the
// signs of parameters 32 w .. 32 w + 31 (a set bit for z = +1), at
// n * bit_words(P) + w, unshuffled: parameter 32 w + 2 i at bit i and
// 32 w + 2 i + 1 at bit 16 + i (sign_word_unshuffle of the generator's word),
// the order in which the bf16 products turn a pair of flags into a packed
// fp16 pair with one shift. The update can read the same words
// (zo_update_cached) instead of regenerating them.
inline bool bit_cache_kind(const zo_config& c) { return c.probe == ZO_RADEMACHER && c.wdtype == ZO_WBF16; }
__host__ __device__ inline uint64_t bit_words(uint64_t P) { return (P + 127) / 128 * 4; }

// A word of 32 flags with the even-indexed flags moved to bits 0..15 and the
// odd-indexed ones to bits 16..31, each half in order (four delta swaps);
// sign_word_shuffle is its inverse (the same swaps in reverse order).
__host__ __device__ inline uint32_t sign_word_unshuffle(uint32_t x) {
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
__host__ __device__ inline uint32_t sign_word_shuffle(uint32_t x) {
  uint32_t t;
  t = (x ^ (x >> 8)) & 0x0000FF00u;
  x = x ^ t ^ (t << 8);
  t = (x ^ (x >> 4)) & 0x00F000F0u;
  x = x ^ t ^ (t << 4);
  t = (x ^ (x >> 2)) & 0x0C0C0C0Cu;
  x = x ^ t ^ (t << 2);
  t = (x ^ (x >> 1)) & 0x22222222u;
  x = x ^ t ^ (t << 1);
  return x;
}

// Kernel variants for normal probes read from the probe cache (fp16(eps z)
// as a second operand stream; or, bf16 weights with fused products, the
// perturbed weights fp16(w +- fp16(eps z)) as the B operand itself) and for
// sign probes read from the sign-probe cache (next to the probe kinds
// ZO_RADEMACHER and ZO_GAUSSIAN, which regenerate them).
constexpr int kGaussCached = 2;
constexpr int kSignsCached = 3;
constexpr int kGaussPerturbed = 4;

// Workspace plan (byte offsets from the workspace base, 256-aligned).
struct WsPlan {
  size_t x0;         // f32 [M][E]         perturbed embeddings of one timestep
  size_t hbuf;       // f32 [L-1][2][M][H] double-buffered states of the lower layers
  size_t hist;       // f32 [T][M][H]      top-layer states of the current time chunk
  size_t cbuf;       // f32 [L][M][H]      cell states
  size_t zb;         // f32 [L][N][4H]     eps * z of the gate biases, per probe
  size_t zbo;        // f32 [N][V]         eps * z of the head bias, per probe
  size_t pmax;       // f32 [nvt][T*M]     per vocabulary tile: running max
  size_t psum;       // f32 [nvt][T*M]     per vocabulary tile: sum of exp(y - max)
  size_t ptgt;       // f32 [T*M]          target logit
  size_t row_loss;   // f64 [M]            masked loss sum of each row
  size_t w16;        // f16 [P_g]          bf16 weights: the product matrices in fp16 (ZCacheMap layout)
  size_t min_total;  // bytes without the probe cache
  size_t zcache;     // probe cache (normal probes; see ZCacheMap): fp32 weights [N][P_g] eps z;
                     // bf16 weights [N][2][P_g] fp16: probe n's perturbed weights
                     // fp16(w + fp16(eps z)) and fp16(w - fp16(eps z)) (fused products), or
                     // fp16(eps z) in the first N P_g values (two-stream products)
  size_t bits;       // sign-probe cache [N][bit_words(P)] u32 (bf16 weights with sign probes)
  size_t total;      // bytes with the probe cache
  int nvt;           // vocabulary tiles
  int T;             // time chunk
};

inline WsPlan plan_workspace(const zo_config& c, const Rows& r, int32_t C) {
  WsPlan w{};
  const size_t M = (size_t)r.M, E = (size_t)c.embed, H = (size_t)c.hidden, V = (size_t)c.vocab;
  const size_t L = (size_t)c.n_layers;
  const size_t el = c.wdtype == ZO_WBF16 ? 2 : 4;  // activation operand element size
  w.T = C < kTimeChunk ? C : kTimeChunk;
  const size_t vt = (size_t)vocab_tile(c);
  w.nvt = (int)((V + vt - 1) / vt);
  size_t p = 0;
  auto take = [&](size_t bytes) {
    size_t o = p;
    p = align_up(p + bytes, 256);
    return o;
  };
  // perturbed embeddings: one timestep (bf16 path), a time chunk (fp32 path)
  w.x0 = take((c.wdtype == ZO_WBF16 ? 1 : (size_t)w.T) * M * E * el);
  w.hbuf = take((L - 1) * 2 * M * H * el);
  w.hist = take((size_t)w.T * M * H * el);
  w.cbuf = take(L * M * H * 4);
  w.zb = take(L * (size_t)r.N * 4 * H * 4);
  w.zbo = take((size_t)r.N * V * 4);
  w.pmax = take((size_t)w.nvt * w.T * M * 4);
  w.psum = take((size_t)w.nvt * w.T * M * 4);
  w.ptgt = take((size_t)w.T * M * 4);
  w.row_loss = take(M * 8);
  w.w16 = p;
  if (c.wdtype == ZO_WBF16) take((size_t)make_zcache_map(c).pg * 2);
  w.min_total = p;
  w.zcache = p;
  if (probe_cache_kind(c)) take((size_t)r.N * make_zcache_map(c).pg * (c.wdtype == ZO_WBF16 ? 2 * 2 : 4));
  w.bits = p;
  if (bit_cache_kind(c)) take((size_t)r.N * bit_words(make_layout(c).total) * 4);
  w.total = p;
  return w;
}

}  // namespace zo
