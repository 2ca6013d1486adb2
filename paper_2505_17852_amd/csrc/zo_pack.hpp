// Address arithmetic of the bf16 path's matrix operands, shared by the
// kernels and the host-side bounds checks (every function here is plain
// integer arithmetic, callable on the host and on the device).
//
// Fragment-packed fp16 matrices. The products of the bf16 path read their B
// operand (the fp16 copy of a weight matrix, and the cached fp16(eps z) of
// normal probes) straight from global memory into registers, one 16-byte
// piece per lane. So that one wave instruction reads 1 KB of consecutive
// memory, the call writes those matrices in the order the v_mfma_f32_32x32x16
// fragments are consumed: the matrix's columns, in the kernels' column
// order, are cut into blocks of 32 and its K dimension into steps of 16;
// block (cb, ks) is 1 KB at ((cb * KS + ks) * 64) * 8 values, and its lane
// L = lr + 32 lg holds the 8 values (column 32 cb + lr, k = 16 ks + 8 lg ..
// 16 ks + 8 lg + 7).
//
// Column order: a gate matrix (4H weight rows, K = E_l or H) takes column
// rho = 64 ug + c to weight row (c / 16) H + 16 ug + c % 16, i.e. gate c / 16
// (i, f, g, o) of hidden unit 16 ug + c % 16, so that one 64-column wave tile
// holds all four gates of 16 units. The head (V rows, K = H) takes column rho
// to vocabulary row rho, padded with zero rows up to out_rows (a whole number
// of 256-wide vocabulary tiles).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zo {

constexpr int kPackBlockCols = 32;  // columns per packed block
constexpr int kPackKStep = 16;      // k per packed block
constexpr int kPackBlockBytes = 1024;

// Weight row of gate-matrix column rho (H hidden units).
__host__ __device__ inline int64_t gate_row_of_column(int64_t rho, int64_t H) {
  const int64_t c = rho & 63, ug = rho >> 6;
  return (c >> 4) * H + 16 * ug + (c & 15);
}

// Source of 16-byte chunk u of a packed matrix with K columns of k: the
// column (in the kernels' order) and the first k of its 8 values.
struct PackedChunk {
  int64_t col;
  int64_t k;
};
__host__ __device__ inline PackedChunk packed_chunk(uint64_t u, int64_t K) {
  const int64_t KS = K / kPackKStep;
  const int64_t lane = (int64_t)(u & 63u), rest = (int64_t)(u >> 6);
  const int64_t ks = rest % KS, cb = rest / KS;
  return PackedChunk{kPackBlockCols * cb + (lane & 31), kPackKStep * ks + 8 * (lane >> 5)};
}

// Byte offset, inside a packed matrix with K columns of k, of the 16 bytes
// lane `lane` reads for the fragment of column block cb at k step ks.
__host__ __device__ inline uint64_t packed_lane_offset(int64_t cb, int64_t K, int lane) {
  return ((uint64_t)cb * (uint64_t)(K / kPackKStep) * 64u + (uint64_t)lane) * 16u;
}
__host__ __device__ inline uint32_t packed_step_offset(int64_t ks) { return (uint32_t)ks * kPackBlockBytes; }

// Packed column block of column tile nt (of 2) of wave column wn (64
// columns each) in workgroup column block nb of tn columns: the same for the
// gate (nb = block of tn / 4 hidden units) and the head (nb = vocabulary tile
// of tn).
__host__ __device__ inline int64_t packed_block_of(int64_t nb, int wn, int nt, int tn) {
  return (int64_t)(tn / kPackBlockCols) * nb + 2 * wn + nt;
}

// Activation tile copies (global -> LDS, 1 KB per wave instruction): copy q
// of wave w fills LDS rows 8 (q NW + w) .. + 7 of the 256-row tile (128-byte
// rows of 64 fp16 k, 16-byte chunks XOR-swizzled by row so that the 16 rows
// of one fragment read cover all banks). Lane L writes row 8 (q NW + w) +
// L / 8, slot L % 8, which must hold chunk (L % 8) ^ swz(row); this is the
// byte offset of that chunk from the tile's first row at k0 = 0 (lda: the
// row stride in elements); the K tile adds 2 k0 bytes.
__host__ __device__ inline int act_row_of_copy(int q, int w, int lane, int nwaves) {
  return 8 * (q * nwaves + w) + lane / 8;
}
__host__ __device__ inline int act_swizzle(int row) { return (row >> 1) & 7; }
__host__ __device__ inline uint64_t act_copy_offset(int q, int w, int lane, int nwaves, int64_t lda) {
  const int r = act_row_of_copy(q, w, lane, nwaves);
  return (uint64_t)r * (uint64_t)lda * 2u + 16u * (uint64_t)((lane % 8) ^ act_swizzle(r));
}

// Byte offset, in the sign-probe cache of one probe, of the word holding the
// sign of parameter j (32 per word).
__host__ __device__ inline uint32_t sign_word_offset(uint64_t j) { return (uint32_t)(j >> 5) * 4u; }

// The gate's cell-state tile (the workgroup's 256 rows x 64 hidden units,
// fp32, row stride H in global memory, 256 bytes per row in LDS): 64 copies
// of 1 KB, 4 rows each; lane L of copy cp writes row 4 cp + L / 16, units
// u0 + 4 (L % 16) .. + 3, at LDS byte 1024 cp + 16 L. Byte offset from the
// tile's first row:
__host__ __device__ inline int cell_row_of_copy(int cp, int lane) { return 4 * cp + (lane >> 4); }
__host__ __device__ inline uint32_t cell_copy_offset(int cp, int lane, int64_t H, int64_t u0) {
  return ((uint32_t)cell_row_of_copy(cp, lane) * (uint32_t)H + (uint32_t)u0) * 4u + 16u * (uint32_t)(lane & 15);
}

// The head's bias values of vocabulary tile v0 .. v0 + 255: the bias probe
// values (fp32) one column per lane, lane L of copy q < 4 reading column
// v0 + 64 q + L; the bf16 bias as 4-byte words from the 4-byte boundary at
// or below its first element (lead: 0 or 2 bytes before it), word d < 256 of
// the tile at this offset from that boundary. Column c's bias is then at
// byte lead + 2 (c - v0) of the tile's words.
__host__ __device__ inline uint32_t head_probe_offset(int64_t v0, int q, int lane) {
  return 4u * (uint32_t)(v0 + 64 * q + lane);
}
__host__ __device__ inline uint32_t head_bias_word_offset(int64_t v0, int d) {
  return 2u * (uint32_t)v0 + 4u * (uint32_t)d;
}
__host__ __device__ inline uint32_t head_bias_bytes(uint32_t lead, int64_t V) {
  return (lead + 2u * (uint32_t)V + 3u) & ~3u;
}

}  // namespace zo
