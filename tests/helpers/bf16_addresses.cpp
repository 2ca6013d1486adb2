// Host replay of the bf16 kernels' operand addressing (zo_pack.hpp, the same
// functions the kernels call): for one model shape and batch, every
// workgroup, wave, lane, copy and k step of the gate and head launches, it
// checks that
// each activation copy, packed B-fragment load, sign-probe cache load, cell
// state copy and head bias copy lies
// inside the buffer resource it is issued against (and inside the tensor that
// resource covers), that every offset fits in 32 bits, that the copies fill
// each LDS row and slot of a tile exactly once with the chunk the swizzle
// puts there, that each wave loads the weight fragments of its own columns
// and k, and that the packed layout and the gate column order are
// bijections. Usage: bf16_addresses L V E H N B fd -> prints "ok" or the
// first violation (exit status 1).
#include <cstdint>
#include <cstdio>
#include <algorithm>
#include <cstdlib>
#include <vector>

#include "../../paper_2505_17852_amd/csrc/zo_common.hpp"
#include "../../paper_2505_17852_amd/csrc/zo_pack.hpp"

using namespace zo;

static int fails = 0;
#define CHECK(cond, ...)                                    \
  do {                                                      \
    if (!(cond)) {                                          \
      if (fails++ < 10) {                                   \
        std::printf("violation: " __VA_ARGS__);             \
        std::printf("\n");                                  \
      }                                                     \
    }                                                       \
  } while (0)

constexpr int TN = kVocabTileWide, TM = 65536 / TN, TK = 64;
// the loop's copy roles: 8 waves, TM / 64 activation copies each per K tile
struct Geometry {
  int nwaves, acopies;
};
constexpr Geometry kGeo8{8, TM * 128 / 1024 / 8};

// the activation copies of one workgroup tile against a resource of TM rows of lda
static void check_copies(int64_t lda, int64_t K, const char* what, Geometry g) {
  const uint64_t records = (uint64_t)TM * lda * 2;
  CHECK(records < (1ull << 31), "%s: resource of %llu bytes", what, (unsigned long long)records);
  std::vector<int> seen(TM * 8, 0);
  for (int q = 0; q < g.acopies; ++q)
    for (int w = 0; w < g.nwaves; ++w)
      for (int lane = 0; lane < 64; ++lane) {
        const int row = act_row_of_copy(q, w, lane, g.nwaves);
        CHECK(row >= 0 && row < TM, "%s: copy row %d", what, row);
        const int lds = (q * g.nwaves + w) * 1024 + 16 * lane;  // LDS byte this lane writes
        CHECK(lds == row * 128 + 16 * (lane % 8), "%s: LDS byte %d for row %d", what, lds, row);
        seen[row * 8 + lane % 8] += 1;
        const uint64_t off0 = act_copy_offset(q, w, lane, g.nwaves, lda);
        const int chunk = (int)((off0 - (uint64_t)row * lda * 2) / 16);
        CHECK(chunk == ((lane % 8) ^ act_swizzle(row)), "%s: chunk %d in slot %d of row %d", what, chunk,
              lane % 8, row);
        for (int64_t k0 : {(int64_t)0, K - TK}) {
          const uint64_t off = off0 + 2 * (uint64_t)k0;
          CHECK(off + 16 <= records && off < (1ull << 32), "%s: copy offset %llu of %llu (k0 %lld)", what,
                (unsigned long long)off, (unsigned long long)records, (long long)k0);
        }
      }
  for (int i = 0; i < TM * 8; ++i) CHECK(seen[i] == 1, "%s: LDS row %d slot %d written %d times", what, i / 8, i % 8, seen[i]);
}

// the packed B loads of column block nb (TN / 64 wave columns wn of 2 tiles
// nt, every lane and k step): each wave's tiles are its own columns
static void check_b_loads(int64_t nb, int64_t cols, int64_t K, const char* what) {
  const uint64_t records = (uint64_t)cols * K * 2;
  CHECK(records < (1ull << 31), "%s: packed matrix of %llu bytes", what, (unsigned long long)records);
  const int64_t KS = K / kPackKStep;
  for (int wn = 0; wn < TN / 64; ++wn)
    for (int nt = 0; nt < 2; ++nt)
      for (int lane = 0; lane < 64; ++lane)
        for (int64_t ks : {(int64_t)0, KS - 1}) {
          const int64_t cb = packed_block_of(nb, wn, nt, TN);
          CHECK(cb == (TN * nb + 64 * wn + 32 * nt) / 32, "%s: block of wave column %d tile %d", what, wn, nt);
          const uint64_t off = packed_lane_offset(cb, K, lane) + packed_step_offset(ks);
          // no 32-bit wrap: an offset past the resource reads zeros, one that
          // wrapped would read real data
          CHECK(off < (1ull << 32), "%s: B offset %llu wraps", what, (unsigned long long)off);
          if (32 * cb >= cols) {
            // a column block past the matrix (a last workgroup it does not fill)
            CHECK(off >= records, "%s: block %lld past the matrix reads inside it", what, (long long)cb);
            continue;
          }
          CHECK(off + 16 <= records, "%s: B offset %llu of %llu", what, (unsigned long long)off,
                (unsigned long long)records);
          // the chunk read is the fragment piece of column 32 cb + lr at k 16 ks + 8 lg
          const PackedChunk pc = packed_chunk(off / 16, K);
          CHECK(pc.col == 32 * cb + (lane & 31) && pc.k == 16 * ks + 8 * (lane >> 5), "%s: packed chunk", what);
        }
}

// the gate's cell-state copies of column block nb (hidden units u0 = 64 nb
// .. + 63) against the resource of the tile's 256 rows of H fp32: inside it,
// and each LDS row (256 bytes) and 16-byte slot written once, with the units
// it must hold
static void check_cell_copies(int64_t nb, int64_t H) {
  const uint64_t records = (uint64_t)TM * (uint64_t)H * 4u;
  CHECK(records < (1ull << 31), "cell tile resource of %llu bytes", (unsigned long long)records);
  const int64_t u0 = (TN / 4) * nb;
  CHECK(u0 + TN / 4 <= H, "cell tile units %lld.. of %lld", (long long)u0, (long long)H);
  std::vector<int> seen(TM * 16, 0);
  for (int cp = 0; cp < 64; ++cp)
    for (int lane = 0; lane < 64; ++lane) {
      const int row = cell_row_of_copy(cp, lane);
      const uint64_t off = cell_copy_offset(cp, lane, H, u0);
      CHECK(row >= 0 && row < TM, "cell copy row %d", row);
      CHECK(off + 16 <= records, "cell copy offset %llu of %llu", (unsigned long long)off, (unsigned long long)records);
      CHECK(off == ((uint64_t)row * H + u0 + 4 * (lane & 15)) * 4, "cell copy %d lane %d offset", cp, lane);
      const int lds = 1024 * cp + 16 * lane;  // LDS byte this lane writes
      CHECK(lds == row * 256 + 16 * (lane & 15), "cell copy %d lane %d LDS byte %d", cp, lane, lds);
      if (row >= 0 && row < TM) seen[row * 16 + (lane & 15)] += 1;
    }
  for (int i = 0; i < TM * 16; ++i) CHECK(seen[i] == 1, "cell LDS row %d slot %d written %d times", i / 16, i % 16, seen[i]);
}

// the head's bias copies of vocabulary tile vt: the probe values (one column
// per lane, past V reading zeros) and the bias words from the 4-byte boundary
// (lead 0 or 2 bytes), every column of the tile inside V covered and inside
// the resource, the epilogue's 2-byte reads inside the 1 KB of words
static void check_head_bias(int64_t vt, int64_t V) {
  const int64_t v0 = vt * TN;
  for (int q = 0; q < 4; ++q)
    for (int lane = 0; lane < 64; ++lane) {
      const uint64_t off = head_probe_offset(v0, q, lane);
      const int64_t col = v0 + 64 * q + lane;
      CHECK(off == 4 * (uint64_t)col && off < (1ull << 32), "head probe copy offset %llu", (unsigned long long)off);
      CHECK((col < V) == (off + 4 <= 4 * (uint64_t)V), "head probe column %lld against V", (long long)col);
      CHECK(256 * q + 4 * lane < 1024, "head probe LDS byte");
    }
  CHECK(4 * (uint64_t)V < (1ull << 31), "head probe resource");
  for (uint32_t lead : {0u, 2u}) {
    const uint64_t bytes = head_bias_bytes(lead, V);
    CHECK(bytes >= lead + 2 * (uint64_t)V && bytes < lead + 2 * (uint64_t)V + 4 && bytes % 4 == 0 && bytes < (1ull << 31),
          "head bias resource of %llu bytes (lead %u)", (unsigned long long)bytes, lead);
    for (int64_t c = v0; c < std::min<int64_t>(V, v0 + TN); ++c) {
      const uint64_t at = lead + 2 * (uint64_t)c;  // byte of column c from the boundary
      const uint64_t rel = lead + 2 * (uint64_t)(c - v0);  // and in the tile's words
      CHECK(rel + 2 <= 1024, "head bias LDS read of column %lld", (long long)c);
      const int d = (int)(rel / 4);  // the word holding it
      const uint64_t woff = head_bias_word_offset(v0, d);
      CHECK(woff <= at && at + 2 <= woff + 4 && woff + 4 <= bytes && d < 256,
            "head bias column %lld (lead %u): word %d at %llu of %llu", (long long)c, lead, d,
            (unsigned long long)woff, (unsigned long long)bytes);
    }
  }
}

// the sign-probe cache loads: the two words (32 k each; one 8-byte load by
// one thread of the column's pair) of K tile k0 of the parameter row n of a matrix at zoff (row
// stride ldw), inside the bit_words(P) words of one probe
static void check_words(uint64_t zoff, int64_t n, int64_t ldw, int64_t K, uint64_t P, const char* what) {
  const uint64_t bytes = 4 * (4 * ((P + 127) / 128));
  for (int64_t k0 : {(int64_t)0, K - TK}) {
    // one 8-byte load per thread and tile: both words, 8-byte aligned
    const uint64_t jt = zoff + (uint64_t)n * (uint64_t)ldw + (uint64_t)k0;
    CHECK(jt % 64 == 0 && sign_word_offset(jt) % 8 == 0, "%s: sign words of parameter %llu not 8-byte aligned", what,
          (unsigned long long)jt);
    for (int i = 0; i < 2; ++i) {
      const uint64_t j = zoff + (uint64_t)n * (uint64_t)ldw + (uint64_t)k0 + 32u * (uint64_t)i;
      const uint64_t off = sign_word_offset(j);
      CHECK(j < P && off + 4 <= bytes && off == (j / 32) * 4, "%s: sign word of parameter %llu at %llu of %llu",
            what, (unsigned long long)j, (unsigned long long)off, (unsigned long long)bytes);
    }
  }
}

// the sign-probe cache's word order: sign_word_unshuffle puts flag 2 i at
// bit i and flag 2 i + 1 at bit 16 + i, and sign_word_shuffle undoes it
static void check_word_order() {
  uint64_t s = 0x9E3779B97F4A7C15ull;
  for (int r = 0; r < 4096; ++r) {
    s = s * 6364136223846793005ull + 1442695040888963407ull;
    const uint32_t x = r < 32 ? (1u << r) : (uint32_t)(s >> 32);
    uint32_t want = 0;
    for (int b = 0; b < 32; ++b)
      if (x >> b & 1u) want |= 1u << ((b >> 1) + 16 * (b & 1));
    CHECK(sign_word_unshuffle(x) == want, "unshuffle of %08x", x);
    CHECK(sign_word_shuffle(sign_word_unshuffle(x)) == x, "shuffle does not undo unshuffle of %08x", x);
  }
}

int main(int argc, char** argv) {
  if (argc != 8) {
    std::printf("usage: bf16_addresses L V E H N B fd\n");
    return 2;
  }
  const int L = std::atoi(argv[1]);
  const int64_t V = std::atoll(argv[2]), E = std::atoll(argv[3]), H = std::atoll(argv[4]);
  const int64_t N = std::atoll(argv[5]), B = std::atoll(argv[6]);
  const bool fd = std::atoi(argv[7]) != 0;
  const int64_t gran = fd ? 256 : 128;
  const int64_t Bp = (B + gran - 1) / gran * gran;
  const int64_t M = fd ? (N + 1) * Bp : 2 * N * Bp;
  check_word_order();
  const int64_t nvt = (V + TN - 1) / TN;
  const int64_t out_rows = nvt * TN;
  CHECK(M % TM == 0, "rows %lld not a whole number of tiles", (long long)M);
  // the gate column order is a permutation of the 4H weight rows
  {
    std::vector<int> hit(4 * H, 0);
    for (int64_t rho = 0; rho < 4 * H; ++rho) {
      const int64_t r = gate_row_of_column(rho, H);
      CHECK(r >= 0 && r < 4 * H, "gate column %lld -> row %lld", (long long)rho, (long long)r);
      if (r >= 0 && r < 4 * H) hit[r]++;
    }
    for (int64_t r = 0; r < 4 * H; ++r) CHECK(hit[r] == 1, "gate row %lld hit %d times", (long long)r, hit[r]);
  }
  // the packed layout: chunk u <-> (column, k) is a bijection on one matrix
  for (int64_t K : {E, H}) {
    const int64_t cols = 4 * H;
    std::vector<uint8_t> hit((size_t)(cols * K / 8), 0);
    for (uint64_t u = 0; u < (uint64_t)(cols * K / 8); ++u) {
      const PackedChunk pc = packed_chunk(u, K);
      CHECK(pc.col >= 0 && pc.col < cols && pc.k >= 0 && pc.k + 8 <= K && pc.k % 8 == 0, "packed chunk %llu",
            (unsigned long long)u);
      if (pc.col >= 0 && pc.col < cols && pc.k >= 0 && pc.k + 8 <= K) hit[(size_t)(pc.col * (K / 8) + pc.k / 8)]++;
    }
    for (size_t i = 0; i < hit.size(); ++i) CHECK(hit[i] == 1, "packed (col, k) %zu hit %d times", i, hit[i]);
  }
  // the flat parameter layout: EMB, per layer W_ih, W_hh, b, then W_out, b_out
  std::vector<uint64_t> off_ih(L), off_hh(L);
  uint64_t P = (uint64_t)V * E;
  for (int l = 0; l < L; ++l) {
    const int64_t El = l == 0 ? E : H;
    off_ih[l] = P;
    P += 4 * H * El;
    off_hh[l] = P;
    P += 4 * H * H;
    P += 4 * H;
  }
  const uint64_t off_out = P;
  P += (uint64_t)V * H + V;
  // gate launches: every layer's two segments, every workgroup (TN / 4
  // hidden units each; the last may be partly past the 4H columns)
  const int64_t nm = M / TM, nn = (4 * H + TN - 1) / TN;
  for (int l = 0; l < L; ++l) {
    const int64_t El = l == 0 ? E : H;
    check_copies(El, El, "gate x", kGeo8);
    check_copies(H, H, "gate h", kGeo8);
    for (int64_t mb = 0; mb < nm; ++mb) CHECK((mb + 1) * TM <= M, "gate row block %lld", (long long)mb);
    for (int64_t nb = 0; nb < nn; ++nb) {
      if (l == 0) check_cell_copies(nb, H);
      check_b_loads(nb, 4 * H, El, "gate W_ih");
      check_b_loads(nb, 4 * H, H, "gate W_hh");
      // the sign words of every workgroup column (the gate column order)
      for (int rho = 0; rho < TN; ++rho) {
        const int c = rho & 63;
        const int64_t n = std::min<int64_t>((c >> 4) * H + TN / 4 * nb + 16 * (rho >> 6) + (c & 15), 4 * H - 1);
        if (TN * nb + rho < 4 * H)
          CHECK(n == gate_row_of_column(TN * nb + rho, H), "gate sign-word row of column %d", rho);
        check_words(off_ih[l], n, El, El, P, "gate W_ih");
        check_words(off_hh[l], n, H, H, P, "gate W_hh");
      }
    }
  }
  // head launches: Tc timesteps of M rows (Tc <= 16), every vocabulary tile
  for (int64_t Tc : {(int64_t)1, (int64_t)16}) {
    const int64_t rows = Tc * M;
    CHECK(rows % TM == 0, "head rows");
    check_copies(H, H, "head h", kGeo8);
  }
  for (int64_t vt = 0; vt < nvt; ++vt) {
    check_b_loads(vt, out_rows, H, "head W_out");
    check_head_bias(vt, V);
    for (int rho = 0; rho < TN; ++rho) {
      const int64_t n = std::min<int64_t>(TN * vt + rho, V - 1);
      check_words(off_out, n, H, H, P, "head W_out");
    }
  }
  if (fails) {
    std::printf("%d violations\n", fails);
    return 1;
  }
  std::printf("ok\n");
  return 0;
}
