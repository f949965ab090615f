// Host-side model check of the LDS tile layouts used by the MFMA kernels.
//
// The direct global->LDS loads (TileFetch, SFetch) are replayed on the CPU to
// fill a model tile with the logical (row, column) index of every bf16 slot;
// then every lane offset the kernels read through (tile_offsets/tile_row16/
// tile_col8 and s_offsets/s_row16/s_col8) must return the elements the MFMA
// operand layout asks for, and every read must be bank-conflict free under the
// gfx950 LDS model: 64 banks of 4 bytes, 16-byte reads served 16 lanes per
// phase, 8-byte transposing reads 32 lanes per phase.  The transposing read
// delivers, in each 16-lane group, to lane i the column i of the four rows
// named by source lanes 4j + i/4 (element i % 4 of each).
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "mfma_common.h"
#include "sparse_common.h"

static int failures = 0;
#define CHECK(cond, ...)                         \
  do {                                           \
    if (!(cond)) {                               \
      if (failures < 20) {                       \
        printf("FAIL %s:%d: ", __FILE__, __LINE__); \
        printf(__VA_ARGS__);                     \
        printf("\n");                            \
      }                                          \
      ++failures;                                \
    }                                            \
  } while (0)

// distinct 16-byte bank groups within each 16-lane phase
static void check_b128_phases(const int* off, const char* what) {
  for (int ph = 0; ph < 4; ++ph) {
    int seen = 0;
    for (int l = 16 * ph; l < 16 * ph + 16; ++l) {
      const int g = (off[l] & 255) >> 4;
      CHECK(!(seen & (1 << g)), "%s: bank conflict in 16-byte read, phase %d lane %d", what, ph, l);
      seen |= 1 << g;
    }
  }
}

// distinct 16-byte bank groups within each eight consecutive lanes
static void check_b128_octets(const int* off, const char* what) {
  for (int oc = 0; oc < 8; ++oc) {
    int seen = 0;
    for (int l = 8 * oc; l < 8 * oc + 8; ++l) {
      const int g = (off[l] & 255) >> 4;
      CHECK(!(seen & (1 << g)), "%s: two lanes of octet %d on one bank group, lane %d", what, oc, l);
      seen |= 1 << g;
    }
  }
}

// distinct 8-byte bank pairs within each 32-lane phase
static void check_b64_phases(const int* off, const char* what) {
  for (int ph = 0; ph < 2; ++ph) {
    unsigned seen = 0;
    for (int l = 32 * ph; l < 32 * ph + 32; ++l) {
      const int g = (off[l] & 255) >> 3;
      CHECK(!(seen & (1u << g)), "%s: bank conflict in transposing read, phase %d lane %d", what, ph, l);
      seen |= 1u << g;
    }
  }
}

// Transposing read: output element j of lane l from the model tile.
static int tr_elem(const std::vector<int>& tag, const int* src_off, int l, int j) {
  const int g = l >> 4, i = l & 15;
  const int src = 16 * g + 4 * j + (i >> 2);
  return tag[src_off[src] / 2 + (i & 3)];
}

static void dense() {
  using namespace ls;
  const int cols = kTileRow / 2;
  std::vector<int> tag(kTileBytes / 2, -1);
  for (int w = 0; w < 4; ++w)
    for (int lane = 0; lane < 64; ++lane) {
      TileFetch f;
      f.init(nullptr, cols, lane, w);
      for (int i = 0; i < 4; ++i) {
        const int dst = f.lds_row[i] * kTileRow + 16 * lane;   // 1 KiB per instruction, linear
        for (int e = 0; e < 8; ++e) {
          CHECK(tag[dst / 2 + e] == -1, "dense fetch writes slot %d twice", dst / 2 + e);
          tag[dst / 2 + e] = f.lane_row[i] * cols + (int)(f.lane_off[i] / 2) + e;
        }
      }
    }
  for (int v : tag) CHECK(v >= 0, "dense fetch leaves a slot unwritten");
  // eight waves with two instructions each write the same tile image
  {
    std::vector<int> tag8(kTileBytes / 2, -1);
    for (int w = 0; w < 8; ++w)
      for (int lane = 0; lane < 64; ++lane) {
        TileFetchN<2> f;
        f.init(nullptr, cols, lane, w);
        for (int i = 0; i < 2; ++i) {
          const int dst = f.lds_row[i] * kTileRow + 16 * lane;
          for (int e = 0; e < 8; ++e) {
            CHECK(tag8[dst / 2 + e] == -1, "8-wave fetch writes slot %d twice", dst / 2 + e);
            tag8[dst / 2 + e] = f.lane_row[i] * cols + (int)(f.lane_off[i] / 2) + e;
          }
        }
      }
    CHECK(tag8 == tag, "8-wave fetch lays the tile out differently");
  }

  TileOffsets o[64];
  for (int l = 0; l < 64; ++l) o[l] = tile_offsets(l);
  // the one-register form gives the table's offsets
  for (int l = 0; l < 64; ++l) {
    const TileBase b = tile_base(l);
    for (int ks = 0; ks < 16; ++ks)
      CHECK(tile_row_offset(b, ks) == o[l].row_off[ks & 7] + 256 * (ks >> 3),
            "compact row offset lane=%d ks=%d", l, ks);
    for (int db = 0; db < 8; ++db)
      for (int r = 0; r < 32; r += 8)
        CHECK(tile_col_offset(b, db, r) ==
                  256 * (db >> 2) + o[l].col_off[(r >> 3) & 1][db & 3] + r * kTileRow,
              "compact column offset lane=%d db=%d r=%d", l, db, r);
  }
  for (int ks = 0; ks < 16; ++ks) {
    int off[64];
    for (int l = 0; l < 64; ++l) {
      off[l] = o[l].row_off[ks & 7] + 256 * (ks >> 3);
      const int row = l & 31, c0 = 16 * ks + 8 * (l >> 5);
      for (int e = 0; e < 8; ++e)
        CHECK(tag[off[l] / 2 + e] == row * cols + c0 + e, "dense row operand ks=%d lane=%d e=%d", ks, l, e);
    }
    check_b128_phases(off, "dense row operand");
  }
  for (int db = 0; db < 8; ++db)
    for (int r = 0; r < 32; r += 8) {
      int off[64];
      for (int l = 0; l < 64; ++l) off[l] = 256 * (db >> 2) + o[l].col_off[(r >> 3) & 1][db & 3] + r * kTileRow;
      for (int l = 0; l < 64; ++l)
        for (int j = 0; j < 4; ++j) {
          const int want = (r + 4 * (l >> 5) + j) * cols + 32 * db + (l & 31);
          CHECK(tr_elem(tag, off, l, j) == want, "dense transposed operand db=%d r=%d lane=%d j=%d", db, r, l, j);
        }
      check_b64_phases(off, "dense transposed operand");
    }
}

static void sparse() {
  using namespace ls::sparse;
  const int cols = kRow / 2;
  std::vector<int> tag(kTile / 2, -1);
  for (int w = 0; w < 4; ++w)
    for (int lane = 0; lane < 64; ++lane) {
      SFetch f;
      f.init(lane, w);
      for (int i = 0; i < 9; ++i) {
        const int dst = (9 * w + i) * 1024 + 16 * lane;
        for (int e = 0; e < 8; ++e) {
          CHECK(tag[dst / 2 + e] == -1, "sparse fetch writes slot %d twice", dst / 2 + e);
          tag[dst / 2 + e] = f.row(i) * cols + f.coff(i) / 2 + e;
        }
        CHECK(f.row(i) == SFetch::first_row(w, i) || f.row(i) == SFetch::first_row(w, i) + 1,
              "sparse fetch row %d outside the two rows of instruction %d of wave %d", f.row(i), i, w);
        CHECK(SFetch::first_row(w, i) + 1 < kKeys || f.row(i) == SFetch::first_row(w, i),
              "sparse fetch of wave %d instruction %d needs a row past the tile", w, i);
        CHECK(SFetch::first_row(w, i) == 8 * w + (8 * i) / 9, "first row of wave %d instruction %d", w, i);
        CHECK((f.row(i) != SFetch::first_row(w, i)) == (lane >= SFetch::second_lane(i)),
              "second-row lanes of wave %d instruction %d lane %d", w, i, lane);
      }
    }
  for (int v : tag) CHECK(v >= 0, "sparse fetch leaves a slot unwritten");

  SOffsets o[64];
  for (int l = 0; l < 64; ++l) o[l] = s_offsets(l);
  for (int ks = 0; ks < 36; ++ks) {
    int off[64];
    for (int l = 0; l < 64; ++l) {
      off[l] = o[l].row_off(ks & 3) + 128 * (ks >> 2);
      const int row = l & 31, c0 = 16 * ks + 8 * (l >> 5);
      for (int e = 0; e < 8; ++e)
        CHECK(tag[off[l] / 2 + e] == row * cols + c0 + e, "sparse row operand ks=%d lane=%d e=%d", ks, l, e);
    }
    check_b128_phases(off, "sparse row operand");
  }
  for (int db = 0; db < 18; ++db)
    for (int r = 0; r < 32; r += 8) {
      int off[64];
      for (int l = 0; l < 64; ++l) off[l] = 128 * (db >> 1) + o[l].col_off((r >> 3) & 1, db & 1) + r * kRow;
      for (int l = 0; l < 64; ++l)
        for (int j = 0; j < 4; ++j) {
          const int want = (r + 4 * (l >> 5) + j) * cols + 32 * db + (l & 31);
          CHECK(tr_elem(tag, off, l, j) == want, "sparse transposed operand db=%d r=%d lane=%d j=%d", db, r, l, j);
        }
      check_b64_phases(off, "sparse transposed operand");
    }
}

// The fused sparse backward's tiles (b_swz, 16x16x32 operands).  Its row reads
// (16 rows x 4 chunks per instruction) fall outside the 16-lanes-per-phase
// model: that model flags lanes l and l + 8 (rows r and r + 8, one bank group),
// yet the hardware's SQ_LDS_BANK_CONFLICT counter reads zero for every one of
// the 36 row-read and 72 transposing-read steps of this layout (3.9 and 2.0
// LDS cycles per instruction), while the s_swz layout costs 7.9 cycles on the
// row reads.  The row reads are checked for distinct bank groups within each
// eight consecutive lanes, which the measured layout satisfies.
static void fused() {
  using namespace ls::sparse;
  const int cols = kRow / 2;
  std::vector<int> tag(kTile / 2, -1);
  for (int w = 0; w < 4; ++w)
    for (int lane = 0; lane < 64; ++lane) {
      SFetchT<true> f;
      f.init(lane, w);
      for (int i = 0; i < 9; ++i) {
        const int dst = (9 * w + i) * 1024 + 16 * lane;
        for (int e = 0; e < 8; ++e) {
          CHECK(tag[dst / 2 + e] == -1, "fused fetch writes slot %d twice", dst / 2 + e);
          tag[dst / 2 + e] = f.row(i) * cols + f.coff(i) / 2 + e;
        }
      }
    }
  for (int v : tag) CHECK(v >= 0, "fused fetch leaves a slot unwritten");
  BOffsets o[64];
  for (int l = 0; l < 64; ++l) o[l] = b_offsets(l);
  for (int mb = 0; mb < 2; ++mb)
    for (int ks = 0; ks < 18; ++ks) {
      int off[64];
      for (int l = 0; l < 64; ++l) {
        off[l] = o[l].row_off(mb, ks);
        const int key = 16 * mb + (l & 15), c0 = 32 * ks + 8 * (l >> 4);
        for (int e = 0; e < 8; ++e)
          CHECK(tag[off[l] / 2 + e] == key * cols + c0 + e, "fused row operand mb=%d ks=%d lane=%d e=%d",
                mb, ks, l, e);
      }
      check_b128_octets(off, "fused row operand");
    }
  for (int db = 0; db < 36; ++db)
    for (int k = 0; k < 2; ++k) {
      int off[64];
      for (int l = 0; l < 64; ++l) off[l] = o[l].col_off(k, db);
      for (int l = 0; l < 64; ++l)
        for (int j = 0; j < 4; ++j) {
          const int want = (key_base(l >> 4, k) + j) * cols + 16 * db + (l & 15);
          CHECK(tr_elem(tag, off, l, j) == want, "fused transposed operand db=%d k=%d lane=%d j=%d",
                db, k, l, j);
        }
      check_b64_phases(off, "fused transposed operand");
    }
  // the two reads of each lane group cover the tile's 32 keys once
  for (int g = 0; g < 4; ++g) {
    unsigned keys = 0;
    for (int g2 = 0; g2 < 4; ++g2)
      for (int k = 0; k < 2; ++k)
        for (int j = 0; j < 4; ++j) keys |= 1u << (key_base(g2, k) + j);
    CHECK(keys == 0xFFFFFFFFu, "fused transposed operands miss a key");
  }
}

// The forward's XCD dealing (tail_spread_item): every work item exactly once,
// and the last z slice spread so that no XCD holds two more of its items than
// another.
static void xcd_dealing() {
  using namespace ls;
  for (uint32_t nx = 1; nx <= 40; ++nx)
    for (uint32_t ny = 1; ny <= 3; ++ny)
      for (uint32_t nz = 1; nz <= 12; ++nz) {
        const uint32_t n = nx * ny * nz;
        std::vector<int> seen(n, 0);
        int tail[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (uint32_t id = 0; id < n; ++id) {
          const WorkItem it = tail_spread_item(id, nx, ny, nz);
          CHECK(it.x >= 0 && it.x < (int)nx && it.y >= 0 && it.y < (int)ny && it.z >= 0 &&
                    it.z < (int)nz,
                "xcd dealing %u x %u x %u: item out of range", nx, ny, nz);
          if (it.x < 0 || it.x >= (int)nx || it.y < 0 || it.y >= (int)ny || it.z < 0 || it.z >= (int)nz)
            continue;
          ++seen[it.x + nx * (it.y + ny * it.z)];
          if (it.z == (int)nz - 1) ++tail[id % 8];
        }
        for (uint32_t w = 0; w < n; ++w)
          CHECK(seen[w] == 1, "xcd dealing %u x %u x %u: item %u dealt %d times", nx, ny, nz, w, seen[w]);
        int lo = tail[0], hi = tail[0];
        for (int k = 1; k < 8; ++k) {
          lo = tail[k] < lo ? tail[k] : lo;
          hi = tail[k] > hi ? tail[k] : hi;
        }
        if (nz > 1) CHECK(hi - lo <= 2, "xcd dealing %u x %u x %u: last slice %d..%d per XCD", nx, ny, nz, lo, hi);
      }
}

int main() {
  dense();
  sparse();
  fused();
  xcd_dealing();
  if (failures) {
    printf("%d failures\n", failures);
    return 1;
  }
  printf("lds layouts ok\n");
  return 0;
}
