// Host-side integer layout of the observed ratings: minibatch blocks, per-block CSR by
// user in canonical (user, item, load index) order, and the work units the sweep kernels
// walk.  Integer work only; bit-exact by construction.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace psmf {

constexpr int kXcds = 8;       // MI355X: 8 accelerator complex dies, each with its own L2
constexpr int kUnitAlign = 8;  // a unit's ratings start at, and are padded to, a multiple of this
constexpr int kWaveUnits = 32; // units of one wavefront (at most 32 lane groups) share a worker class
constexpr int kDenseRows = 64; // rows on each side of a dense tile (4 wavefronts x 16 MFMA rows)
constexpr int kDenseTile = kDenseRows * kDenseRows;

// Position of rating (x, y) of a dense tile (x, y local in [0, 64)) in its 4096-float
// block of values: the order in which the MFMA cell reads them.  Wavefront w = x / 16
// holds rows x of the stationary side; for its 16-row slice yb = y / 16 of the staged
// side, lane l = (x % 16) + 16 * ((y % 16) / 4) reads the 4 values y % 4 = 0..3 as one
// float4 (the C/D fragment of a 16x16x4 fp32 MFMA whose rows are y and columns x).
constexpr int32_t dense_frag_index(int32_t x, int32_t y) {
  const int32_t w = x >> 4, yb = y >> 4, lane = (x & 15) + 16 * ((y & 15) >> 2);
  return (((w * 4 + yb) * 64 + lane) << 2) + (y & 3);
}

// SplitMix64 (Steele, Lea & Flood 2014): one step of the sequential generator from
// `state`.  Used for the minibatch block of a rating.
inline uint64_t splitmix64_next(uint64_t state) {
  uint64_t z = state + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

inline int32_t block_of(uint64_t seed, int32_t B, int64_t i, int64_t j) {
  if (B == 1) return 0;
  const uint64_t key = seed ^ ((static_cast<uint64_t>(i) << 32) | static_cast<uint64_t>(static_cast<uint32_t>(j)));
  return static_cast<int32_t>(splitmix64_next(key) % static_cast<uint64_t>(B));
}

// The ratings of one block cut into work units for one sweep direction.  The sweep keeps
// one "stationary" row x in registers and gathers the rows y of the other factor from a
// tile of y rows small enough to stay in one XCD's L2:
//   user-major (dL): x = user, y = item, tiles = (worker class, item id range);
//   item-major (dR): x = item, y = user, tiles = class-pure ranges of users.
// A unit is a run of one x's ratings inside one tile, split at unit_max ratings.  Units
// are stored in execution order (tile, longest first) and cut into kXcds contiguous
// chunks of about equal rating count; chunk x runs on XCD x.  Each unit writes one
// partial row; the partial rows of x are [x_pp[x], x_pp[x+1]).
struct UnitSet {
  std::vector<int32_t> y;         // gathered row of each rating, in unit order (padded)
  std::vector<float> val;         // rating value, in unit order (padding: 0)
  std::vector<int32_t> unit_x, unit_cls, unit_len, unit_out;
  std::vector<int64_t> unit_beg;
  std::vector<int64_t> xcd_off;   // [kXcds + 1]
  std::vector<int64_t> x_pp;      // [rows of x + 1]
  std::vector<uint8_t> sole;      // [rows of x]: 1 where x's only partial row is one unit's
  int64_t ntiles = 0;
  int64_t nreal = 0;              // units with ratings; empty padding units write partial row nreal
};

// The dense part of one sweep direction, staged through LDS.  A cell is one workgroup:
// ng stationary rows x (one per lane group, -1 = unused) of one worker class, and a
// sequence of steps; a step is a sub-tile of ts gathered rows that the workgroup copies
// into LDS before every lane group sweeps its row's ratings inside the sub-tile:
//   user-major: x = heavy users of one class (similar degree), steps = item ranges;
//               x = light users of one class, steps = the sub-tiles of the hot items;
//   item-major: x = items (similar heavy-rater count), steps = ranges of the class's
//               heavy users; x = hot items, steps = ranges of the class's light users.
// The ratings of (cell, k-th step, group) are ly/lv[run_beg .. run_beg + run_len): ly the
// row's position inside the sub-tile.  Runs start at multiples of kUnitAlign and are
// padded to one.  Each used (cell, group) writes one partial row cell_out.
struct CellSet {
  int32_t ts = 0, ng = 0;
  std::vector<int32_t> step_rows;      // [nsteps * ts], -1 = no row
  std::vector<int32_t> cell_x;         // [ncells * ng]
  std::vector<int32_t> cell_cls;       // [ncells]
  std::vector<int32_t> cell_step_ptr;  // [ncells + 1] into cell_steps
  std::vector<int32_t> cell_steps;     // step ids
  std::vector<int32_t> run_beg, run_len;  // [cell_steps.size() * ng]
  std::vector<int32_t> cell_out;       // [ncells * ng], -1 for unused groups
  std::vector<uint16_t> ly;
  std::vector<float> lv;
  int64_t nnz = 0;                     // ratings covered by the cells
};

// The densest part of a block as 64 x 64 tiles, swept with matrix-core (MFMA) products
// instead of per-rating dot products.  A tile is 64 users of one worker class (ranked
// by their rating count in the block) x 64 items (ranked by their rating count) holding
// at least dense_min ratings; both sweep directions walk the same tiles:
//   user-major: a cell is one user tile (x = 64 users) and a run of its dense item
//               tiles (steps, y = 64 items each);
//   item-major: a cell is one item tile (x = 64 items) and a run of the dense user
//               tiles of one class (steps).
// A step's ratings are stored as a 64 x 64 block in dense_frag_index order, NaN where
// there is no rating.  Each used (cell, x row) writes one partial row cell_out.
struct DenseSet {
  std::vector<int32_t> cell_x;         // [ncells * 64], -1 = no row
  std::vector<int32_t> cell_cls;       // [ncells]
  std::vector<int32_t> cell_step_ptr;  // [ncells + 1] into the steps
  std::vector<int32_t> step_rows;      // [nsteps * 64] staged rows of each step, -1 = no row
  std::vector<float> dval;             // [nsteps * 4096]
  std::vector<int32_t> step_twin;      // [nsteps] the other direction's step of the same tile
  std::vector<int32_t> cell_out;       // [ncells * 64], -1 for unused rows
  int64_t nnz = 0;                     // ratings covered
};

// The sequential step (each worker applies its ratings one by one to its own copies of the
// rows): the block's ratings in the order the workers apply them.  Worker p's ratings run in
// G sub-epochs; in sub-epoch t the stratum (user group g, item group (g + t) mod G) of every
// g, each in canonical order -- user group (i div P) mod G, item group j mod G.  A chain is
// one (sub-epoch, worker, user group) stratum with ratings; chains are stored by sub-epoch,
// and the strata of one sub-epoch share no row, so its chains run side by side.
// Flags of a rating: kSeqRunStart on the first rating of a user's run inside a chain, with
// kSeqFirstL when the run is the user's first of the clock (L_i is read from the view, later
// runs from the work copy); kSeqFirstR when it is worker p's first rating of item j in the
// clock (R_j is read from the view, later ones from the worker's copy).  Bits 4..7 hold the
// distance k in [1, kSeqAhead] to the latest of the kSeqAhead ratings before it in the chain
// with the same item (0: none): the sweep fetches item rows kSeqAhead ratings ahead, before
// those ratings store theirs, so such a rating takes the row that rating k back wrote.
constexpr uint8_t kSeqFirstL = 1, kSeqRunStart = 2, kSeqFirstR = 4;
constexpr int kSeqAhead = 8;
constexpr int kSeqDistShift = 4;
struct SeqSet {
  int32_t G = 0;
  std::vector<int64_t> epoch_chain;   // [G + 1]: the chains of sub-epoch t
  std::vector<int64_t> chain_beg;     // [nchains + 1] into the rating arrays
  std::vector<int32_t> chain_worker;  // [nchains]
  std::vector<int32_t> user, item;    // [nnz] in application order
  std::vector<float> val;
  std::vector<uint8_t> flag;
  std::vector<int32_t> canon;         // [nnz] canonical position of each rating (host only)
  std::vector<int64_t> item_wptr;     // [items + 1]
  std::vector<int32_t> item_workers;  // the workers with a rating of item j, ascending
};

struct BlockLayout {
  int64_t nnz = 0;
  // ratings of the block in canonical (user, item, load index) order
  std::vector<int32_t> col;
  std::vector<float> val;
  std::vector<int64_t> perm;     // load index of each entry
  std::vector<int64_t> row_ptr;  // [users + 1], users in id order
  std::vector<int32_t> ucount;   // [users]
  std::vector<int32_t> icount;   // [items]
  std::vector<int32_t> icount_cls;  // [items * nclass]: raters of the item per worker class
  UnitSet by_user, by_item;
  CellSet cells_user, cells_item;
  DenseSet dense_user, dense_item;
  SeqSet seq;
  int64_t partial_rows_user = 0, partial_rows_item = 0;  // rows of x_pp (units and cells)
};

struct LayoutParams {
  int64_t users = 0, items = 0;
  int32_t B = 1;
  uint64_t seed = 0;
  int32_t nclass = 1;               // worker classes that share one view schedule
  const int32_t *owner = nullptr;   // [users]
  const int32_t *cls_of_worker = nullptr;  // [P]
  int32_t threads = 1;
  int64_t tile_rows_item = 1 << 30; // items per tile of the user-major sweep
  int64_t tile_rows_user = 1 << 30; // users per tile of the item-major sweep
  int32_t unit_max = 1024;          // ratings per work unit
  int32_t cell_rows = 0;            // ts: gathered rows per LDS sub-tile (0: no cells)
  int32_t cell_groups = 0;          // ng: lane groups per cell workgroup
  int64_t heavy_min = 1 << 30;      // users with at least this many ratings in the block go to cells
  int32_t cell_target = 1024;       // about this many cells per family and direction
  int32_t hot_steps = 0;            // sub-tiles of the most rated items whose ratings by the other
                                    // (light) users also go to cells
  int32_t dense_min = 0;            // ratings from which a 64 x 64 tile goes to the MFMA cells
                                    // (0: none)
  int32_t dense_target = 1024;      // about this many dense cells per direction
  int32_t min_cell_steps = 4;       // runs of cells and dense cells are not cut below this many
                                    // steps (each cut costs every row of the cell a partial row)
  int32_t workers = 1;              // P
  int32_t seq_groups = 0;           // G > 0: build the sequential step's order (SeqSet) instead of
                                    // units, cells and dense tiles
};

// Validates the COO input (EINVAL message in err) and fills one BlockLayout per block.
// Returns 0, -1 (invalid input) or -2 (allocation failure).
int build_layout(const LayoutParams &p, const int32_t *user, const int32_t *item, const float *val, int64_t n,
                 std::vector<BlockLayout> &out, std::string &err);

// Self-check of one block's layout against its canonical entries: in each sweep direction
// the units, cells and dense cells together hold every entry exactly once (same stationary row,
// gathered row and value), every unit and cell reads the ring slot of its ratings' user
// class (wave-uniform for units), padding is (row 0, value 0), and the partial rows of
// each x are written exactly once each.  For the sequential step: the order holds every
// entry once, sorted by (sub-epoch, worker, user group, canonical position), chains are
// maximal runs of one stratum, and the flags and item worker lists match their
// definitions.  Returns 0, or -1 with err naming the first fault.
int check_layout(const LayoutParams &p, const BlockLayout &L, std::string &err);

}  // namespace psmf
