// Host-side integer layout of the observed ratings: minibatch blocks, per-block CSR by
// user in canonical (user, item, load index) order, and the segment schedule the sweep
// kernels walk.  Integer work only; bit-exact by construction.
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace psmf {

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
  // segment schedule: users with >= 1 rating, longest first (ties: lower id first)
  std::vector<int32_t> seg_user;
  std::vector<int64_t> seg_beg;
  std::vector<int32_t> seg_len;
  std::vector<int32_t> seg_cls;
  int32_t nheavy = 0;  // the first nheavy segments are long enough for a whole workgroup
  std::vector<int32_t> untouched;  // users with no rating in the block
};

struct LayoutParams {
  int64_t users = 0, items = 0;
  int32_t B = 1;
  uint64_t seed = 0;
  int32_t nclass = 1;               // worker classes that share one view schedule
  const int32_t *owner = nullptr;   // [users]
  const int32_t *cls_of_worker = nullptr;  // [P]
  int32_t heavy_min = 1 << 30;      // segments with at least this many ratings are "heavy"
  int32_t threads = 1;
};

// Validates the COO input (EINVAL message in err) and fills one BlockLayout per block.
// Returns 0, -1 (invalid input) or -2 (allocation failure).
int build_layout(const LayoutParams &p, const int32_t *user, const int32_t *item, const float *val, int64_t n,
                 std::vector<BlockLayout> &out, std::string &err);

}  // namespace psmf
