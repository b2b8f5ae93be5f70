// Bounds-checked CPU build of the host layout (minibatch blocks, canonical CSR, work units,
// LDS cells, dense tiles, the sequential step's order): compiled by test_layout_bounds.py
// with the host compiler's address and undefined-behaviour sanitizers and the C++ library's
// container assertions.  It builds the layout of several seeded inputs under many parameter
// sets and runs the layout's own self-check on every block; any out-of-bounds access,
// undefined behaviour or failed check ends the program with a non-zero status.
#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "../paper_1410_8043_amd/csrc/layout.h"

namespace {

struct Coo {
  int64_t N = 0, M = 0;
  std::vector<int32_t> u, i;
  std::vector<float> v;
};

uint64_t next(uint64_t &s) { return s = psmf::splitmix64_next(s); }

// n ratings; skew > 0 draws users and items from a squared uniform (more weight on low ids)
Coo make(int64_t N, int64_t M, int64_t n, uint64_t seed, bool skew) {
  Coo c;
  c.N = N;
  c.M = M;
  uint64_t s = seed;
  for (int64_t t = 0; t < n; ++t) {
    double a = (next(s) >> 11) * (1.0 / 9007199254740992.0), b = (next(s) >> 11) * (1.0 / 9007199254740992.0);
    if (skew) { a *= a; b *= b; }
    c.u.push_back(static_cast<int32_t>(a * N));
    c.i.push_back(static_cast<int32_t>(b * M));
    c.v.push_back(static_cast<float>(1 + next(s) % 5));
  }
  return c;
}

int run(const char *name, const Coo &c, int P, int nclass, int B, int Kp, int64_t heavy_min, int hot_steps,
        int dense_min, int unit_max, int64_t tile_rows, int seq_groups) {
  std::vector<int32_t> owner(static_cast<size_t>(c.N)), cls(static_cast<size_t>(P));
  for (int64_t x = 0; x < c.N; ++x) owner[static_cast<size_t>(x)] = static_cast<int32_t>((x * 7 + 3) % P);
  for (int p = 0; p < P; ++p) cls[static_cast<size_t>(p)] = p % nclass;
  psmf::LayoutParams lp;
  lp.users = c.N;
  lp.items = c.M;
  lp.B = B;
  lp.seed = 0x14108043u + static_cast<uint64_t>(B);
  lp.nclass = nclass;
  lp.owner = owner.data();
  lp.cls_of_worker = cls.data();
  lp.threads = 4;
  lp.tile_rows_user = tile_rows;
  lp.tile_rows_item = 2 * tile_rows;
  lp.unit_max = unit_max;
  lp.workers = P;
  if (seq_groups > 0) {
    lp.seq_groups = seq_groups;
  } else {
    lp.cell_rows = 32768 / Kp;
    lp.cell_groups = 1024 / (Kp >= 128 ? 8 : Kp >= 32 ? 8 : 4);
    lp.heavy_min = heavy_min;
    lp.hot_steps = hot_steps;
    lp.dense_min = dense_min;
    lp.dense_target = 64;
  }
  std::vector<psmf::BlockLayout> L;
  std::string err;
  const int rc = psmf::build_layout(lp, c.u.data(), c.i.data(), c.v.data(), static_cast<int64_t>(c.u.size()), L, err);
  if (rc) {
    std::printf("FAIL %s: build_layout %d %s\n", name, rc, err.c_str());
    return 1;
  }
  int bad = 0;
  int64_t total = 0;
  for (int b = 0; b < B; ++b) {
    total += L[static_cast<size_t>(b)].nnz;
    if (psmf::check_layout(lp, L[static_cast<size_t>(b)], err)) {
      std::printf("FAIL %s: block %d: %s\n", name, b, err.c_str());
      ++bad;
    }
  }
  if (total != static_cast<int64_t>(c.u.size())) {
    std::printf("FAIL %s: blocks hold %lld of %zu ratings\n", name, static_cast<long long>(total), c.u.size());
    ++bad;
  }
  if (!bad) std::printf("ok %s\n", name);
  return bad;
}

}  // namespace

int main() {
  int bad = 0;
  const Coo uni = make(300, 120, 6000, 11, false);
  const Coo skew = make(400, 150, 12000, 12, true);
  const Coo tiny = make(1, 1, 5, 13, false);
  const Coo empty = make(50, 40, 0, 14, false);
  char name[128];
  for (const Coo *c : {&uni, &skew}) {
    for (int B : {1, 3}) {
      for (int nclass : {1, 3}) {
        for (int dense : {0, 1, 60}) {
          for (int hot : {0, 2}) {
            std::snprintf(name, sizeof name, "%s B=%d classes=%d dense=%d hot=%d", c == &uni ? "uniform" : "skewed", B,
                          nclass, dense, hot);
            bad += run(name, *c, 5, nclass, B, 16, 20, hot, dense, 16, 64, 0);
          }
        }
      }
      for (int Kp : {8, 128, 512}) {
        std::snprintf(name, sizeof name, "%s B=%d Kp=%d", c == &uni ? "uniform" : "skewed", B, Kp);
        bad += run(name, *c, 4, 2, B, Kp, 30, 1, Kp >= 16 && Kp <= 256 ? 10 : 0, 256, 1 << 20, 0);
      }
      for (int G : {1, 7}) {
        std::snprintf(name, sizeof name, "%s B=%d seq G=%d", c == &uni ? "uniform" : "skewed", B, G);
        bad += run(name, *c, 5, 3, B, 16, 0, 0, 0, 256, 64, G);
      }
    }
  }
  bad += run("one rating row", tiny, 1, 1, 1, 16, 1, 1, 1, 1, 1, 0);
  bad += run("one rating row seq", tiny, 1, 1, 2, 16, 0, 0, 0, 1, 1, 3);
  bad += run("empty", empty, 3, 2, 2, 16, 1, 1, 1, 8, 8, 0);
  bad += run("empty seq", empty, 3, 2, 2, 16, 0, 0, 0, 8, 8, 4);
  std::printf("%d failures\n", bad);
  return bad ? 1 : 0;
}
