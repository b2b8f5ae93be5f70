// Host-side integer layout (see layout.h).
#include "layout.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <functional>
#include <new>
#include <numeric>
#include <thread>

namespace psmf {

namespace {

template <class F>
void parallel_for(int threads, int64_t n, F &&fn) {
  if (threads <= 1 || n < (1 << 16)) {
    fn(int64_t(0), n);
    return;
  }
  std::vector<std::thread> pool;
  for (int t = 0; t < threads; ++t) {
    const int64_t lo = n * t / threads, hi = n * (t + 1) / threads;
    pool.emplace_back([&fn, lo, hi] { fn(lo, hi); });
  }
  for (auto &th : pool) th.join();
}

// one stable counting-sort pass: dst receives src ordered by key(src[x]) in [0, range)
template <class Key>
void counting_pass(const std::vector<int64_t> &src, std::vector<int64_t> &dst, int64_t range, Key key) {
  std::vector<int64_t> cnt(static_cast<size_t>(range) + 1, 0);
  for (int64_t x : src) cnt[static_cast<size_t>(key(x)) + 1] += 1;
  for (int64_t r = 0; r < range; ++r) cnt[r + 1] += cnt[r];
  for (int64_t x : src) dst[static_cast<size_t>(cnt[static_cast<size_t>(key(x))]++)] = x;
}

// Work units of one sweep direction over the canonical entries e of a block with
// in_units[e] != 0.
//   xrow(e), yrow(e): stationary and gathered row of entry e;
//   tile(e) in [0, ntiles), cls_of_tile(t): the worker class whose view the tile reads.
// The canonical order must already be sorted by y within equal x (true for both
// directions: canonical is (user, item)), so two stable passes give (tile, x, y).
// Partial rows: x owns [x_pp[x], x_pp[x+1]) = its units' rows, then extra[x] rows that
// the cells of x fill from cell_base[x] on.  Padding units write row x_pp[nx].
void build_units(int64_t nb, int64_t nx, int64_t ntiles, const std::function<int32_t(int64_t)> &xrow,
                 const std::function<int32_t(int64_t)> &yrow, const std::function<int32_t(int64_t)> &tile,
                 const std::function<int32_t(int64_t)> &cls_of_tile, const std::vector<float> &val,
                 int32_t unit_max, const std::vector<uint8_t> &in_units, const std::vector<int64_t> &extra,
                 std::vector<int64_t> &cell_base, UnitSet &U) {
  U.ntiles = ntiles;
  std::vector<int64_t> a, b;
  for (int64_t e = 0; e < nb; ++e)
    if (in_units[e]) a.push_back(e);
  const int64_t na = static_cast<int64_t>(a.size());
  b.resize(static_cast<size_t>(na));
  counting_pass(a, b, nx, xrow);
  counting_pass(b, a, ntiles, tile);
  std::vector<int64_t>().swap(b);
  struct Unit { int32_t tile, x; int64_t beg; int32_t len; };
  std::vector<Unit> units;
  std::vector<int64_t> tile_units(static_cast<size_t>(ntiles) + 1, 0);
  for (int64_t e = 0; e < na;) {
    const int32_t t = tile(a[e]), x = xrow(a[e]);
    int64_t f = e;
    while (f < na && xrow(a[f]) == x && tile(a[f]) == t) ++f;
    for (int64_t c = e; c < f; c += unit_max) {
      units.push_back({t, x, c, static_cast<int32_t>(std::min<int64_t>(unit_max, f - c))});
      tile_units[t + 1] += 1;
    }
    e = f;
  }
  for (int64_t t = 0; t < ntiles; ++t) tile_units[t + 1] += tile_units[t];
  const int64_t nu = static_cast<int64_t>(units.size());
  // partial rows in (x, tile, chunk) order: units are generated in (tile, x) order, so a
  // stable pass by x gives it; the cells' rows of x follow its units' rows
  std::vector<int64_t> ucnt(static_cast<size_t>(nx), 0);
  for (const Unit &u : units) ucnt[u.x] += 1;
  U.x_pp.assign(static_cast<size_t>(nx) + 1, 0);
  for (int64_t x = 0; x < nx; ++x) U.x_pp[x + 1] = U.x_pp[x] + ucnt[x] + (extra.empty() ? 0 : extra[x]);
  cell_base.assign(static_cast<size_t>(nx), 0);
  for (int64_t x = 0; x < nx; ++x) cell_base[x] = U.x_pp[x] + ucnt[x];
  const int64_t spare = U.x_pp[nx];
  std::vector<int32_t> out_of(static_cast<size_t>(nu));
  {
    std::vector<int64_t> fill(U.x_pp.begin(), U.x_pp.end() - 1);
    for (int64_t k = 0; k < nu; ++k) out_of[k] = static_cast<int32_t>(fill[units[k].x]++);
  }
  nb = na;  // the chunks below balance the rating count of the unit path
  // execution order: tile by tile, longest unit first; kXcds contiguous chunks of about
  // equal rating count.  Each unit's ratings start at a multiple of kUnitAlign entries and
  // are padded with (row 0, value 0) entries to a multiple of kUnitAlign.  Empty units
  // (length 0, writing the spare partial row nu) pad every chunk start and every change
  // of worker class to a multiple of kWaveUnits, so the units of one wavefront always
  // read the same ring slot.
  std::vector<int64_t> order;
  order.reserve(static_cast<size_t>(nu));
  std::vector<int64_t> ids;
  for (int64_t t = 0; t < ntiles; ++t) {
    ids.resize(static_cast<size_t>(tile_units[t + 1] - tile_units[t]));
    std::iota(ids.begin(), ids.end(), tile_units[t]);
    std::stable_sort(ids.begin(), ids.end(), [&](int64_t q, int64_t r) { return units[q].len > units[r].len; });
    order.insert(order.end(), ids.begin(), ids.end());
  }
  int64_t padded = 0;
  for (const Unit &u : units) padded += (u.len + kUnitAlign - 1) / kUnitAlign * kUnitAlign;
  U.y.assign(static_cast<size_t>(padded), 0);
  U.val.assign(static_cast<size_t>(padded), 0.f);
  U.unit_x.clear();
  U.unit_cls.clear();
  U.unit_len.clear();
  U.unit_out.clear();
  U.unit_beg.clear();
  U.xcd_off.assign(kXcds + 1, 0);
  int64_t pos = 0, rated = 0;
  int next_xcd = 0;
  int32_t prev_cls = -1;
  auto pad_to_wave = [&](int32_t cls) {
    while (U.unit_x.size() % kWaveUnits != 0) {
      U.unit_x.push_back(0);
      U.unit_cls.push_back(cls);
      U.unit_len.push_back(0);
      U.unit_out.push_back(static_cast<int32_t>(spare));
      U.unit_beg.push_back(0);
    }
  };
  for (int64_t q : order) {
    const Unit &u = units[q];
    const int32_t cls = cls_of_tile(u.tile);
    bool chunk_start = false;
    while (next_xcd < kXcds && rated * kXcds >= next_xcd * nb) {
      if (!chunk_start) pad_to_wave(prev_cls < 0 ? cls : prev_cls);
      chunk_start = true;
      U.xcd_off[next_xcd++] = static_cast<int64_t>(U.unit_x.size());
    }
    if (!chunk_start && cls != prev_cls && prev_cls >= 0) pad_to_wave(prev_cls);
    prev_cls = cls;
    U.unit_x.push_back(u.x);
    U.unit_cls.push_back(cls);
    U.unit_len.push_back(u.len);
    U.unit_out.push_back(out_of[q]);
    U.unit_beg.push_back(pos);
    for (int64_t c = 0; c < u.len; ++c) {
      const int64_t e = a[u.beg + c];
      U.y[pos + c] = yrow(e);
      U.val[pos + c] = val[e];
    }
    rated += u.len;
    pos += (u.len + kUnitAlign - 1) / kUnitAlign * kUnitAlign;
  }
  pad_to_wave(prev_cls < 0 ? 0 : prev_cls);
  while (next_xcd < kXcds) U.xcd_off[next_xcd++] = static_cast<int64_t>(U.unit_x.size());
  U.xcd_off[kXcds] = static_cast<int64_t>(U.unit_x.size());
  U.nreal = nu;
}

// number of distinct (x, tile) runs for a tile function (entries sorted by x already)
int64_t count_runs(int64_t nb, const std::vector<int64_t> &by_x, const std::function<int32_t(int64_t)> &xrow,
                   const std::function<int32_t(int64_t)> &tile, int64_t ntiles, const std::vector<uint8_t> &in_units,
                   std::vector<int64_t> &last) {
  last.assign(static_cast<size_t>(ntiles), -1);
  int64_t runs = 0;
  for (int64_t e = 0; e < nb; ++e) {
    if (!in_units[by_x[e]]) continue;
    const int64_t x = xrow(by_x[e]);
    const int32_t t = tile(by_x[e]);
    if (last[t] != x) {
      last[t] = x;
      ++runs;
    }
  }
  return runs;
}

// Append the ratings [lo, hi) of the (already ordered) list `ents` as one 8-aligned run.
void append_run(CellSet &C, const std::vector<int64_t> &ents, int64_t lo, int64_t hi,
                const std::function<int32_t(int64_t)> &local, const std::vector<float> &val) {
  const int64_t beg = static_cast<int64_t>(C.ly.size());
  C.run_beg.push_back(static_cast<int32_t>(beg));
  C.run_len.push_back(static_cast<int32_t>(hi - lo));
  for (int64_t q = lo; q < hi; ++q) {
    C.ly.push_back(static_cast<uint16_t>(local(ents[q])));
    C.lv.push_back(val[ents[q]]);
  }
  while (C.ly.size() % kUnitAlign) {
    C.ly.push_back(0);
    C.lv.push_back(0.f);
  }
  C.nnz += hi - lo;
}

void empty_run(CellSet &C) {
  C.run_beg.push_back(static_cast<int32_t>(C.ly.size()));
  C.run_len.push_back(0);
}

// User-major cells: heavy users of one class, sorted by degree, ng per cell; steps are
// item ranges of ts items; the item space is cut into R ranges of steps so that there are
// about cell_target cells.  Each heavy user owns R partial rows.
void build_user_cells(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                      const std::vector<uint8_t> &heavy, CellSet &C, std::vector<int64_t> &extra) {
  const int64_t N = p.users, M = p.items, ts = p.cell_rows, ng = p.cell_groups;
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  extra.assign(static_cast<size_t>(N), 0);
  std::vector<std::vector<int32_t>> by_cls(static_cast<size_t>(p.nclass));
  for (int64_t i = 0; i < N; ++i)
    if (heavy[i]) by_cls[ucls[i]].push_back(static_cast<int32_t>(i));
  int64_t groups = 0;
  for (auto &v : by_cls) {
    std::stable_sort(v.begin(), v.end(), [&](int32_t a, int32_t b) { return L.ucount[a] > L.ucount[b]; });
    groups += (static_cast<int64_t>(v.size()) + ng - 1) / ng;
  }
  if (groups == 0) return;
  const int64_t nsub = (M + ts - 1) / ts;
  const int64_t R = std::max<int64_t>(1, std::min<int64_t>(nsub, (p.cell_target + groups - 1) / groups));
  C.step_rows.resize(static_cast<size_t>(nsub * ts));
  for (int64_t t = 0; t < nsub * ts; ++t) C.step_rows[t] = t < M ? static_cast<int32_t>(t) : -1;
  std::vector<int64_t> ents(L.col.size());
  std::iota(ents.begin(), ents.end(), int64_t(0));
  const std::function<int32_t(int64_t)> local = [&](int64_t e) { return static_cast<int32_t>(L.col[e] % ts); };
  C.cell_step_ptr.push_back(0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    const auto &us = by_cls[c];
    for (size_t g0 = 0; g0 < us.size(); g0 += static_cast<size_t>(ng)) {
      for (int64_t r = 0; r < R; ++r) {
        const int64_t s0 = r * nsub / R, s1 = (r + 1) * nsub / R;
        C.cell_cls.push_back(c);
        for (int64_t q = 0; q < ng; ++q) {
          const size_t k = g0 + static_cast<size_t>(q);
          C.cell_x.push_back(k < us.size() ? us[k] : -1);
          C.cell_out.push_back(-1);  // assigned once the partial rows are laid out
        }
        for (int64_t st = s0; st < s1; ++st) {
          C.cell_steps.push_back(static_cast<int32_t>(st));
          for (int64_t q = 0; q < ng; ++q) {
            const size_t k = g0 + static_cast<size_t>(q);
            if (k >= us.size()) { empty_run(C); continue; }
            const int32_t u = us[k];
            const int32_t *b = L.col.data() + L.row_ptr[u], *e = L.col.data() + L.row_ptr[u + 1];
            const int64_t lo = std::lower_bound(b, e, static_cast<int32_t>(st * ts)) - L.col.data();
            const int64_t hi = std::lower_bound(b, e, static_cast<int32_t>(std::min<int64_t>((st + 1) * ts, M))) - L.col.data();
            append_run(C, ents, lo, hi, local, L.val);
          }
        }
        C.cell_step_ptr.push_back(static_cast<int32_t>(C.cell_steps.size()));
      }
      for (size_t k = g0; k < std::min(us.size(), g0 + static_cast<size_t>(ng)); ++k) extra[us[k]] += R;
    }
  }
}

// Item-major cells: items sorted by heavy-rater count, ng per cell; for each class the
// steps are consecutive ranges of ts of its heavy users (in id order), cut into ranges so
// that there are about cell_target cells.  Each item owns one partial row per (class,
// range).
void build_item_cells(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                      const std::vector<uint8_t> &heavy, const std::vector<int32_t> &ent_user, CellSet &C,
                      std::vector<int64_t> &extra) {
  const int64_t N = p.users, M = p.items, ts = p.cell_rows, ng = p.cell_groups;
  const int64_t nb = static_cast<int64_t>(L.col.size());
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  extra.assign(static_cast<size_t>(M), 0);
  // heavy users of each class in id order; their rank and sub-tile
  std::vector<int64_t> hrank(static_cast<size_t>(N), -1), nheavy(static_cast<size_t>(p.nclass), 0);
  for (int64_t i = 0; i < N; ++i)
    if (heavy[i]) hrank[i] = nheavy[ucls[i]]++;
  std::vector<int64_t> nsub(static_cast<size_t>(p.nclass)), sub_base(static_cast<size_t>(p.nclass) + 1, 0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    nsub[c] = (nheavy[c] + ts - 1) / ts;
    sub_base[c + 1] = sub_base[c] + nsub[c];
  }
  if (sub_base[p.nclass] == 0) return;
  C.step_rows.assign(static_cast<size_t>(sub_base[p.nclass] * ts), -1);
  for (int64_t i = 0; i < N; ++i)
    if (heavy[i]) C.step_rows[(sub_base[ucls[i]] + hrank[i] / ts) * ts + hrank[i] % ts] = static_cast<int32_t>(i);
  // heavy entries ordered by (item, class, user): canonical is (user, item)
  std::vector<int64_t> a, b;
  for (int64_t e = 0; e < nb; ++e)
    if (heavy[ent_user[e]]) a.push_back(e);
  b.resize(a.size());
  counting_pass(a, b, p.nclass, [&](int64_t e) { return ucls[ent_user[e]]; });
  counting_pass(b, a, M, [&](int64_t e) { return L.col[e]; });
  // run boundaries: bnd[(j * nclass + c) .. ] holds nsub[c] + 1 offsets into a
  std::vector<int64_t> jc_base(static_cast<size_t>(M * p.nclass) + 1, 0);
  for (int64_t j = 0; j < M; ++j)
    for (int32_t c = 0; c < p.nclass; ++c) jc_base[j * p.nclass + c + 1] = jc_base[j * p.nclass + c] + nsub[c] + 1;
  std::vector<int64_t> bnd(static_cast<size_t>(jc_base[M * p.nclass]), 0);
  {
    int64_t e = 0;
    const int64_t na = static_cast<int64_t>(a.size());
    for (int64_t j = 0; j < M; ++j)
      for (int32_t c = 0; c < p.nclass; ++c) {
        int64_t *o = bnd.data() + jc_base[j * p.nclass + c];
        for (int64_t st = 0; st < nsub[c]; ++st) {
          o[st] = e;
          while (e < na && L.col[a[e]] == j && ucls[ent_user[a[e]]] == c && hrank[ent_user[a[e]]] / ts == st) ++e;
        }
        o[nsub[c]] = e;
      }
  }
  // items by heavy-rater count
  std::vector<int64_t> hcount(static_cast<size_t>(M), 0);
  for (int64_t e : a) hcount[L.col[e]] += 1;
  std::vector<int32_t> items;
  for (int64_t j = 0; j < M; ++j)
    if (hcount[j] > 0) items.push_back(static_cast<int32_t>(j));
  std::stable_sort(items.begin(), items.end(), [&](int32_t x, int32_t y) { return hcount[x] > hcount[y]; });
  const int64_t groups = (static_cast<int64_t>(items.size()) + ng - 1) / ng;
  int64_t classes_used = 0;
  for (int32_t c = 0; c < p.nclass; ++c) classes_used += nsub[c] > 0;
  if (groups == 0) return;
  const int64_t R = std::max<int64_t>(1, (p.cell_target + groups * classes_used - 1) / (groups * classes_used));
  const std::function<int32_t(int64_t)> local = [&](int64_t e) { return static_cast<int32_t>(hrank[ent_user[e]] % ts); };
  C.cell_step_ptr.push_back(0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    if (nsub[c] == 0) continue;
    const int64_t Rc = std::min<int64_t>(R, nsub[c]);
    for (int64_t g0 = 0; g0 < static_cast<int64_t>(items.size()); g0 += ng) {
      for (int64_t r = 0; r < Rc; ++r) {
        const int64_t s0 = r * nsub[c] / Rc, s1 = (r + 1) * nsub[c] / Rc;
        C.cell_cls.push_back(c);
        for (int64_t q = 0; q < ng; ++q) {
          const int64_t k = g0 + q;
          C.cell_x.push_back(k < static_cast<int64_t>(items.size()) ? items[k] : -1);
          C.cell_out.push_back(-1);
        }
        for (int64_t st = s0; st < s1; ++st) {
          C.cell_steps.push_back(static_cast<int32_t>(sub_base[c] + st));
          for (int64_t q = 0; q < ng; ++q) {
            const int64_t k = g0 + q;
            if (k >= static_cast<int64_t>(items.size())) { empty_run(C); continue; }
            const int64_t *o = bnd.data() + jc_base[items[k] * p.nclass + c];
            append_run(C, a, o[st], o[st + 1], local, L.val);
          }
        }
        C.cell_step_ptr.push_back(static_cast<int32_t>(C.cell_steps.size()));
        for (int64_t q = 0; q < ng && g0 + q < static_cast<int64_t>(items.size()); ++q) extra[items[g0 + q]] += 1;
      }
    }
  }
}

// cell_out of every used (cell, group): the next of x's cell rows from cell_base[x] on
void assign_cell_rows(CellSet &C, std::vector<int64_t> cell_base) {
  for (size_t k = 0; k < C.cell_x.size(); ++k)
    if (C.cell_x[k] >= 0) C.cell_out[k] = static_cast<int32_t>(cell_base[C.cell_x[k]]++);
}

}  // namespace

int build_layout(const LayoutParams &p, const int32_t *user, const int32_t *item, const float *val, int64_t n,
                 std::vector<BlockLayout> &out, std::string &err) {
  try {
    const int64_t N = p.users, M = p.items;
    // ---- validate
    std::atomic<int64_t> bad{-1};
    parallel_for(p.threads, n, [&](int64_t lo, int64_t hi) {
      for (int64_t t = lo; t < hi; ++t) {
        if (user[t] < 0 || user[t] >= N || item[t] < 0 || item[t] >= M || !std::isfinite(val[t])) {
          int64_t expect = -1;
          bad.compare_exchange_strong(expect, t);
          return;
        }
      }
    });
    if (bad.load() >= 0) {
      const int64_t t = bad.load();
      err = "rating " + std::to_string(t) + " is invalid (user " + std::to_string(user[t]) + ", item " +
            std::to_string(item[t]) + ", value not finite or index out of range)";
      return -1;
    }
    // ---- minibatch block of every rating
    std::vector<int32_t> blk;
    if (p.B > 1) {
      blk.resize(static_cast<size_t>(n));
      parallel_for(p.threads, n, [&](int64_t lo, int64_t hi) {
        for (int64_t t = lo; t < hi; ++t) blk[t] = block_of(p.seed, p.B, user[t], item[t]);
      });
    }
    // ---- canonical order: stable LSD counting sorts by item, then user, then block
    std::vector<int64_t> a(static_cast<size_t>(n)), b(static_cast<size_t>(n));
    std::iota(a.begin(), a.end(), int64_t(0));
    counting_pass(a, b, M, [&](int64_t x) { return item[x]; });
    counting_pass(b, a, N, [&](int64_t x) { return user[x]; });
    if (p.B > 1) {
      counting_pass(a, b, p.B, [&](int64_t x) { return blk[x]; });
      a.swap(b);
    }
    std::vector<int64_t>().swap(b);
    // ---- worker class of each user; class-pure user tiles for the item-major sweep
    std::vector<int32_t> ucls(static_cast<size_t>(N));
    for (int64_t i = 0; i < N; ++i) ucls[i] = p.cls_of_worker[p.owner[i]];
    std::vector<int64_t> rank_in_cls(static_cast<size_t>(N)), in_cls(static_cast<size_t>(p.nclass), 0);
    for (int64_t i = 0; i < N; ++i) rank_in_cls[i] = in_cls[ucls[i]]++;
    // ---- per block arrays
    out.assign(static_cast<size_t>(p.B), BlockLayout());
    std::vector<int64_t> bstart(static_cast<size_t>(p.B) + 1, 0);
    for (int64_t t = 0; t < n; ++t) bstart[static_cast<size_t>(p.B > 1 ? blk[t] : 0) + 1] += 1;
    for (int32_t q = 0; q < p.B; ++q) bstart[q + 1] += bstart[q];
    for (int32_t q = 0; q < p.B; ++q) {
      BlockLayout &L = out[q];
      const int64_t lo = bstart[q], nb = bstart[q + 1] - bstart[q];
      L.nnz = nb;
      L.col.resize(static_cast<size_t>(nb));
      L.val.resize(static_cast<size_t>(nb));
      L.perm.assign(a.begin() + lo, a.begin() + lo + nb);
      parallel_for(p.threads, nb, [&](int64_t x0, int64_t x1) {
        for (int64_t x = x0; x < x1; ++x) {
          const int64_t t = L.perm[x];
          L.col[x] = item[t];
          L.val[x] = val[t];
        }
      });
      L.ucount.assign(static_cast<size_t>(N), 0);
      L.icount.assign(static_cast<size_t>(M), 0);
      L.icount_cls.assign(static_cast<size_t>(M * p.nclass), 0);
      std::vector<int32_t> ent_user(static_cast<size_t>(nb));
      for (int64_t x = 0; x < nb; ++x) {
        const int64_t t = L.perm[x];
        ent_user[x] = user[t];
        L.ucount[user[t]] += 1;
        L.icount[item[t]] += 1;
        L.icount_cls[static_cast<size_t>(item[t]) * p.nclass + ucls[user[t]]] += 1;
      }
      L.row_ptr.assign(static_cast<size_t>(N) + 1, 0);
      for (int64_t i = 0; i < N; ++i) L.row_ptr[i + 1] = L.row_ptr[i] + L.ucount[i];

      // ---- cells (the dense part: heavy users, staged through LDS) and units (the rest)
      std::vector<uint8_t> heavy(static_cast<size_t>(N), 0);
      if (p.cell_rows > 0 && p.cell_groups > 0)
        for (int64_t i = 0; i < N; ++i) heavy[i] = L.ucount[i] >= p.heavy_min;
      std::vector<uint8_t> in_units(static_cast<size_t>(nb));
      for (int64_t x = 0; x < nb; ++x) in_units[x] = !heavy[ent_user[x]];
      std::vector<int64_t> extra_u, extra_i, base_u, base_i;
      if (p.cell_rows > 0 && p.cell_groups > 0) {
        build_user_cells(p, L, ucls, heavy, L.cells_user, extra_u);
        build_item_cells(p, L, ucls, heavy, ent_user, L.cells_item, extra_i);
      }
      // ---- units.  Tiles start at the L2-sized row count and grow (x2) while the units
      // would average fewer than 16 ratings (each unit costs one partial row).
      const int64_t min_avg = 16;
      int64_t n_units_entries = 0;
      for (int64_t x = 0; x < nb; ++x) n_units_entries += in_units[x];
      // user-major: x = user, y = item, tile = (class, item range)
      {
        const std::function<int32_t(int64_t)> xr = [&](int64_t e) { return ent_user[e]; };
        const std::function<int32_t(int64_t)> yr = [&](int64_t e) { return L.col[e]; };
        int64_t rows = std::max<int64_t>(1, std::min<int64_t>(p.tile_rows_item, M));
        std::vector<int64_t> by_x(static_cast<size_t>(nb)), last;
        std::iota(by_x.begin(), by_x.end(), int64_t(0));  // canonical is sorted by user
        for (;;) {
          const int64_t nt = (M + rows - 1) / rows;
          const std::function<int32_t(int64_t)> tl = [&, rows, nt](int64_t e) {
            return static_cast<int32_t>(ucls[ent_user[e]] * nt + L.col[e] / rows);
          };
          if (rows >= M || count_runs(nb, by_x, xr, tl, nt * p.nclass, in_units, last) * min_avg <= n_units_entries)
            break;
          rows *= 2;
        }
        const int64_t nt = (M + rows - 1) / rows;
        const std::function<int32_t(int64_t)> tl = [&, rows, nt](int64_t e) {
          return static_cast<int32_t>(ucls[ent_user[e]] * nt + L.col[e] / rows);
        };
        const std::function<int32_t(int64_t)> ct = [nt](int64_t t) { return static_cast<int32_t>(t / nt); };
        build_units(nb, N, nt * p.nclass, xr, yr, tl, ct, L.val, p.unit_max, in_units, extra_u, base_u, L.by_user);
        assign_cell_rows(L.cells_user, base_u);
        L.partial_rows_user = L.by_user.x_pp[N];
      }
      // item-major: x = item, y = user, tile = class-pure user range
      {
        const std::function<int32_t(int64_t)> xr = [&](int64_t e) { return L.col[e]; };
        const std::function<int32_t(int64_t)> yr = [&](int64_t e) { return ent_user[e]; };
        std::vector<int64_t> by_x(static_cast<size_t>(nb)), tmp(static_cast<size_t>(nb)), last;
        std::iota(tmp.begin(), tmp.end(), int64_t(0));
        counting_pass(tmp, by_x, M, xr);
        std::vector<int64_t>().swap(tmp);
        int64_t rows = std::max<int64_t>(1, std::min<int64_t>(p.tile_rows_user, N));
        std::vector<int64_t> cls_base;
        auto tiles_for = [&](int64_t r) {
          cls_base.assign(static_cast<size_t>(p.nclass) + 1, 0);
          for (int32_t c = 0; c < p.nclass; ++c) cls_base[c + 1] = cls_base[c] + (in_cls[c] + r - 1) / r;
          return cls_base[p.nclass];
        };
        for (;;) {
          const int64_t nt = tiles_for(rows);
          const std::function<int32_t(int64_t)> tl = [&, rows](int64_t e) {
            const int32_t u = ent_user[e];
            return static_cast<int32_t>(cls_base[ucls[u]] + rank_in_cls[u] / rows);
          };
          if (rows >= N ||
              count_runs(nb, by_x, xr, tl, std::max<int64_t>(nt, 1), in_units, last) * min_avg <= n_units_entries)
            break;
          rows *= 2;
        }
        const int64_t nt = std::max<int64_t>(tiles_for(rows), 1);
        const std::function<int32_t(int64_t)> tl = [&, rows](int64_t e) {
          const int32_t u = ent_user[e];
          return static_cast<int32_t>(cls_base[ucls[u]] + rank_in_cls[u] / rows);
        };
        std::vector<int32_t> tile_cls(static_cast<size_t>(nt), 0);
        for (int32_t c = 0; c < p.nclass; ++c)
          for (int64_t t = cls_base[c]; t < cls_base[c + 1]; ++t) tile_cls[t] = c;
        const std::function<int32_t(int64_t)> ct = [&](int64_t t) { return tile_cls[t]; };
        build_units(nb, M, nt, xr, yr, tl, ct, L.val, p.unit_max, in_units, extra_i, base_i, L.by_item);
        assign_cell_rows(L.cells_item, base_i);
        L.partial_rows_item = L.by_item.x_pp[M];
      }
    }
    return 0;
  } catch (const std::bad_alloc &) {
    err = "host allocation failed while building the layout";
    return -2;
  }
}

}  // namespace psmf
