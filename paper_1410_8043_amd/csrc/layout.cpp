// Host-side integer layout (see layout.h).
#include "layout.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <exception>
#include <functional>
#include <limits>
#include <new>
#include <numeric>
#include <thread>
#include <tuple>

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
  U.sole.assign(static_cast<size_t>(nx), 0);
  for (int64_t x = 0; x < nx; ++x) U.sole[x] = ucnt[x] == 1 && (extra.empty() || extra[x] == 0);
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

// number of distinct (x, tile) runs for a tile function (entries sorted by x already);
// threads take slices of by_x cut at changes of x, so no run spans two slices
int64_t count_runs(int64_t nb, const std::vector<int64_t> &by_x, const std::function<int32_t(int64_t)> &xrow,
                   const std::function<int32_t(int64_t)> &tile, int64_t ntiles, const std::vector<uint8_t> &in_units,
                   int threads) {
  const int T = nb >= (1 << 20) ? std::max(1, threads) : 1;
  std::vector<int64_t> cut(static_cast<size_t>(T) + 1, nb);
  cut[0] = 0;
  for (int t = 1; t < T; ++t) {
    int64_t e = std::max(cut[t - 1], nb * t / T);
    while (e > cut[t - 1] && e < nb && xrow(by_x[e]) == xrow(by_x[e - 1])) ++e;
    cut[t] = e;
  }
  std::vector<int64_t> runs(static_cast<size_t>(T), 0);
  auto work = [&](int t) {
    std::vector<int64_t> last(static_cast<size_t>(ntiles), -1);
    for (int64_t e = cut[t]; e < cut[t + 1]; ++e) {
      if (!in_units[by_x[e]]) continue;
      const int64_t x = xrow(by_x[e]);
      const int32_t tl = tile(by_x[e]);
      if (last[tl] != x) {
        last[tl] = x;
        ++runs[t];
      }
    }
  };
  if (T == 1) {
    work(0);
  } else {
    std::vector<std::thread> pool;
    for (int t = 0; t < T; ++t) pool.emplace_back(work, t);
    for (auto &th : pool) th.join();
  }
  int64_t total = 0;
  for (int64_t r : runs) total += r;
  return total;
}

// Append the ratings [lo, hi) of the (already ordered) list `ents` as one 8-aligned run,
// leaving out the entries e with skip[e] != 0 (those stored in dense tiles).
void append_run(CellSet &C, const std::vector<int64_t> &ents, int64_t lo, int64_t hi,
                const std::function<int32_t(int64_t)> &local, const std::vector<float> &val,
                const std::vector<uint8_t> &skip) {
  const int64_t beg = static_cast<int64_t>(C.ly.size());
  C.run_beg.push_back(static_cast<int32_t>(beg));
  int64_t len = 0;
  for (int64_t q = lo; q < hi; ++q) {
    if (skip[ents[q]]) continue;
    C.ly.push_back(static_cast<uint16_t>(local(ents[q])));
    C.lv.push_back(val[ents[q]]);
    ++len;
  }
  C.run_len.push_back(static_cast<int32_t>(len));
  while (C.ly.size() % kUnitAlign) {
    C.ly.push_back(0);
    C.lv.push_back(0.f);
  }
  C.nnz += len;
}

void empty_run(CellSet &C) {
  C.run_beg.push_back(static_cast<int32_t>(C.ly.size()));
  C.run_len.push_back(0);
}

// User-major cells: heavy users of one class, sorted by degree, ng per cell; steps are
// item ranges of ts items; the item space is cut into R ranges of steps so that there are
// about cell_target cells.  Each heavy user owns R partial rows.
void build_user_cells(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                      const std::vector<uint8_t> &heavy, const std::vector<int64_t> &deg,
                      const std::vector<uint8_t> &in_dense, CellSet &C, std::vector<int64_t> &extra) {
  const int64_t N = p.users, M = p.items, ts = p.cell_rows, ng = p.cell_groups;
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  if (extra.empty()) extra.assign(static_cast<size_t>(N), 0);
  std::vector<std::vector<int32_t>> by_cls(static_cast<size_t>(p.nclass));
  for (int64_t i = 0; i < N; ++i)
    if (heavy[i]) by_cls[ucls[i]].push_back(static_cast<int32_t>(i));
  int64_t groups = 0;
  for (auto &v : by_cls) {
    std::stable_sort(v.begin(), v.end(), [&](int32_t a, int32_t b) { return deg[a] > deg[b]; });
    groups += (static_cast<int64_t>(v.size()) + ng - 1) / ng;
  }
  if (groups == 0) return;
  const int64_t nsub = (M + ts - 1) / ts;
  const int64_t R = std::max<int64_t>(1, std::min<int64_t>(nsub / std::max(1, p.min_cell_steps),
                                                            (p.cell_target + groups - 1) / groups));
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
            append_run(C, ents, lo, hi, local, L.val, in_dense);
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
                      const std::vector<uint8_t> &heavy, const std::vector<int32_t> &ent_user,
                      const std::vector<uint8_t> &in_dense, CellSet &C, std::vector<int64_t> &extra) {
  const int64_t N = p.users, M = p.items, ts = p.cell_rows, ng = p.cell_groups;
  const int64_t nb = static_cast<int64_t>(L.col.size());
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  if (extra.empty()) extra.assign(static_cast<size_t>(M), 0);
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
    if (heavy[ent_user[e]] && !in_dense[e]) a.push_back(e);
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
    const int64_t Rc = std::max<int64_t>(1, std::min<int64_t>(R, nsub[c] / std::max(1, p.min_cell_steps)));
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
            append_run(C, a, o[st], o[st + 1], local, L.val, in_dense);
          }
        }
        C.cell_step_ptr.push_back(static_cast<int32_t>(C.cell_steps.size()));
        for (int64_t q = 0; q < ng && g0 + q < static_cast<int64_t>(items.size()); ++q) extra[items[g0 + q]] += 1;
      }
    }
  }
}

// Light users x hot items, user-major: light users of one class with hot ratings, sorted
// by their hot-rating count, ng per cell; the steps are the hot sub-tiles (hot items in
// popularity order, ts per sub-tile).  Each such user owns one more partial row.
void build_user_cells_hot(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                          const std::vector<uint8_t> &heavy, const std::vector<int32_t> &hot_pos,
                          const std::vector<int32_t> &hot_items, const std::vector<uint8_t> &in_dense, CellSet &C,
                          std::vector<int64_t> &extra) {
  const int64_t N = p.users, ts = p.cell_rows, ng = p.cell_groups;
  const int64_t nhot = static_cast<int64_t>(hot_items.size());
  if (nhot == 0) return;
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  if (extra.empty()) extra.assign(static_cast<size_t>(N), 0);
  const int64_t nsub = (nhot + ts - 1) / ts;
  const int32_t step0 = static_cast<int32_t>(C.step_rows.size() / ts);
  for (int64_t t = 0; t < nsub * ts; ++t) C.step_rows.push_back(t < nhot ? hot_items[t] : -1);
  // each light user's hot entries, sorted by hot position (sub-tile, then place)
  std::vector<std::vector<int32_t>> by_cls(static_cast<size_t>(p.nclass));
  std::vector<int64_t> hot_cnt(static_cast<size_t>(N), 0);
  for (int64_t i = 0; i < N; ++i) {
    if (heavy[i]) continue;
    for (int64_t e = L.row_ptr[i]; e < L.row_ptr[i + 1]; ++e) hot_cnt[i] += hot_pos[L.col[e]] >= 0 && !in_dense[e];
    if (hot_cnt[i] > 0) by_cls[ucls[i]].push_back(static_cast<int32_t>(i));
  }
  std::vector<int64_t> ents;
  const std::function<int32_t(int64_t)> local = [&](int64_t e) { return static_cast<int32_t>(hot_pos[L.col[e]] % ts); };
  if (C.cell_step_ptr.empty()) C.cell_step_ptr.push_back(0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    auto &us = by_cls[c];
    std::stable_sort(us.begin(), us.end(), [&](int32_t a, int32_t b) { return hot_cnt[a] > hot_cnt[b]; });
    for (size_t g0 = 0; g0 < us.size(); g0 += static_cast<size_t>(ng)) {
      C.cell_cls.push_back(c);
      for (int64_t q = 0; q < ng; ++q) {
        const size_t k = g0 + static_cast<size_t>(q);
        C.cell_x.push_back(k < us.size() ? us[k] : -1);
        C.cell_out.push_back(-1);
      }
      // per member: its hot entries grouped by sub-tile
      std::vector<std::vector<int64_t>> mine(static_cast<size_t>(ng));
      for (int64_t q = 0; q < ng && g0 + q < us.size(); ++q) {
        const int32_t u = us[g0 + q];
        for (int64_t e = L.row_ptr[u]; e < L.row_ptr[u + 1]; ++e)
          if (hot_pos[L.col[e]] >= 0 && !in_dense[e]) mine[q].push_back(e);
        std::stable_sort(mine[q].begin(), mine[q].end(),
                         [&](int64_t a, int64_t b) { return hot_pos[L.col[a]] < hot_pos[L.col[b]]; });
      }
      for (int64_t st = 0; st < nsub; ++st) {
        C.cell_steps.push_back(step0 + static_cast<int32_t>(st));
        for (int64_t q = 0; q < ng; ++q) {
          if (g0 + q >= us.size()) { empty_run(C); continue; }
          const auto &m = mine[q];
          const auto lo = std::lower_bound(m.begin(), m.end(), st * ts,
                                           [&](int64_t e, int64_t v) { return hot_pos[L.col[e]] < v; });
          const auto hi = std::lower_bound(m.begin(), m.end(), (st + 1) * ts,
                                           [&](int64_t e, int64_t v) { return hot_pos[L.col[e]] < v; });
          append_run(C, m, lo - m.begin(), hi - m.begin(), local, L.val, in_dense);
        }
      }
      C.cell_step_ptr.push_back(static_cast<int32_t>(C.cell_steps.size()));
      for (size_t k = g0; k < std::min(us.size(), g0 + static_cast<size_t>(ng)); ++k) extra[us[k]] += 1;
    }
  }
}

// Light users x hot items, item-major: hot items in popularity order, ng per cell; for
// each class the steps are consecutive ranges of ts of its light users that rated a hot
// item (in id order), cut into ranges so that there are about cell_target cells.  Each
// hot item owns one more partial row per (class, range).
void build_item_cells_hot(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                          const std::vector<uint8_t> &heavy, const std::vector<int32_t> &ent_user,
                          const std::vector<int32_t> &hot_pos, const std::vector<int32_t> &hot_items,
                          const std::vector<uint8_t> &in_dense, CellSet &C, std::vector<int64_t> &extra) {
  const int64_t N = p.users, M = p.items, ts = p.cell_rows, ng = p.cell_groups;
  const int64_t nb = static_cast<int64_t>(L.col.size());
  const int64_t nhot = static_cast<int64_t>(hot_items.size());
  if (nhot == 0) return;
  C.ts = static_cast<int32_t>(ts);
  C.ng = static_cast<int32_t>(ng);
  if (extra.empty()) extra.assign(static_cast<size_t>(M), 0);
  // light users with hot ratings, ranked within their class in id order
  std::vector<uint8_t> has_hot(static_cast<size_t>(N), 0);
  std::vector<int64_t> a, b;
  for (int64_t e = 0; e < nb; ++e)
    if (!heavy[ent_user[e]] && hot_pos[L.col[e]] >= 0 && !in_dense[e]) {
      a.push_back(e);
      has_hot[ent_user[e]] = 1;
    }
  if (a.empty()) return;
  std::vector<int64_t> rank(static_cast<size_t>(N), -1), nlight(static_cast<size_t>(p.nclass), 0);
  for (int64_t i = 0; i < N; ++i)
    if (has_hot[i]) rank[i] = nlight[ucls[i]]++;
  std::vector<int64_t> nsub(static_cast<size_t>(p.nclass)), sub_base(static_cast<size_t>(p.nclass) + 1, 0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    nsub[c] = (nlight[c] + ts - 1) / ts;
    sub_base[c + 1] = sub_base[c] + nsub[c];
  }
  const int32_t step0 = static_cast<int32_t>(C.step_rows.size() / ts);
  C.step_rows.resize(C.step_rows.size() + static_cast<size_t>(sub_base[p.nclass] * ts), -1);
  for (int64_t i = 0; i < N; ++i)
    if (has_hot[i])
      C.step_rows[(step0 + sub_base[ucls[i]] + rank[i] / ts) * ts + rank[i] % ts] = static_cast<int32_t>(i);
  // entries by (hot position, class, user): canonical is (user, item)
  b.resize(a.size());
  counting_pass(a, b, p.nclass, [&](int64_t e) { return ucls[ent_user[e]]; });
  counting_pass(b, a, nhot, [&](int64_t e) { return hot_pos[L.col[e]]; });
  // boundaries of (hot position h, class c, sub-tile st)
  std::vector<int64_t> hc_base(static_cast<size_t>(nhot * p.nclass) + 1, 0);
  for (int64_t h = 0; h < nhot; ++h)
    for (int32_t c = 0; c < p.nclass; ++c) hc_base[h * p.nclass + c + 1] = hc_base[h * p.nclass + c] + nsub[c] + 1;
  std::vector<int64_t> bnd(static_cast<size_t>(hc_base[nhot * p.nclass]), 0);
  {
    int64_t e = 0;
    const int64_t na = static_cast<int64_t>(a.size());
    for (int64_t h = 0; h < nhot; ++h)
      for (int32_t c = 0; c < p.nclass; ++c) {
        int64_t *o = bnd.data() + hc_base[h * p.nclass + c];
        for (int64_t st = 0; st < nsub[c]; ++st) {
          o[st] = e;
          while (e < na && hot_pos[L.col[a[e]]] == h && ucls[ent_user[a[e]]] == c && rank[ent_user[a[e]]] / ts == st) ++e;
        }
        o[nsub[c]] = e;
      }
  }
  // Hot items differ a lot in popularity, and a cell step lasts as long as its longest run:
  // an item of class weight w gets m = max(1, round(w / w_med)) lane groups ("slots"), slot
  // r taking the users whose place in the sub-tile is r mod m; slots are sorted by weight
  // per slot and packed ng to a cell.
  struct Slot { int32_t h, r, m; int64_t w; };
  std::vector<std::vector<Slot>> slots(static_cast<size_t>(p.nclass));
  int64_t cells_per_range = 0;
  for (int32_t c = 0; c < p.nclass; ++c) {
    if (nsub[c] == 0) continue;
    std::vector<int64_t> wts;
    for (int64_t h = 0; h < nhot; ++h) {
      const int64_t *o = bnd.data() + hc_base[h * p.nclass + c];
      if (o[nsub[c]] > o[0]) wts.push_back(o[nsub[c]] - o[0]);
    }
    if (wts.empty()) continue;
    std::vector<int64_t> sorted_w = wts;
    std::nth_element(sorted_w.begin(), sorted_w.begin() + sorted_w.size() / 2, sorted_w.end());
    const int64_t w_med = std::max<int64_t>(1, sorted_w[sorted_w.size() / 2]);
    for (int64_t h = 0; h < nhot; ++h) {
      const int64_t *o = bnd.data() + hc_base[h * p.nclass + c];
      const int64_t w = o[nsub[c]] - o[0];
      if (w == 0) continue;
      const int32_t m = static_cast<int32_t>(std::min<int64_t>(ts, std::max<int64_t>(1, (2 * w + w_med) / (2 * w_med))));
      for (int32_t r = 0; r < m; ++r) slots[c].push_back({static_cast<int32_t>(h), r, m, w});
    }
    std::stable_sort(slots[c].begin(), slots[c].end(),
                     [](const Slot &x, const Slot &y) { return x.w * y.m > y.w * x.m; });
    cells_per_range += (static_cast<int64_t>(slots[c].size()) + ng - 1) / ng;
  }
  if (cells_per_range == 0) return;
  const int64_t R = std::max<int64_t>(1, (p.cell_target + cells_per_range - 1) / cells_per_range);
  const std::function<int32_t(int64_t)> local = [&](int64_t e) { return static_cast<int32_t>(rank[ent_user[e]] % ts); };
  if (C.cell_step_ptr.empty()) C.cell_step_ptr.push_back(0);
  std::vector<int64_t> run;
  for (int32_t c = 0; c < p.nclass; ++c) {
    if (slots[c].empty()) continue;
    const auto &sl = slots[c];
    const int64_t ns = static_cast<int64_t>(sl.size());
    const int64_t Rc = std::max<int64_t>(1, std::min<int64_t>(R, nsub[c] / std::max(1, p.min_cell_steps)));
    for (int64_t g0 = 0; g0 < ns; g0 += ng) {
      for (int64_t r = 0; r < Rc; ++r) {
        const int64_t s0 = r * nsub[c] / Rc, s1 = (r + 1) * nsub[c] / Rc;
        C.cell_cls.push_back(c);
        for (int64_t q = 0; q < ng; ++q) {
          C.cell_x.push_back(g0 + q < ns ? hot_items[sl[g0 + q].h] : -1);
          C.cell_out.push_back(-1);
        }
        for (int64_t st = s0; st < s1; ++st) {
          C.cell_steps.push_back(step0 + static_cast<int32_t>(sub_base[c] + st));
          for (int64_t q = 0; q < ng; ++q) {
            if (g0 + q >= ns) { empty_run(C); continue; }
            const Slot &z = sl[g0 + q];
            const int64_t *o = bnd.data() + hc_base[static_cast<int64_t>(z.h) * p.nclass + c];
            run.clear();
            for (int64_t e = o[st]; e < o[st + 1]; ++e)
              if (local(a[e]) % z.m == z.r) run.push_back(a[e]);
            append_run(C, run, 0, static_cast<int64_t>(run.size()), local, L.val, in_dense);
          }
        }
        C.cell_step_ptr.push_back(static_cast<int32_t>(C.cell_steps.size()));
        for (int64_t q = 0; q < ng && g0 + q < ns; ++q) extra[hot_items[sl[g0 + q].h]] += 1;
      }
    }
  }
}

// cell_out of every used (cell, group), then of every used (dense cell, row): the next of
// x's rows from cell_base[x] on
void assign_cell_rows(CellSet &C, DenseSet &D, std::vector<int64_t> cell_base) {
  for (size_t k = 0; k < C.cell_x.size(); ++k)
    if (C.cell_x[k] >= 0) C.cell_out[k] = static_cast<int32_t>(cell_base[C.cell_x[k]]++);
  for (size_t k = 0; k < D.cell_x.size(); ++k)
    if (D.cell_x[k] >= 0) D.cell_out[k] = static_cast<int32_t>(cell_base[D.cell_x[k]]++);
}

// Dense tiles of one block (see DenseSet) and the cells of both directions.  Users of
// each class are ranked by their rating count in the block and items by theirs (ties by
// id); tile (c, ut, it) = users of class c at ranks [64 ut, 64 ut + 64) x items at ranks
// [64 it, 64 it + 64).  A tile with at least dense_min ratings is dense: its entries go
// to the dense blocks (of duplicate (user, item) pairs only the first, the others stay
// with the sparse part) and in_dense[e] is set for them.  A user or item row owns one
// partial row per dense cell it belongs to (extra_u / extra_i).
void build_dense(const LayoutParams &p, const BlockLayout &L, const std::vector<int32_t> &ucls,
                 std::vector<uint8_t> &in_dense, DenseSet &DU, DenseSet &DI, std::vector<int64_t> &extra_u,
                 std::vector<int64_t> &extra_i) {
  const int64_t N = p.users, M = p.items, T = kDenseRows;
  if (p.dense_min <= 0 || L.nnz == 0) return;
  const int64_t nit = (M + T - 1) / T;
  std::vector<int32_t> item_at(static_cast<size_t>(M)), irank(static_cast<size_t>(M));
  std::iota(item_at.begin(), item_at.end(), 0);
  std::stable_sort(item_at.begin(), item_at.end(), [&](int32_t x, int32_t y) { return L.icount[x] > L.icount[y]; });
  for (int64_t r = 0; r < M; ++r) irank[item_at[r]] = static_cast<int32_t>(r);
  std::vector<std::vector<int32_t>> ulist(static_cast<size_t>(p.nclass));
  for (int64_t i = 0; i < N; ++i)
    if (L.ucount[i] > 0) ulist[ucls[i]].push_back(static_cast<int32_t>(i));
  // dense item tiles of each (class, user tile), ascending
  struct UTile { int32_t c, ut; std::vector<int32_t> its; };
  std::vector<UTile> utiles;
  std::vector<int64_t> cnt(static_cast<size_t>(nit), 0);
  for (int32_t c = 0; c < p.nclass; ++c) {
    auto &us = ulist[c];
    std::stable_sort(us.begin(), us.end(), [&](int32_t a, int32_t b) { return L.ucount[a] > L.ucount[b]; });
    for (int64_t u0 = 0; u0 < static_cast<int64_t>(us.size()); u0 += T) {
      const int64_t u1 = std::min<int64_t>(u0 + T, static_cast<int64_t>(us.size()));
      int64_t total = 0;
      for (int64_t q = u0; q < u1; ++q) total += L.ucount[us[q]];
      if (total < p.dense_min) break;  // later tiles of the class hold fewer ratings
      std::fill(cnt.begin(), cnt.end(), 0);
      for (int64_t q = u0; q < u1; ++q)
        for (int64_t e = L.row_ptr[us[q]]; e < L.row_ptr[us[q] + 1]; ++e) cnt[irank[L.col[e]] / T] += 1;
      UTile t{c, static_cast<int32_t>(u0 / T), {}};
      for (int64_t it = 0; it < nit; ++it)
        if (cnt[it] >= p.dense_min) t.its.push_back(static_cast<int32_t>(it));
      if (!t.its.empty()) utiles.push_back(std::move(t));
    }
  }
  int64_t ntiles = 0;
  for (const auto &t : utiles) ntiles += static_cast<int64_t>(t.its.size());
  if (ntiles == 0) return;
  // entries of the dense tiles
  std::vector<uint8_t> dense_it(static_cast<size_t>(nit), 0);
  for (const auto &t : utiles) {
    for (int32_t it : t.its) dense_it[it] = 1;
    const auto &us = ulist[t.c];
    for (int64_t q = int64_t(t.ut) * T; q < std::min<int64_t>((int64_t(t.ut) + 1) * T, us.size()); ++q)
      for (int64_t e = L.row_ptr[us[q]]; e < L.row_ptr[us[q] + 1]; ++e)
        if (dense_it[irank[L.col[e]] / T] && (e == L.row_ptr[us[q]] || L.col[e - 1] != L.col[e])) in_dense[e] = 1;
    for (int32_t it : t.its) dense_it[it] = 0;
  }
  const int64_t per_cell = std::max<int64_t>(std::max(1, p.min_cell_steps),
                                             (ntiles + p.dense_target - 1) / std::max(1, p.dense_target));
  // step index of every dense tile in each direction: tile t of utiles[u] is tile_base[u] + t
  std::vector<int64_t> tile_base(utiles.size() + 1, 0);
  for (size_t u = 0; u < utiles.size(); ++u) tile_base[u + 1] = tile_base[u] + static_cast<int64_t>(utiles[u].its.size());
  std::vector<int64_t> step_u(static_cast<size_t>(ntiles)), step_i(static_cast<size_t>(ntiles));
  // A cell = (x tile, class, a run of at most per_cell dense y tiles, given as tile ids);
  // cells are emitted longest first.
  struct Seg { int32_t c, xt; std::vector<int32_t> ys; std::vector<int64_t> tiles; };
  auto cut = [&](std::vector<Seg> &segs, int32_t c, int32_t xt, const std::vector<int32_t> &ys,
                 const std::vector<int64_t> &tiles) {
    const int64_t n = static_cast<int64_t>(ys.size());
    const int64_t parts = (n + per_cell - 1) / per_cell;
    for (int64_t r = 0; r < parts; ++r)
      segs.push_back({c, xt, std::vector<int32_t>(ys.begin() + r * n / parts, ys.begin() + (r + 1) * n / parts),
                      std::vector<int64_t>(tiles.begin() + r * n / parts, tiles.begin() + (r + 1) * n / parts)});
  };
  auto emit = [&](DenseSet &D, std::vector<Seg> &segs, bool user_major, std::vector<int64_t> &extra,
                  std::vector<int64_t> &step_of) {
    std::stable_sort(segs.begin(), segs.end(), [](const Seg &a, const Seg &b) { return a.ys.size() > b.ys.size(); });
    D.cell_step_ptr.assign(1, 0);
    D.step_rows.reserve(static_cast<size_t>(ntiles * T));
    int64_t k = 0;
    for (const auto &g : segs) {
      D.cell_cls.push_back(g.c);
      for (int64_t q = 0; q < T; ++q) {
        int32_t x = -1;
        const int64_t pos = int64_t(g.xt) * T + q;
        if (user_major) x = pos < static_cast<int64_t>(ulist[g.c].size()) ? ulist[g.c][pos] : -1;
        else x = pos < M ? item_at[pos] : -1;
        D.cell_x.push_back(x);
        D.cell_out.push_back(-1);
        if (x >= 0) extra[x] += 1;
      }
      for (size_t t = 0; t < g.ys.size(); ++t) {
        for (int64_t q = 0; q < T; ++q) {
          const int64_t pos = int64_t(g.ys[t]) * T + q;
          if (user_major) D.step_rows.push_back(pos < M ? item_at[pos] : -1);
          else D.step_rows.push_back(pos < static_cast<int64_t>(ulist[g.c].size()) ? ulist[g.c][pos] : -1);
        }
        step_of[g.tiles[t]] = k++;
      }
      D.cell_step_ptr.push_back(static_cast<int32_t>(k));
    }
    D.dval.assign(static_cast<size_t>(k * kDenseTile), std::numeric_limits<float>::quiet_NaN());
  };
  if (extra_u.empty()) extra_u.assign(static_cast<size_t>(N), 0);
  if (extra_i.empty()) extra_i.assign(static_cast<size_t>(M), 0);
  {
    std::vector<Seg> segs;
    for (size_t u = 0; u < utiles.size(); ++u) {
      std::vector<int64_t> ids(utiles[u].its.size());
      std::iota(ids.begin(), ids.end(), tile_base[u]);
      cut(segs, utiles[u].c, utiles[u].ut, utiles[u].its, ids);
    }
    emit(DU, segs, true, extra_u, step_u);
  }
  {
    // (item tile, class) -> its dense user tiles, ascending
    std::vector<std::vector<std::vector<int32_t>>> uts(static_cast<size_t>(nit),
                                                        std::vector<std::vector<int32_t>>(static_cast<size_t>(p.nclass)));
    std::vector<std::vector<std::vector<int64_t>>> ids(static_cast<size_t>(nit),
                                                        std::vector<std::vector<int64_t>>(static_cast<size_t>(p.nclass)));
    for (size_t u = 0; u < utiles.size(); ++u)
      for (size_t t = 0; t < utiles[u].its.size(); ++t) {
        const int32_t it = utiles[u].its[t];
        uts[it][utiles[u].c].push_back(utiles[u].ut);
        ids[it][utiles[u].c].push_back(tile_base[u] + static_cast<int64_t>(t));
      }
    std::vector<Seg> segs;
    for (int64_t it = 0; it < nit; ++it)
      for (int32_t c = 0; c < p.nclass; ++c)
        if (!uts[it][c].empty()) cut(segs, c, static_cast<int32_t>(it), uts[it][c], ids[it][c]);
    emit(DI, segs, false, extra_i, step_i);
  }
  DU.step_twin.resize(static_cast<size_t>(ntiles));
  DI.step_twin.resize(static_cast<size_t>(ntiles));
  for (int64_t t = 0; t < ntiles; ++t) {
    DU.step_twin[step_u[t]] = static_cast<int32_t>(step_i[t]);
    DI.step_twin[step_i[t]] = static_cast<int32_t>(step_u[t]);
  }
  // the values: one pass over the rows of each dense user tile fills both directions' blocks
  // (user tiles write disjoint steps; parallel_for hands each thread the tiles u with
  // u * 2^16 in its range)
  parallel_for(p.threads, static_cast<int64_t>(utiles.size()) << 16, [&](int64_t lo, int64_t hi) {
    std::vector<int64_t> ku(static_cast<size_t>(nit), -1), ki(static_cast<size_t>(nit), -1);
    for (int64_t u = (lo + 0xffff) >> 16; u < (hi + 0xffff) >> 16; ++u) {
      const UTile &t = utiles[u];
      for (size_t x = 0; x < t.its.size(); ++x) {
        ku[t.its[x]] = step_u[tile_base[u] + x];
        ki[t.its[x]] = step_i[tile_base[u] + x];
      }
      const auto &us = ulist[t.c];
      for (int64_t q = int64_t(t.ut) * T; q < std::min<int64_t>((int64_t(t.ut) + 1) * T, us.size()); ++q) {
        const int32_t ul = static_cast<int32_t>(q - int64_t(t.ut) * T);
        for (int64_t e = L.row_ptr[us[q]]; e < L.row_ptr[us[q] + 1]; ++e) {
          if (!in_dense[e]) continue;
          const int32_t r = irank[L.col[e]];
          const int32_t it = r / static_cast<int32_t>(T), il = r - it * static_cast<int32_t>(T);
          DU.dval[static_cast<size_t>(ku[it] * kDenseTile + dense_frag_index(ul, il))] = L.val[e];
          DI.dval[static_cast<size_t>(ki[it] * kDenseTile + dense_frag_index(il, ul))] = L.val[e];
        }
      }
      for (int32_t it : t.its) ku[it] = ki[it] = -1;
    }
  });
  int64_t nd = 0;
  for (uint8_t f : in_dense) nd += f;
  DU.nnz = DI.nnz = nd;
}

// The sequential step's order of one block (see SeqSet).
void build_seq(const LayoutParams &p, BlockLayout &L, const std::vector<int32_t> &ent_user) {
  const int64_t nb = L.nnz, M = p.items, G = p.seq_groups, P = p.workers;
  SeqSet &S = L.seq;
  S.G = static_cast<int32_t>(G);
  auto ugroup = [&](int64_t e) { return (static_cast<int64_t>(ent_user[e]) / P) % G; };
  auto epoch = [&](int64_t e) { return ((L.col[e] % G) - ugroup(e) + G) % G; };
  // canonical positions, stably by user group, then by (sub-epoch, worker)
  std::vector<int64_t> a(static_cast<size_t>(nb)), b(static_cast<size_t>(nb));
  std::iota(a.begin(), a.end(), int64_t(0));
  counting_pass(a, b, G, ugroup);
  counting_pass(b, a, G * P, [&](int64_t e) { return epoch(e) * P + p.owner[ent_user[e]]; });
  std::vector<int64_t>().swap(b);
  S.user.resize(static_cast<size_t>(nb));
  S.item.resize(static_cast<size_t>(nb));
  S.val.resize(static_cast<size_t>(nb));
  S.flag.assign(static_cast<size_t>(nb), 0);
  S.canon.resize(static_cast<size_t>(nb));
  for (int64_t x = 0; x < nb; ++x) {
    const int64_t e = a[x];
    S.user[x] = ent_user[e];
    S.item[x] = L.col[e];
    S.val[x] = L.val[e];
    S.canon[x] = static_cast<int32_t>(e);
  }
  // chains: maximal runs of one (sub-epoch, worker, user group)
  S.epoch_chain.assign(static_cast<size_t>(G) + 1, 0);
  S.chain_beg.clear();
  S.chain_worker.clear();
  int64_t prev_key = -1;
  for (int64_t x = 0; x < nb; ++x) {
    const int64_t e = a[x];
    const int64_t key = (epoch(e) * P + p.owner[ent_user[e]]) * G + ugroup(e);
    if (key != prev_key) {
      S.chain_beg.push_back(x);
      S.chain_worker.push_back(p.owner[ent_user[e]]);
      S.epoch_chain[static_cast<size_t>(epoch(e)) + 1] += 1;
      prev_key = key;
    }
  }
  S.chain_beg.push_back(nb);
  for (int64_t t = 0; t < G; ++t) S.epoch_chain[t + 1] += S.epoch_chain[t];
  const int64_t nch = static_cast<int64_t>(S.chain_worker.size());
  // run starts, and the user's first run of the clock
  std::vector<uint8_t> seen(static_cast<size_t>(p.users), 0);
  for (int64_t ch = 0; ch < nch; ++ch)
    for (int64_t x = S.chain_beg[ch]; x < S.chain_beg[ch + 1]; ++x)
      if (x == S.chain_beg[ch] || S.user[x] != S.user[x - 1]) {
        S.flag[x] |= kSeqRunStart;
        if (!seen[S.user[x]]) {
          seen[S.user[x]] = 1;
          S.flag[x] |= kSeqFirstL;
        }
      }
  // items read again within the prefetch distance: the distance to the latest occurrence
  for (int64_t ch = 0; ch < nch; ++ch)
    for (int64_t x = S.chain_beg[ch]; x < S.chain_beg[ch + 1]; ++x)
      for (int64_t k = 1; k <= kSeqAhead && x - k >= S.chain_beg[ch]; ++k)
        if (S.item[x - k] == S.item[x]) {
          S.flag[x] |= static_cast<uint8_t>(k << kSeqDistShift);
          break;
        }
  // R flags: each worker's first rating of an item, scanning the worker's chains in order;
  // the (item, worker) pairs give the item worker lists, ascending in the worker
  std::vector<std::vector<int64_t>> chains_of(static_cast<size_t>(P));
  for (int64_t ch = 0; ch < nch; ++ch) chains_of[S.chain_worker[ch]].push_back(ch);
  std::vector<int32_t> stamp(static_cast<size_t>(M), -1);
  std::vector<int64_t> pair_item;
  std::vector<int32_t> pair_worker;
  for (int64_t w = 0; w < P; ++w)
    for (int64_t ch : chains_of[w])
      for (int64_t x = S.chain_beg[ch]; x < S.chain_beg[ch + 1]; ++x)
        if (stamp[S.item[x]] != w) {
          stamp[S.item[x]] = static_cast<int32_t>(w);
          S.flag[x] |= kSeqFirstR;
          pair_item.push_back(S.item[x]);
          pair_worker.push_back(static_cast<int32_t>(w));
        }
  S.item_wptr.assign(static_cast<size_t>(M) + 1, 0);
  for (int64_t j : pair_item) S.item_wptr[j + 1] += 1;
  for (int64_t j = 0; j < M; ++j) S.item_wptr[j + 1] += S.item_wptr[j];
  S.item_workers.resize(pair_item.size());
  std::vector<int64_t> fill(S.item_wptr.begin(), S.item_wptr.end() - 1);
  for (size_t q = 0; q < pair_item.size(); ++q) S.item_workers[fill[pair_item[q]]++] = pair_worker[q];
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
    // ---- canonical order (block, user, item, load index): a parallel stable counting sort
    // by (block, user) -- each thread scatters its own contiguous slice of the input, so
    // equal keys keep their load order -- then each (block, user) segment sorted by
    // (item, load index)
    std::vector<int64_t> a(static_cast<size_t>(n));
    const int64_t nkeys = static_cast<int64_t>(p.B) * N;
    if (nkeys > 4 * n + (int64_t(1) << 22)) {
      // many blocks and few ratings: stable LSD counting passes by item, user, block
      std::vector<int64_t> b(static_cast<size_t>(n));
      std::iota(a.begin(), a.end(), int64_t(0));
      counting_pass(a, b, M, [&](int64_t x) { return item[x]; });
      counting_pass(b, a, N, [&](int64_t x) { return user[x]; });
      if (p.B > 1) {
        counting_pass(a, b, p.B, [&](int64_t x) { return blk[x]; });
        a.swap(b);
      }
    } else {
      auto key = [&](int64_t t) { return (p.B > 1 ? static_cast<int64_t>(blk[t]) * N : 0) + user[t]; };
      const int T = n >= (1 << 20) ? std::max(1, std::min<int>(p.threads, static_cast<int>((int64_t(1) << 28) / (nkeys + 1)))) : 1;
      std::vector<std::vector<int64_t>> cnt(static_cast<size_t>(T));
      std::vector<int64_t> seg(static_cast<size_t>(nkeys) + 1, 0);
      std::vector<std::thread> pool;
      auto each = [&](auto &&fn) {
        if (T == 1) {
          fn(0);
          return;
        }
        pool.clear();
        for (int t = 0; t < T; ++t) pool.emplace_back([&fn, t] { fn(t); });
        for (auto &th : pool) th.join();
      };
      each([&](int t) {
        cnt[t].assign(static_cast<size_t>(nkeys), 0);
        for (int64_t x = n * t / T; x < n * (t + 1) / T; ++x) cnt[t][key(x)] += 1;
      });
      // exclusive offsets: key-major, thread-minor
      for (int64_t k = 0; k < nkeys; ++k) {
        int64_t tot = 0;
        for (int t = 0; t < T; ++t) {
          const int64_t c = cnt[t][k];
          cnt[t][k] = seg[k] + tot;
          tot += c;
        }
        seg[k + 1] = seg[k] + tot;
      }
      each([&](int t) {
        std::vector<int64_t> &o = cnt[t];
        for (int64_t x = n * t / T; x < n * (t + 1) / T; ++x) a[o[key(x)]++] = x;
      });
      std::vector<std::vector<int64_t>>().swap(cnt);
      each([&](int t) {
        for (int64_t k = nkeys * t / T; k < nkeys * (t + 1) / T; ++k)
          if (seg[k + 1] - seg[k] > 1)
            std::sort(a.begin() + seg[k], a.begin() + seg[k + 1], [&](int64_t x, int64_t y) {
              return item[x] != item[y] ? item[x] < item[y] : x < y;
            });
      });
    }
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
      parallel_for(p.threads, nb, [&](int64_t x0, int64_t x1) {
        for (int64_t x = x0; x < x1; ++x) ent_user[x] = user[L.perm[x]];
      });
      for (int64_t x = 0; x < nb; ++x) {
        const int32_t u = ent_user[x], j = L.col[x];
        L.ucount[u] += 1;
        L.icount[j] += 1;
        L.icount_cls[static_cast<size_t>(j) * p.nclass + ucls[u]] += 1;
      }
      L.row_ptr.assign(static_cast<size_t>(N) + 1, 0);
      for (int64_t i = 0; i < N; ++i) L.row_ptr[i + 1] = L.row_ptr[i] + L.ucount[i];
      if (p.seq_groups > 0) {
        build_seq(p, L, ent_user);
        continue;
      }

      // ---- dense tiles (matrix-core cells), then cells (staged through LDS) and units (the
      // rest) for the other ratings.  Heavy users' remaining ratings all go to cells; with
      // hot_steps > 0 so do the other users' ratings of the hot_steps * cell_rows most
      // rated items of the block.
      std::vector<uint8_t> in_dense(static_cast<size_t>(nb), 0);
      std::vector<int64_t> extra_u, extra_i, base_u, base_i;
      build_dense(p, L, ucls, in_dense, L.dense_user, L.dense_item, extra_u, extra_i);
      std::vector<int64_t> rem(L.ucount.begin(), L.ucount.end());  // ratings outside the dense tiles
      if (L.dense_user.nnz > 0)
        for (int64_t x = 0; x < nb; ++x) rem[ent_user[x]] -= in_dense[x];
      const bool use_cells = p.cell_rows > 0 && p.cell_groups > 0;
      std::vector<uint8_t> heavy(static_cast<size_t>(N), 0);
      if (use_cells)
        for (int64_t i = 0; i < N; ++i) heavy[i] = rem[i] > 0 && L.ucount[i] >= p.heavy_min;
      std::vector<int32_t> hot_items, hot_pos(static_cast<size_t>(M), -1);
      if (use_cells && p.hot_steps > 0) {
        hot_items.resize(static_cast<size_t>(M));
        std::iota(hot_items.begin(), hot_items.end(), 0);
        std::stable_sort(hot_items.begin(), hot_items.end(),
                         [&](int32_t x, int32_t y) { return L.icount[x] > L.icount[y]; });
        hot_items.resize(static_cast<size_t>(std::min<int64_t>(M, int64_t(p.hot_steps) * p.cell_rows)));
        while (!hot_items.empty() && L.icount[hot_items.back()] == 0) hot_items.pop_back();
        for (size_t h = 0; h < hot_items.size(); ++h) hot_pos[hot_items[h]] = static_cast<int32_t>(h);
      }
      std::vector<uint8_t> in_units(static_cast<size_t>(nb));
      for (int64_t x = 0; x < nb; ++x) in_units[x] = !in_dense[x] && !heavy[ent_user[x]] && hot_pos[L.col[x]] < 0;
      // ---- units.  Tiles start at the L2-sized row count and grow (x2) while the units
      // would average fewer than 16 ratings (each unit costs one partial row).
      const int64_t min_avg = 16;
      int64_t n_units_entries = 0;
      for (int64_t x = 0; x < nb; ++x) n_units_entries += in_units[x];
      // The two sweep directions only read the block's arrays: build them concurrently.
      std::exception_ptr user_side_error;
      std::thread user_side([&] {
      try {
      if (use_cells) {
        build_user_cells(p, L, ucls, heavy, rem, in_dense, L.cells_user, extra_u);
        build_user_cells_hot(p, L, ucls, heavy, hot_pos, hot_items, in_dense, L.cells_user, extra_u);
      }
      // user-major: x = user, y = item, tile = (class, item range)
      {
        const std::function<int32_t(int64_t)> xr = [&](int64_t e) { return ent_user[e]; };
        const std::function<int32_t(int64_t)> yr = [&](int64_t e) { return L.col[e]; };
        int64_t rows = std::max<int64_t>(1, std::min<int64_t>(p.tile_rows_item, M));
        std::vector<int64_t> by_x(static_cast<size_t>(nb));
        std::iota(by_x.begin(), by_x.end(), int64_t(0));  // canonical is sorted by user
        for (;;) {
          const int64_t nt = (M + rows - 1) / rows;
          const std::function<int32_t(int64_t)> tl = [&, rows, nt](int64_t e) {
            return static_cast<int32_t>(ucls[ent_user[e]] * nt + L.col[e] / rows);
          };
          if (rows >= M || count_runs(nb, by_x, xr, tl, nt * p.nclass, in_units, p.threads) * min_avg <= n_units_entries)
            break;
          rows *= 2;
        }
        const int64_t nt = (M + rows - 1) / rows;
        const std::function<int32_t(int64_t)> tl = [&, rows, nt](int64_t e) {
          return static_cast<int32_t>(ucls[ent_user[e]] * nt + L.col[e] / rows);
        };
        const std::function<int32_t(int64_t)> ct = [nt](int64_t t) { return static_cast<int32_t>(t / nt); };
        build_units(nb, N, nt * p.nclass, xr, yr, tl, ct, L.val, p.unit_max, in_units, extra_u, base_u, L.by_user);
        assign_cell_rows(L.cells_user, L.dense_user, base_u);
        L.partial_rows_user = L.by_user.x_pp[N];
      }
      } catch (...) {
        user_side_error = std::current_exception();
      }
      });
      struct Join {
        std::thread &t;
        ~Join() { if (t.joinable()) t.join(); }
      } join_user_side{user_side};
      if (use_cells) {
        build_item_cells(p, L, ucls, heavy, ent_user, in_dense, L.cells_item, extra_i);
        build_item_cells_hot(p, L, ucls, heavy, ent_user, hot_pos, hot_items, in_dense, L.cells_item, extra_i);
      }
      // item-major: x = item, y = user, tile = class-pure user range
      {
        const std::function<int32_t(int64_t)> xr = [&](int64_t e) { return L.col[e]; };
        const std::function<int32_t(int64_t)> yr = [&](int64_t e) { return ent_user[e]; };
        std::vector<int64_t> by_x(static_cast<size_t>(nb)), tmp(static_cast<size_t>(nb));
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
              count_runs(nb, by_x, xr, tl, std::max<int64_t>(nt, 1), in_units, p.threads) * min_avg <= n_units_entries)
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
        assign_cell_rows(L.cells_item, L.dense_item, base_i);
        L.partial_rows_item = L.by_item.x_pp[M];
      }
      user_side.join();
      if (user_side_error) std::rethrow_exception(user_side_error);
    }
    return 0;
  } catch (const std::bad_alloc &) {
    err = "host allocation failed while building the layout";
    return -2;
  }
}

namespace {

struct Triple {
  int32_t x, y;
  float v;
  bool operator<(const Triple &o) const {
    if (x != o.x) return x < o.x;
    if (y != o.y) return y < o.y;
    return std::memcmp(&v, &o.v, sizeof v) < 0;
  }
  bool operator==(const Triple &o) const { return x == o.x && y == o.y && std::memcmp(&v, &o.v, sizeof v) == 0; }
};

// one direction: `want` holds the block's (x, y, value) triples; ucls_of_entry(x, y) is the
// class the unit or cell must read
int check_direction(const char *dir, int64_t nx, int64_t ny, std::vector<Triple> want, const UnitSet &U,
                    const CellSet &C, const DenseSet &D, const std::function<int32_t(int32_t, int32_t)> &cls_of,
                    std::string &err) {
  auto bad = [&](const std::string &what) {
    err = std::string(dir) + ": " + what;
    return -1;
  };
  std::vector<Triple> got;
  got.reserve(want.size());
  const int64_t nunits = static_cast<int64_t>(U.unit_x.size());
  if (U.x_pp.size() != static_cast<size_t>(nx) + 1) return bad("x_pp has the wrong length");
  const int64_t nrows = U.x_pp[nx];
  std::vector<int32_t> written(static_cast<size_t>(nrows), 0);
  if (nunits % kWaveUnits) return bad("unit count is not a multiple of the wave size");
  for (int64_t w = 0; w < nunits; w += kWaveUnits)
    for (int64_t k = w + 1; k < w + kWaveUnits; ++k)
      if (U.unit_cls[k] != U.unit_cls[w]) return bad("units of one wave read different classes");
  for (int x = 0; x < kXcds; ++x)
    if (U.xcd_off[x] > U.xcd_off[x + 1] || U.xcd_off[x] % kWaveUnits) return bad("bad XCD chunk offsets");
  if (U.xcd_off[0] != 0 || U.xcd_off[kXcds] != nunits) return bad("XCD chunks do not cover the units");
  for (int64_t k = 0; k < nunits; ++k) {
    const int32_t x = U.unit_x[k], len = U.unit_len[k], out = U.unit_out[k];
    const int64_t beg = U.unit_beg[k];
    if (len == 0) {
      if (out != nrows) return bad("an empty unit does not write the spare row");
      continue;
    }
    if (x < 0 || x >= nx) return bad("unit row out of range");
    if (beg % kUnitAlign || beg + (len + kUnitAlign - 1) / kUnitAlign * kUnitAlign > static_cast<int64_t>(U.y.size()))
      return bad("unit entries misaligned or out of range");
    if (out < U.x_pp[x] || out >= U.x_pp[x + 1]) return bad("unit writes a partial row of another x");
    written[out] += 1;
    for (int64_t t = beg; t < beg + len; ++t) {
      const int32_t y = U.y[t];
      if (y < 0 || y >= ny) return bad("unit gathers a row out of range");
      if (cls_of(x, y) != U.unit_cls[k]) return bad("unit reads the slot of another class");
      got.push_back({x, y, U.val[t]});
    }
    for (int64_t t = beg + len; t < beg + (len + kUnitAlign - 1) / kUnitAlign * kUnitAlign; ++t)
      if (U.y[t] != 0 || U.val[t] != 0.f) return bad("unit padding is not (row 0, value 0)");
  }
  const int64_t ncells = static_cast<int64_t>(C.cell_cls.size());
  if (ncells > 0) {
    const int64_t ng = C.ng, ts = C.ts;
    if (C.cell_step_ptr.size() != static_cast<size_t>(ncells) + 1 || C.cell_x.size() != static_cast<size_t>(ncells * ng) ||
        C.cell_out.size() != C.cell_x.size() || C.run_beg.size() != C.cell_steps.size() * static_cast<size_t>(ng) ||
        C.run_len.size() != C.run_beg.size() || C.step_rows.size() % static_cast<size_t>(ts))
      return bad("cell arrays have inconsistent lengths");
    const int64_t nsteps = static_cast<int64_t>(C.step_rows.size()) / ts;
    for (int64_t c = 0; c < ncells; ++c) {
      if (C.cell_step_ptr[c] > C.cell_step_ptr[c + 1]) return bad("cell step pointers decrease");
      for (int64_t q = 0; q < ng; ++q) {
        const int32_t x = C.cell_x[c * ng + q], out = C.cell_out[c * ng + q];
        if (x >= nx) return bad("cell row out of range");
        if (x < 0 && out >= 0) return bad("an unused cell group writes a partial row");
        if (x >= 0) {
          if (out < U.x_pp[x] || out >= U.x_pp[x + 1]) return bad("cell writes a partial row of another x");
          written[out] += 1;
        }
        for (int64_t k = C.cell_step_ptr[c]; k < C.cell_step_ptr[c + 1]; ++k) {
          const int64_t st = C.cell_steps[k];
          if (st < 0 || st >= nsteps) return bad("cell step out of range");
          const int64_t beg = C.run_beg[k * ng + q], len = C.run_len[k * ng + q];
          if (x < 0 && len) return bad("an unused cell group has ratings");
          if (beg % kUnitAlign || beg + (len + kUnitAlign - 1) / kUnitAlign * kUnitAlign > static_cast<int64_t>(C.ly.size()))
            return bad("cell run misaligned or out of range");
          for (int64_t t = beg; t < beg + len; ++t) {
            if (C.ly[t] >= ts) return bad("cell index beyond the sub-tile");
            const int32_t y = C.step_rows[st * ts + C.ly[t]];
            if (y < 0 || y >= ny) return bad("cell rating reads an empty or out-of-range staged row");
            if (cls_of(x, y) != C.cell_cls[c]) return bad("cell reads the slot of another class");
            got.push_back({x, y, C.lv[t]});
          }
          for (int64_t t = beg + len; t < beg + (len + kUnitAlign - 1) / kUnitAlign * kUnitAlign; ++t)
            if (C.ly[t] != 0 || C.lv[t] != 0.f) return bad("cell padding is not (row 0, value 0)");
        }
      }
    }
    for (int32_t r : C.step_rows)
      if (r < -1 || r >= ny) return bad("staged row out of range");
  }
  const int64_t ndense = static_cast<int64_t>(D.cell_cls.size());
  if (ndense > 0) {
    const int64_t T = kDenseRows;
    const int64_t nsteps = static_cast<int64_t>(D.step_rows.size()) / T;
    if (D.cell_step_ptr.size() != static_cast<size_t>(ndense) + 1 || D.cell_x.size() != static_cast<size_t>(ndense * T) ||
        D.cell_out.size() != D.cell_x.size() || D.step_rows.size() % T ||
        D.dval.size() != static_cast<size_t>(nsteps * kDenseTile) || D.cell_step_ptr[0] != 0 ||
        D.cell_step_ptr[ndense] != nsteps)
      return bad("dense cell arrays have inconsistent lengths");
    for (int32_t r : D.step_rows)
      if (r < -1 || r >= ny) return bad("dense staged row out of range");
    int64_t held = 0;
    for (int64_t c = 0; c < ndense; ++c) {
      if (D.cell_step_ptr[c] > D.cell_step_ptr[c + 1]) return bad("dense cell step pointers decrease");
      for (int64_t q = 0; q < T; ++q) {
        const int32_t x = D.cell_x[c * T + q], out = D.cell_out[c * T + q];
        if (x >= nx) return bad("dense cell row out of range");
        if (x < 0 && out >= 0) return bad("an unused dense row writes a partial row");
        if (x >= 0) {
          if (out < U.x_pp[x] || out >= U.x_pp[x + 1]) return bad("dense cell writes a partial row of another x");
          written[out] += 1;
        }
      }
      for (int64_t k = D.cell_step_ptr[c]; k < D.cell_step_ptr[c + 1]; ++k)
        for (int32_t q = 0; q < T; ++q)
          for (int32_t t = 0; t < T; ++t) {
            const float v = D.dval[static_cast<size_t>(k * kDenseTile + dense_frag_index(q, t))];
            if (std::isnan(v)) continue;
            const int32_t x = D.cell_x[c * T + q], y = D.step_rows[k * T + t];
            if (x < 0 || y < 0) return bad("a dense rating sits on an empty row");
            if (cls_of(x, y) != D.cell_cls[c]) return bad("dense cell reads the slot of another class");
            got.push_back({x, y, v});
            ++held;
          }
    }
    if (held != D.nnz) return bad("dense cells hold " + std::to_string(held) + " ratings, not " + std::to_string(D.nnz));
  }
  for (int64_t r = 0; r < nrows; ++r)
    if (written[r] != 1) return bad("partial row " + std::to_string(r) + " is written " + std::to_string(written[r]) + " times");
  if (got.size() != want.size())
    return bad("units, cells and dense cells hold " + std::to_string(got.size()) + " ratings, the block " + std::to_string(want.size()));
  std::sort(got.begin(), got.end());
  std::sort(want.begin(), want.end());
  for (size_t t = 0; t < got.size(); ++t)
    if (!(got[t] == want[t])) return bad("units and cells do not hold the block's ratings exactly once");
  return 0;
}

// The two directions' dense steps pair up tile by tile (step_twin): the item-major twin of
// a user-major step stages the users the user-major cell holds, belongs to a cell that
// holds the items the user-major step stages, reads the same class and holds the same
// values, transposed.  The user-major sweep writes its residuals where the item-major
// sweep reads them on exactly this correspondence.
int check_dense_twins(const DenseSet &U, const DenseSet &I, std::string &err) {
  auto bad = [&](const std::string &what) {
    err = "dense twins: " + what;
    return -1;
  };
  const int64_t T = kDenseRows;
  const int64_t nu = static_cast<int64_t>(U.step_rows.size()) / T, ni = static_cast<int64_t>(I.step_rows.size()) / T;
  if (nu != ni || U.step_twin.size() != static_cast<size_t>(nu) || I.step_twin.size() != static_cast<size_t>(ni))
    return bad("step counts or twin maps disagree");
  std::vector<int64_t> cell_of_i(static_cast<size_t>(ni), -1);
  for (size_t c = 0; c + 1 < I.cell_step_ptr.size(); ++c)
    for (int64_t k = I.cell_step_ptr[c]; k < I.cell_step_ptr[c + 1]; ++k) cell_of_i[k] = static_cast<int64_t>(c);
  for (size_t c = 0; c + 1 < U.cell_step_ptr.size(); ++c)
    for (int64_t k = U.cell_step_ptr[c]; k < U.cell_step_ptr[c + 1]; ++k) {
      const int64_t t = U.step_twin[k];
      if (t < 0 || t >= ni || I.step_twin[t] != k) return bad("the twin map is not a bijection");
      const int64_t ci = cell_of_i[t];
      if (ci < 0 || I.cell_cls[ci] != U.cell_cls[c]) return bad("twin steps read different classes");
      for (int64_t q = 0; q < T; ++q) {
        if (I.step_rows[t * T + q] != U.cell_x[c * T + q]) return bad("a twin step stages other users");
        if (I.cell_x[ci * T + q] != U.step_rows[k * T + q]) return bad("a twin cell holds other items");
      }
      for (int32_t x = 0; x < T; ++x)
        for (int32_t y = 0; y < T; ++y) {
          const float a = U.dval[static_cast<size_t>(k * kDenseTile + dense_frag_index(x, y))];
          const float b = I.dval[static_cast<size_t>(t * kDenseTile + dense_frag_index(y, x))];
          if (std::memcmp(&a, &b, sizeof a) != 0) return bad("twin steps hold different values");
        }
    }
  return 0;
}

// the sequential step's order against its definition, recomputed entry by entry
int check_seq(const LayoutParams &p, const BlockLayout &L, std::string &err) {
  const SeqSet &S = L.seq;
  const int64_t nb = L.nnz, N = p.users, M = p.items, G = p.seq_groups, P = p.workers;
  auto bad = [&](const std::string &what) {
    err = "sequential order: " + what;
    return -1;
  };
  if (S.G != G || static_cast<int64_t>(S.user.size()) != nb || static_cast<int64_t>(S.canon.size()) != nb ||
      S.epoch_chain.size() != static_cast<size_t>(G) + 1 || S.chain_beg.size() != S.chain_worker.size() + 1)
    return bad("array sizes");
  std::vector<int32_t> cuser(static_cast<size_t>(nb));
  for (int64_t i = 0; i < N; ++i)
    for (int64_t e = L.row_ptr[i]; e < L.row_ptr[i + 1]; ++e) cuser[e] = static_cast<int32_t>(i);
  std::vector<uint8_t> used(static_cast<size_t>(nb), 0);
  auto skey = [&](int64_t x) {  // (sub-epoch, worker, user group, canonical position)
    const int64_t i = S.user[x], j = S.item[x], ug = (i / P) % G;
    return std::make_tuple(((j % G) - ug + G) % G, static_cast<int64_t>(p.owner[i]), ug, static_cast<int64_t>(S.canon[x]));
  };
  for (int64_t x = 0; x < nb; ++x) {
    const int64_t e = S.canon[x];
    if (e < 0 || e >= nb || used[e]) return bad("canonical positions are not a permutation");
    used[e] = 1;
    if (S.user[x] != cuser[e] || S.item[x] != L.col[e] || std::memcmp(&S.val[x], &L.val[e], sizeof(float)) != 0)
      return bad("rating " + std::to_string(x) + " differs from its canonical entry");
    if (x > 0 && !(skey(x - 1) < skey(x))) return bad("not sorted at " + std::to_string(x));
  }
  const int64_t nch = static_cast<int64_t>(S.chain_worker.size());
  if (S.chain_beg[0] != 0 || S.chain_beg[nch] != nb || S.epoch_chain[0] != 0 || S.epoch_chain[G] != nch)
    return bad("chain bounds");
  for (int64_t t = 0; t < G; ++t)
    for (int64_t ch = S.epoch_chain[t]; ch < S.epoch_chain[t + 1]; ++ch) {
      const int64_t lo = S.chain_beg[ch], hi = S.chain_beg[ch + 1];
      if (hi <= lo) return bad("empty chain");
      for (int64_t x = lo; x < hi; ++x)
        if (std::get<0>(skey(x)) != t || std::get<1>(skey(x)) != S.chain_worker[ch] ||
            std::get<2>(skey(x)) != std::get<2>(skey(lo)))
          return bad("chain " + std::to_string(ch) + " mixes strata");
      if (ch > S.epoch_chain[t] && std::get<1>(skey(lo)) == std::get<1>(skey(lo - 1)) &&
          std::get<2>(skey(lo)) == std::get<2>(skey(lo - 1)))
        return bad("chain " + std::to_string(ch) + " is not maximal");
    }
  // flags by brute force: run starts, first run of each user, first (worker, item) in order,
  // items repeated within the prefetch distance
  std::vector<int64_t> first_run(static_cast<size_t>(N), -1);
  std::vector<std::vector<int64_t>> first_r(static_cast<size_t>(M));
  std::vector<uint8_t> want(static_cast<size_t>(nb), 0);
  for (int64_t ch = 0; ch < nch; ++ch)
    for (int64_t x = S.chain_beg[ch]; x < S.chain_beg[ch + 1]; ++x) {
      const int32_t i = S.user[x];
      if (x == S.chain_beg[ch] || S.user[x - 1] != i) {
        want[x] |= kSeqRunStart;
        if (first_run[i] < 0) first_run[i] = x;
      }
      bool seen_before = false;
      for (int64_t y : first_r[S.item[x]])
        if (p.owner[S.user[y]] == p.owner[i]) seen_before = true;
      if (!seen_before) first_r[S.item[x]].push_back(x);
      int64_t dist = 0;
      for (int64_t y = S.chain_beg[ch]; y < x; ++y)
        if (S.item[y] == S.item[x] && x - y <= kSeqAhead) dist = x - y;  // the latest wins
      want[x] |= static_cast<uint8_t>(dist << kSeqDistShift);
    }
  for (int64_t i = 0; i < N; ++i)
    if (first_run[i] >= 0) want[first_run[i]] |= kSeqFirstL;
  for (int64_t j = 0; j < M; ++j)
    for (int64_t x : first_r[j]) want[x] |= kSeqFirstR;
  for (int64_t x = 0; x < nb; ++x)
    if (want[x] != S.flag[x]) return bad("flags of rating " + std::to_string(x));
  if (S.item_wptr.size() != static_cast<size_t>(M) + 1) return bad("item worker pointers");
  for (int64_t j = 0; j < M; ++j) {
    std::vector<int32_t> w;
    for (int64_t x : first_r[j]) w.push_back(p.owner[S.user[x]]);
    std::sort(w.begin(), w.end());
    if (S.item_wptr[j + 1] - S.item_wptr[j] != static_cast<int64_t>(w.size()) ||
        !std::equal(w.begin(), w.end(), S.item_workers.begin() + S.item_wptr[j]))
      return bad("workers of item " + std::to_string(j));
  }
  return 0;
}

}  // namespace

int check_layout(const LayoutParams &p, const BlockLayout &L, std::string &err) {
  const int64_t N = p.users, M = p.items;
  if (p.seq_groups > 0) return check_seq(p, L, err);
  std::vector<int32_t> ucls(static_cast<size_t>(N));
  for (int64_t i = 0; i < N; ++i) ucls[i] = p.cls_of_worker[p.owner[i]];
  std::vector<Triple> by_user, by_item;
  by_user.reserve(static_cast<size_t>(L.nnz));
  by_item.reserve(static_cast<size_t>(L.nnz));
  for (int64_t i = 0; i < N; ++i)
    for (int64_t e = L.row_ptr[i]; e < L.row_ptr[i + 1]; ++e) {
      by_user.push_back({static_cast<int32_t>(i), L.col[e], L.val[e]});
      by_item.push_back({L.col[e], static_cast<int32_t>(i), L.val[e]});
    }
  if (static_cast<int64_t>(by_user.size()) != L.nnz) {
    err = "row pointers do not cover the block";
    return -1;
  }
  const std::function<int32_t(int32_t, int32_t)> cu = [&](int32_t x, int32_t) { return ucls[x]; };
  const std::function<int32_t(int32_t, int32_t)> ci = [&](int32_t, int32_t y) { return ucls[y]; };
  if (check_direction("user-major", N, M, std::move(by_user), L.by_user, L.cells_user, L.dense_user, cu, err)) return -1;
  if (check_direction("item-major", M, N, std::move(by_item), L.by_item, L.cells_item, L.dense_item, ci, err)) return -1;
  if (check_dense_twins(L.dense_user, L.dense_item, err)) return -1;
  if (L.partial_rows_user != L.by_user.x_pp[N] || L.partial_rows_item != L.by_item.x_pp[M]) {
    err = "partial row counts disagree with the row offsets";
    return -1;
  }
  return 0;
}

}  // namespace psmf
