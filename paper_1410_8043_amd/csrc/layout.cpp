// Host-side integer layout (see layout.h).
#include "layout.h"

#include <algorithm>
#include <atomic>
#include <cmath>
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
      for (int64_t x = 0; x < nb; ++x) {
        const int64_t t = L.perm[x];
        L.ucount[user[t]] += 1;
        L.icount[item[t]] += 1;
        L.icount_cls[static_cast<size_t>(item[t]) * p.nclass + p.cls_of_worker[p.owner[user[t]]]] += 1;
      }
      L.row_ptr.assign(static_cast<size_t>(N) + 1, 0);
      for (int64_t i = 0; i < N; ++i) L.row_ptr[i + 1] = L.row_ptr[i] + L.ucount[i];
      // segment schedule: longest first so that long rows start early
      std::vector<int32_t> users;
      for (int64_t i = 0; i < N; ++i) {
        if (L.ucount[i] > 0) users.push_back(static_cast<int32_t>(i));
        else L.untouched.push_back(static_cast<int32_t>(i));
      }
      std::stable_sort(users.begin(), users.end(),
                       [&](int32_t x, int32_t y) { return L.ucount[x] > L.ucount[y]; });
      L.seg_user = users;
      L.seg_beg.resize(users.size());
      L.seg_len.resize(users.size());
      L.seg_cls.resize(users.size());
      L.nheavy = 0;
      for (size_t s = 0; s < users.size(); ++s) {
        const int32_t u = users[s];
        L.seg_beg[s] = L.row_ptr[u];
        L.seg_len[s] = L.ucount[u];
        L.seg_cls[s] = p.cls_of_worker[p.owner[u]];
        if (L.ucount[u] >= p.heavy_min) L.nheavy = static_cast<int32_t>(s + 1);
      }
    }
    return 0;
  } catch (const std::bad_alloc &) {
    err = "host allocation failed while building the layout";
    return -2;
  }
}

}  // namespace psmf
