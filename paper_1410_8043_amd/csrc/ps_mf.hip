// ps_mf: clocked SSP / ESSP matrix-factorization SGD, P logical workers on one MI355X.
// C-ABI entry points are declared in include/ps_mf.h; this file holds the gfx950 kernels
// and the host orchestration around them.
//
// Device state (HBM):
//   ring    : (s+1) slots, each [L: users x Kp | R: items x Kp] fp32 row-major; version v
//             lives in slot v mod (s+1); Kp = K rounded up to the kernels' row width,
//             padding columns are kept at zero in every slot.
//   dR      : items x Kp fp32 accumulator of the clock's item updates (zero between clocks).
//   per block: col/val in canonical (user, item, load index) order, the segment schedule
//             (user, first entry, length, worker class), item counts (total and per worker
//             class), the list of users without a rating in the block.
//   slot table: for clock c, the ring slot each worker class reads (Section 3.2 view).
//
// One clock c (Section 3.1 update, Section 3.2 SSP view, Section 4 coalesced commit):
//   sweep  : for every user segment of block c mod B: e = D_ij - L^v_i . R^v_j for each
//            rating, dL_i summed in registers, L^{c+1}_i written once (one writer per
//            user), e * L^v_i added into dR_j with hardware fp32 atomics;
//   commit : R^{c+1}_j = R^c_j + scale_j (dR_j - lambda sum_v n_j^(v) R^v_j); dR_j = 0;
//            users without a rating in the block copy L^c_i into the new slot (s > 0).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <thread>
#include <vector>

#include "../../include/ps_mf.h"
#include "layout.h"

namespace {

constexpr int kBlock = 256;   // threads per workgroup (4 wavefronts of 64)
constexpr int kMaxKp = 512;
constexpr int kHeavyMin = 4096;  // ratings per user from which a whole workgroup takes the row

// ------------------------------------------------------------------ device helpers
template <int E>
__device__ __forceinline__ void load_row(float (&d)[E], const float *__restrict__ p) {
  if constexpr (E == 1) {
    d[0] = p[0];
  } else if constexpr (E == 2) {
    const float2 t = *reinterpret_cast<const float2 *>(p);
    d[0] = t.x; d[1] = t.y;
  } else {
#pragma unroll
    for (int q = 0; q < E / 4; ++q) {
      const float4 t = *reinterpret_cast<const float4 *>(p + 4 * q);
      d[4 * q] = t.x; d[4 * q + 1] = t.y; d[4 * q + 2] = t.z; d[4 * q + 3] = t.w;
    }
  }
}

template <int E>
__device__ __forceinline__ void store_row(float *__restrict__ p, const float (&d)[E]) {
  if constexpr (E == 1) {
    p[0] = d[0];
  } else if constexpr (E == 2) {
    *reinterpret_cast<float2 *>(p) = make_float2(d[0], d[1]);
  } else {
#pragma unroll
    for (int q = 0; q < E / 4; ++q)
      *reinterpret_cast<float4 *>(p + 4 * q) = make_float4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
  }
}

// sum over the G lanes of a lane group (G a power of two dividing 64)
template <int G>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
  for (int m = G / 2; m > 0; m >>= 1) v += __shfl_xor(v, m, G);
  return v;
}

struct SweepArgs {
  const int32_t *seg_user;
  const int64_t *seg_beg;
  const int32_t *seg_len;
  const int32_t *seg_cls;
  int32_t seg_first, nseg;
  const int32_t *col;
  const float *val;
  const int32_t *cls_slot;  // ring slot read by each worker class at this clock
  float *ring;
  int64_t slot_stride;      // floats per slot
  int64_t r_off;            // offset of R inside a slot
  int32_t slot_c, slot_n;   // slots of versions c and c+1
  float *dR;
  float eta, lambda;
  int32_t rowmean;
};

// L^{c+1}_i = L^c_i + scale (dL_i - n lambda L^v_i): the lambda term of each of the n
// ratings is hoisted, scale = eta (SUM) or eta / n (ROWMEAN).
template <int E>
__device__ __forceinline__ void finish_user(const SweepArgs &a, int64_t rowoff, int sv, int n, const float (&lv)[E],
                                            const float (&dl)[E]) {
  float lc[E];
  if (a.slot_c == sv) {
#pragma unroll
    for (int e = 0; e < E; ++e) lc[e] = lv[e];
  } else {
    load_row<E>(lc, a.ring + a.slot_c * a.slot_stride + rowoff);
  }
  const float sc = a.rowmean ? a.eta / static_cast<float>(n) : a.eta;
  const float nl = static_cast<float>(n) * a.lambda;
  float o[E];
#pragma unroll
  for (int e = 0; e < E; ++e) o[e] = lc[e] + sc * (dl[e] - nl * lv[e]);
  store_row<E>(a.ring + a.slot_n * a.slot_stride + rowoff, o);
}

// one lane group of G lanes per user segment; lane g owns columns [g*E, g*E+E)
template <int G, int E>
__global__ __launch_bounds__(kBlock) void k_sweep_light(SweepArgs a) {
  constexpr int Kp = G * E;
  const int lane = threadIdx.x & (G - 1);
  const int64_t gid = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) / G;
  if (gid >= a.nseg) return;  // whole groups leave together
  const int64_t seg = a.seg_first + gid;
  const int64_t u = a.seg_user[seg];
  const int64_t beg = a.seg_beg[seg];
  const int n = a.seg_len[seg];
  const int sv = a.cls_slot[a.seg_cls[seg]];
  const float *__restrict__ Rv = a.ring + sv * a.slot_stride + a.r_off + lane * E;
  const int64_t rowoff = u * Kp + lane * E;
  float lv[E], dl[E];
  load_row<E>(lv, a.ring + sv * a.slot_stride + rowoff);
#pragma unroll
  for (int e = 0; e < E; ++e) dl[e] = 0.f;
  for (int t = 0; t < n; ++t) {
    const int64_t j = a.col[beg + t];
    const float r = a.val[beg + t];
    float rj[E];
    load_row<E>(rj, Rv + j * Kp);
    float p = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) p = fmaf(lv[e], rj[e], p);
    const float err = r - group_sum<G>(p);
    float *dst = a.dR + j * Kp + lane * E;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      dl[e] = fmaf(err, rj[e], dl[e]);
      atomicAdd(dst + e, err * lv[e]);
    }
  }
  finish_user<E>(a, rowoff, sv, n, lv, dl);
}

// one workgroup per long user segment: its kBlock/G lane groups split the ratings and
// combine their partial dL in LDS before the single write of L^{c+1}_i
template <int G, int E>
__global__ __launch_bounds__(kBlock) void k_sweep_heavy(SweepArgs a) {
  constexpr int Kp = G * E;
  constexpr int NG = kBlock / G;
  __shared__ float part[NG * Kp];
  const int lane = threadIdx.x & (G - 1);
  const int grp = threadIdx.x / G;
  const int64_t seg = a.seg_first + blockIdx.x;
  const int64_t u = a.seg_user[seg];
  const int64_t beg = a.seg_beg[seg];
  const int n = a.seg_len[seg];
  const int sv = a.cls_slot[a.seg_cls[seg]];
  const float *__restrict__ Rv = a.ring + sv * a.slot_stride + a.r_off + lane * E;
  const int64_t rowoff = u * Kp + lane * E;
  float lv[E], dl[E];
  load_row<E>(lv, a.ring + sv * a.slot_stride + rowoff);
#pragma unroll
  for (int e = 0; e < E; ++e) dl[e] = 0.f;
  for (int t = grp; t < n; t += NG) {
    const int64_t j = a.col[beg + t];
    const float r = a.val[beg + t];
    float rj[E];
    load_row<E>(rj, Rv + j * Kp);
    float p = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) p = fmaf(lv[e], rj[e], p);
    const float err = r - group_sum<G>(p);
    float *dst = a.dR + j * Kp + lane * E;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      dl[e] = fmaf(err, rj[e], dl[e]);
      atomicAdd(dst + e, err * lv[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) part[grp * Kp + lane * E + e] = dl[e];
  __syncthreads();
  if (grp == 0) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      float s = 0.f;
      for (int g = 0; g < NG; ++g) s += part[g * Kp + lane * E + e];
      dl[e] = s;
    }
    finish_user<E>(a, rowoff, sv, n, lv, dl);
  }
}

struct CommitArgs {
  float *ring;
  int64_t slot_stride, r_off;
  int64_t items;
  int32_t Kp;
  int32_t slot_c, slot_n;
  const int32_t *icount;      // [items]
  const int32_t *icount_cls;  // [items * nclass]
  int32_t nclass;
  const int32_t *cls_slot;    // [nclass]
  float *dR;
  float eta, lambda;
  int32_t rowmean;
};

// R^{c+1}_j = R^c_j + scale_j (dR_j - lambda sum_classes n_j^(class) R^{v(class)}_j), dR_j = 0
__global__ __launch_bounds__(kBlock) void k_commit(CommitArgs a) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= a.items * a.Kp) return;
  const int64_t j = idx / a.Kp;
  const int n = a.icount[j];
  float *R = a.ring + a.r_off;
  const float rc = R[a.slot_c * a.slot_stride + idx];
  float out = rc;
  if (n > 0) {
    float lam = 0.f;
    for (int q = 0; q < a.nclass; ++q) {
      const int cnt = a.icount_cls[j * a.nclass + q];
      if (cnt) lam = fmaf(static_cast<float>(cnt), R[a.cls_slot[q] * a.slot_stride + idx], lam);
    }
    const float sc = a.rowmean ? a.eta / static_cast<float>(n) : a.eta;
    out = rc + sc * (a.dR[idx] - a.lambda * lam);
    a.dR[idx] = 0.f;
  }
  R[a.slot_n * a.slot_stride + idx] = out;
}

// users without a rating in the block: L^{c+1}_i = L^c_i
__global__ __launch_bounds__(kBlock) void k_copy_rows(const int32_t *__restrict__ users, int64_t n, int32_t Kp,
                                                      float *ring, int64_t slot_stride, int32_t slot_c,
                                                      int32_t slot_n) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= n * Kp) return;
  const int64_t off = static_cast<int64_t>(users[idx / Kp]) * Kp + idx % Kp;
  ring[slot_n * slot_stride + off] = ring[slot_c * slot_stride + off];
}

// squared loss partial sums: each lane group takes one segment, e computed in fp32,
// e^2 accumulated in fp64; one partial per workgroup
template <int G, int E>
__global__ __launch_bounds__(kBlock) void k_loss(const int32_t *__restrict__ seg_user,
                                                 const int64_t *__restrict__ seg_beg,
                                                 const int32_t *__restrict__ seg_len, int64_t nseg,
                                                 const int32_t *__restrict__ col, const float *__restrict__ val,
                                                 const float *__restrict__ L, const float *__restrict__ R,
                                                 double *__restrict__ partial) {
  constexpr int Kp = G * E;
  constexpr int NG = kBlock / G;
  __shared__ double acc_sh[NG];
  const int lane = threadIdx.x & (G - 1);
  const int grp = threadIdx.x / G;
  const int64_t gid = static_cast<int64_t>(blockIdx.x) * NG + grp;
  double acc = 0.0;
  if (gid < nseg) {
    const int64_t u = seg_user[gid];
    const int64_t beg = seg_beg[gid];
    const int n = seg_len[gid];
    float lv[E];
    load_row<E>(lv, L + u * Kp + lane * E);
    for (int t = 0; t < n; ++t) {
      float rj[E];
      load_row<E>(rj, R + static_cast<int64_t>(col[beg + t]) * Kp + lane * E);
      float p = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) p = fmaf(lv[e], rj[e], p);
      const float err = val[beg + t] - group_sum<G>(p);
      acc += static_cast<double>(err) * static_cast<double>(err);
    }
  }
  if (lane == 0) acc_sh[grp] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int g = 0; g < NG; ++g) s += acc_sh[g];
    partial[blockIdx.x] = s;
  }
}

// fixed-order final sum of the partials (deterministic for a given layout)
__global__ __launch_bounds__(kBlock) void k_sum_partials(const double *__restrict__ partial, int64_t n,
                                                          double *__restrict__ out) {
  __shared__ double sh[kBlock];
  double s = 0.0;
  for (int64_t x = threadIdx.x; x < n; x += kBlock) s += partial[x];
  sh[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
    for (int x = 0; x < kBlock; ++x) t += sh[x];
    *out = t;
  }
}

// ------------------------------------------------------------------ kernel dispatch on Kp
struct Shape {
  int G, E;
};
Shape shape_for(int Kp) {
  switch (Kp) {
    case 8: return {8, 1};
    case 16: return {8, 2};
    case 32: return {8, 4};
    case 64: return {16, 4};
    case 128: return {32, 4};
    case 256: return {64, 4};
    default: return {64, 8};  // 512
  }
}
int padded_k(int K) {
  int Kp = 8;
  while (Kp < K) Kp *= 2;
  return Kp;
}

template <template <int, int> class F, class... Args>
hipError_t dispatch(int Kp, Args &&...args) {
  switch (Kp) {
    case 8: return F<8, 1>::run(args...);
    case 16: return F<8, 2>::run(args...);
    case 32: return F<8, 4>::run(args...);
    case 64: return F<16, 4>::run(args...);
    case 128: return F<32, 4>::run(args...);
    case 256: return F<64, 4>::run(args...);
    default: return F<64, 8>::run(args...);
  }
}

template <int G, int E>
struct LaunchLight {
  static hipError_t run(const SweepArgs &a, hipStream_t st) {
    const int64_t threads = static_cast<int64_t>(a.nseg) * G;
    const unsigned grid = static_cast<unsigned>((threads + kBlock - 1) / kBlock);
    hipLaunchKernelGGL((k_sweep_light<G, E>), dim3(grid), dim3(kBlock), 0, st, a);
    return hipGetLastError();
  }
};
template <int G, int E>
struct LaunchHeavy {
  static hipError_t run(const SweepArgs &a, hipStream_t st) {
    hipLaunchKernelGGL((k_sweep_heavy<G, E>), dim3(static_cast<unsigned>(a.nseg)), dim3(kBlock), 0, st, a);
    return hipGetLastError();
  }
};
template <int G, int E>
struct LaunchLoss {
  static hipError_t run(const int32_t *su, const int64_t *sb, const int32_t *sl, int64_t nseg, const int32_t *col,
                        const float *val, const float *L, const float *R, double *partial, hipStream_t st) {
    constexpr int NG = kBlock / G;
    const unsigned grid = static_cast<unsigned>((nseg + NG - 1) / NG);
    hipLaunchKernelGGL((k_loss<G, E>), dim3(grid), dim3(kBlock), 0, st, su, sb, sl, nseg, col, val, L, R, partial);
    return hipGetLastError();
  }
};

}  // namespace

// ------------------------------------------------------------------ handle
struct DeviceBlock {
  int64_t nnz = 0, nseg = 0, nheavy = 0, nuntouched = 0;
  int32_t *col = nullptr;
  float *val = nullptr;
  int32_t *seg_user = nullptr, *seg_len = nullptr, *seg_cls = nullptr;
  int64_t *seg_beg = nullptr;
  int32_t *icount = nullptr, *icount_cls = nullptr;
  int32_t *untouched = nullptr;
};

struct ps_mf {
  // problem
  int64_t N = 0, M = 0;
  int32_t K = 0, Kp = 0, P = 0, s = 0;
  float eta = 0, lambda = 0;
  // options
  int32_t policy = PS_MF_SSP_LAZY, step = PS_MF_STEP_ROWMEAN, B = 1;
  uint64_t seed = 0;
  bool host_only = false, timing = false;
  std::vector<int32_t> owner;
  // host state
  bool loaded = false, has_factors = false;
  int64_t clock = 0;
  std::vector<int64_t> vlog;
  std::vector<psmf::BlockLayout> layout;
  int32_t nclass = 1;
  std::vector<int32_t> cls_of_worker;
  std::string err;
  // device state
  int device = -1;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  hipStream_t user_stream = nullptr;
  float *ring = nullptr;
  float *dR = nullptr;
  int32_t *slot_table = nullptr;  // [(2s+1) * nclass]
  double *loss_partial = nullptr;
  int64_t loss_partial_len = 0;
  double *loss_out = nullptr;
  std::vector<DeviceBlock> dblocks;
  std::vector<void *> allocations;
  // timing
  struct Ev {
    int kernel;
    hipEvent_t a, b;
  };
  std::vector<Ev> events;
  double kernel_ms[2] = {0, 0};
  int64_t kernel_count[2] = {0, 0};
};

namespace {

int fail(ps_mf_t *h, int code, const char *fmt, ...) {
  if (h) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    h->err = buf;
  }
  return code;
}

#define HIP_TRY(h, expr)                                                                          \
  do {                                                                                           \
    hipError_t e_ = (expr);                                                                      \
    if (e_ != hipSuccess) {                                                                      \
      if (e_ == hipErrorOutOfMemory) return fail(h, PS_MF_ENOMEM, "%s: %s", #expr, hipGetErrorString(e_)); \
      return fail(h, PS_MF_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_));                     \
    }                                                                                            \
  } while (0)

int dev_alloc(ps_mf_t *h, void **p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    if (e == hipErrorOutOfMemory) return fail(h, PS_MF_ENOMEM, "hipMalloc(%zu bytes) failed: out of memory", bytes);
    return fail(h, PS_MF_EDEVICE, "hipMalloc(%zu bytes) failed: %s", bytes, hipGetErrorString(e));
  }
  h->allocations.push_back(*p);
  return PS_MF_OK;
}

template <class T>
int upload(ps_mf_t *h, T **dst, const std::vector<T> &src) {
  int rc = dev_alloc(h, reinterpret_cast<void **>(dst), src.size() * sizeof(T));
  if (rc) return rc;
  if (!src.empty()) HIP_TRY(h, hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice));
  return PS_MF_OK;
}

int64_t delay_of(const ps_mf_t *h, int64_t p, int64_t c) {
  const int64_t s = h->s;
  switch (h->policy) {
    case PS_MF_SSP_LAZY: return (c + p % (s + 1)) % (s + 1);
    case PS_MF_SSP_WORST: return s;
    default: return s < 1 ? s : 1;
  }
}
int64_t view_version(const ps_mf_t *h, int64_t p, int64_t c) {
  const int64_t v = c - delay_of(h, p, c);
  return v < 0 ? 0 : v;
}
// row of the slot table used at clock c: clocks below s are listed one by one, from s on
// the slot pattern repeats with period s+1
int64_t table_row(const ps_mf_t *h, int64_t c) { return c < h->s ? c : h->s + (c - h->s) % (h->s + 1); }

int ensure_device(ps_mf_t *h) {
  if (h->device < 0) {
    int dev = 0;
    HIP_TRY(h, hipGetDevice(&dev));
    h->device = dev;
  }
  HIP_TRY(h, hipSetDevice(h->device));
  if (!h->stream) {
    if (h->user_stream) {
      h->stream = h->user_stream;
    } else {
      HIP_TRY(h, hipStreamCreateWithFlags(&h->stream, hipStreamNonBlocking));
      h->own_stream = true;
    }
  }
  return PS_MF_OK;
}

int host_threads() {
  unsigned n = std::thread::hardware_concurrency();
  if (n == 0) n = 1;
  return static_cast<int>(std::min(16u, n));
}

int record(ps_mf_t *h, int kernel, hipEvent_t *a) {
  if (!h->timing) return PS_MF_OK;
  HIP_TRY(h, hipEventCreate(a));
  HIP_TRY(h, hipEventRecord(*a, h->stream));
  (void)kernel;
  return PS_MF_OK;
}
int record_end(ps_mf_t *h, int kernel, hipEvent_t a) {
  if (!h->timing) return PS_MF_OK;
  hipEvent_t b;
  HIP_TRY(h, hipEventCreate(&b));
  HIP_TRY(h, hipEventRecord(b, h->stream));
  h->events.push_back({kernel, a, b});
  return PS_MF_OK;
}

int one_clock(ps_mf_t *h) {
  const int64_t c = h->clock;
  const int b = static_cast<int>(c % h->B);
  const int32_t S1 = h->s + 1;
  const int32_t slot_c = static_cast<int32_t>(c % S1), slot_n = static_cast<int32_t>((c + 1) % S1);
  const DeviceBlock &db = h->dblocks[b];
  const int32_t *cls_slot = h->slot_table + table_row(h, c) * h->nclass;
  const int64_t slot_stride = (h->N + h->M) * h->Kp;

  SweepArgs a{};
  a.seg_user = db.seg_user;
  a.seg_beg = db.seg_beg;
  a.seg_len = db.seg_len;
  a.seg_cls = db.seg_cls;
  a.col = db.col;
  a.val = db.val;
  a.cls_slot = cls_slot;
  a.ring = h->ring;
  a.slot_stride = slot_stride;
  a.r_off = h->N * h->Kp;
  a.slot_c = slot_c;
  a.slot_n = slot_n;
  a.dR = h->dR;
  a.eta = h->eta;
  a.lambda = h->lambda;
  a.rowmean = h->step == PS_MF_STEP_ROWMEAN;

  hipEvent_t ev = nullptr;
  int rc = record(h, PS_MF_KERNEL_SWEEP, &ev);
  if (rc) return rc;
  if (db.nheavy > 0) {
    a.seg_first = 0;
    a.nseg = static_cast<int32_t>(db.nheavy);
    HIP_TRY(h, dispatch<LaunchHeavy>(h->Kp, a, h->stream));
  }
  if (db.nseg > db.nheavy) {
    a.seg_first = static_cast<int32_t>(db.nheavy);
    a.nseg = static_cast<int32_t>(db.nseg - db.nheavy);
    HIP_TRY(h, dispatch<LaunchLight>(h->Kp, a, h->stream));
  }
  if ((rc = record_end(h, PS_MF_KERNEL_SWEEP, ev))) return rc;

  if ((rc = record(h, PS_MF_KERNEL_COMMIT, &ev))) return rc;
  if (slot_n != slot_c && db.nuntouched > 0) {
    const int64_t n = db.nuntouched * h->Kp;
    hipLaunchKernelGGL(k_copy_rows, dim3(static_cast<unsigned>((n + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                       h->stream, db.untouched, db.nuntouched, h->Kp, h->ring, slot_stride, slot_c, slot_n);
    HIP_TRY(h, hipGetLastError());
  }
  CommitArgs ca{};
  ca.ring = h->ring;
  ca.slot_stride = slot_stride;
  ca.r_off = h->N * h->Kp;
  ca.items = h->M;
  ca.Kp = h->Kp;
  ca.slot_c = slot_c;
  ca.slot_n = slot_n;
  ca.icount = db.icount;
  ca.icount_cls = db.icount_cls;
  ca.nclass = h->nclass;
  ca.cls_slot = cls_slot;
  ca.dR = h->dR;
  ca.eta = h->eta;
  ca.lambda = h->lambda;
  ca.rowmean = a.rowmean;
  const int64_t ncommit = h->M * h->Kp;
  hipLaunchKernelGGL(k_commit, dim3(static_cast<unsigned>((ncommit + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                     h->stream, ca);
  HIP_TRY(h, hipGetLastError());
  if ((rc = record_end(h, PS_MF_KERNEL_COMMIT, ev))) return rc;

  for (int64_t p = 0; p < h->P; ++p) h->vlog.push_back(view_version(h, p, c));
  h->clock = c + 1;
  return PS_MF_OK;
}

}  // namespace

// ------------------------------------------------------------------ C ABI
extern "C" {

int ps_mf_create(int64_t users, int64_t items, int32_t K, int32_t P, int32_t s, float eta, float lambda,
                 ps_mf_t **out) {
  if (!out) return PS_MF_EINVAL;
  *out = nullptr;
  if (users < 1 || items < 1 || users > 0x7fffffff || items > 0x7fffffff) return PS_MF_EINVAL;
  if (K < 1 || K > kMaxKp || P < 1 || P > 65536 || s < 0 || s > 1024) return PS_MF_EINVAL;
  if (!std::isfinite(eta) || !std::isfinite(lambda)) return PS_MF_EINVAL;
  ps_mf_t *h = new (std::nothrow) ps_mf_t();
  if (!h) return PS_MF_ENOMEM;
  h->N = users;
  h->M = items;
  h->K = K;
  h->Kp = padded_k(K);
  h->P = P;
  h->s = s;
  h->eta = eta;
  h->lambda = lambda;
  *out = h;
  return PS_MF_OK;
}

int ps_mf_set_option(ps_mf_t *h, int32_t key, int64_t value) {
  if (!h) return PS_MF_EINVAL;
  if (h->loaded) return fail(h, PS_MF_ESTATE, "options must be set before ps_mf_load_ratings");
  switch (key) {
    case PS_MF_OPT_POLICY:
      if (value < PS_MF_SSP_LAZY || value > PS_MF_ESSP) return fail(h, PS_MF_EINVAL, "unknown policy %lld", (long long)value);
      h->policy = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_STEP:
      if (value != PS_MF_STEP_ROWMEAN && value != PS_MF_STEP_SUM) return fail(h, PS_MF_EINVAL, "unknown step %lld", (long long)value);
      h->step = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_MB_BLOCKS:
      if (value < 1 || value > 65536) return fail(h, PS_MF_EINVAL, "minibatch blocks must be in [1, 65536]");
      h->B = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_MB_SEED:
      h->seed = static_cast<uint64_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_HOST_ONLY:
      h->host_only = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_TIMING:
      h->timing = value != 0;
      return PS_MF_OK;
    default:
      return fail(h, PS_MF_EINVAL, "unknown option key %d", key);
  }
}

int ps_mf_set_owner_map(ps_mf_t *h, const int32_t *owner) {
  if (!h || !owner) return PS_MF_EINVAL;
  if (h->loaded) return fail(h, PS_MF_ESTATE, "the owner map must be set before ps_mf_load_ratings");
  for (int64_t i = 0; i < h->N; ++i)
    if (owner[i] < 0 || owner[i] >= h->P) return fail(h, PS_MF_EINVAL, "owner[%lld] = %d is not in [0, P)", (long long)i, owner[i]);
  h->owner.assign(owner, owner + h->N);
  return PS_MF_OK;
}

int ps_mf_set_stream(ps_mf_t *h, void *hip_stream) {
  if (!h) return PS_MF_EINVAL;
  if (h->stream && h->own_stream) {
    (void)hipStreamSynchronize(h->stream);
    (void)hipStreamDestroy(h->stream);
    h->own_stream = false;
  } else if (h->stream) {
    (void)hipStreamSynchronize(h->stream);
  }
  h->stream = nullptr;
  h->user_stream = static_cast<hipStream_t>(hip_stream);
  if (h->loaded && !h->host_only) return ensure_device(h);
  return PS_MF_OK;
}

int ps_mf_load_ratings(ps_mf_t *h, const int32_t *user, const int32_t *item, const float *value, int64_t n) {
  if (!h) return PS_MF_EINVAL;
  if (h->loaded) return fail(h, PS_MF_ESTATE, "ratings are already loaded");
  if (n < 0 || (n > 0 && (!user || !item || !value))) return fail(h, PS_MF_EINVAL, "bad rating arrays");
  if (n > 0x7fffffffLL) return fail(h, PS_MF_EINVAL, "at most 2^31-1 ratings");
  if (h->owner.empty()) {
    h->owner.resize(static_cast<size_t>(h->N));
    for (int64_t i = 0; i < h->N; ++i) h->owner[i] = static_cast<int32_t>(i % h->P);
  }
  // worker classes: workers that read the same version at every clock
  h->nclass = (h->policy == PS_MF_SSP_LAZY) ? std::min<int32_t>(h->s + 1, h->P) : 1;
  h->cls_of_worker.resize(static_cast<size_t>(h->P));
  for (int32_t p = 0; p < h->P; ++p) h->cls_of_worker[p] = (h->policy == PS_MF_SSP_LAZY) ? p % (h->s + 1) : 0;

  psmf::LayoutParams lp;
  lp.users = h->N;
  lp.items = h->M;
  lp.B = h->B;
  lp.seed = h->seed;
  lp.nclass = h->nclass;
  lp.owner = h->owner.data();
  lp.cls_of_worker = h->cls_of_worker.data();
  lp.heavy_min = kHeavyMin;
  lp.threads = host_threads();
  std::string err;
  const int rc = psmf::build_layout(lp, user, item, value, n, h->layout, err);
  if (rc == -1) return fail(h, PS_MF_EINVAL, "%s", err.c_str());
  if (rc) return fail(h, PS_MF_ENOMEM, "%s", err.c_str());
  h->loaded = true;
  if (h->host_only) return PS_MF_OK;

  int r = ensure_device(h);
  if (r) { h->loaded = false; return r; }
  const size_t slot = static_cast<size_t>((h->N + h->M) * h->Kp);
  auto undo = [h](int code) { h->loaded = false; return code; };
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->ring), slot * (h->s + 1) * sizeof(float)))) return undo(r);
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->dR), static_cast<size_t>(h->M * h->Kp) * sizeof(float)))) return undo(r);
  hipError_t e = hipMemset(h->dR, 0, static_cast<size_t>(h->M * h->Kp) * sizeof(float));
  if (e != hipSuccess) return undo(fail(h, PS_MF_EDEVICE, "hipMemset: %s", hipGetErrorString(e)));
  h->dblocks.assign(static_cast<size_t>(h->B), DeviceBlock());
  int64_t max_groups = 1;
  for (int b = 0; b < h->B; ++b) {
    const psmf::BlockLayout &L = h->layout[b];
    DeviceBlock &d = h->dblocks[b];
    d.nnz = L.nnz;
    d.nseg = static_cast<int64_t>(L.seg_user.size());
    d.nheavy = L.nheavy;
    d.nuntouched = static_cast<int64_t>(L.untouched.size());
    if ((r = upload(h, &d.col, L.col)) || (r = upload(h, &d.val, L.val)) || (r = upload(h, &d.seg_user, L.seg_user)) ||
        (r = upload(h, &d.seg_beg, L.seg_beg)) || (r = upload(h, &d.seg_len, L.seg_len)) ||
        (r = upload(h, &d.seg_cls, L.seg_cls)) || (r = upload(h, &d.icount, L.icount)) ||
        (r = upload(h, &d.icount_cls, L.icount_cls)) || (r = upload(h, &d.untouched, L.untouched)))
      return undo(r);
    const int G = shape_for(h->Kp).G;
    max_groups = std::max<int64_t>(max_groups, (d.nseg + kBlock / G - 1) / (kBlock / G));
  }
  // loss partials: one per workgroup of each block, laid end to end
  h->loss_partial_len = max_groups * h->B;
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->loss_partial), static_cast<size_t>(h->loss_partial_len) * sizeof(double))))
    return undo(r);
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->loss_out), sizeof(double)))) return undo(r);
  // slot table: row c (c < s) and rows s .. 2s (periodic part), one entry per worker class
  std::vector<int32_t> table(static_cast<size_t>((2 * h->s + 1) * h->nclass));
  std::vector<int32_t> rep(static_cast<size_t>(h->nclass), -1);  // a worker of each class
  for (int32_t p = 0; p < h->P; ++p)
    if (rep[h->cls_of_worker[p]] < 0) rep[h->cls_of_worker[p]] = p;
  for (int64_t row = 0; row < 2 * h->s + 1; ++row) {
    const int64_t c = row;  // rows 0..2s hold clocks 0..2s, which cover the periodic part
    for (int q = 0; q < h->nclass; ++q)
      table[row * h->nclass + q] = static_cast<int32_t>(view_version(h, rep[q] < 0 ? 0 : rep[q], c) % (h->s + 1));
  }
  if ((r = upload(h, &h->slot_table, table))) return undo(r);
  return PS_MF_OK;
}

int ps_mf_set_factors(ps_mf_t *h, const float *L, const float *R) {
  if (!h || !L || !R) return PS_MF_EINVAL;
  if (!h->loaded) return fail(h, PS_MF_ESTATE, "load ratings before setting factors");
  if (h->host_only) return fail(h, PS_MF_ESTATE, "host-only handle has no device state");
  const int64_t nl = h->N * h->K, nr = h->M * h->K;
  for (int64_t x = 0; x < nl; ++x)
    if (!std::isfinite(L[x])) return fail(h, PS_MF_EINVAL, "L[%lld] is not finite", (long long)x);
  for (int64_t x = 0; x < nr; ++x)
    if (!std::isfinite(R[x])) return fail(h, PS_MF_EINVAL, "R[%lld] is not finite", (long long)x);
  int r = ensure_device(h);
  if (r) return r;
  const size_t slot = static_cast<size_t>((h->N + h->M) * h->Kp);
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  HIP_TRY(h, hipMemset(h->ring, 0, slot * (h->s + 1) * sizeof(float)));
  HIP_TRY(h, hipMemset(h->dR, 0, static_cast<size_t>(h->M * h->Kp) * sizeof(float)));
  HIP_TRY(h, hipMemcpy2D(h->ring, h->Kp * sizeof(float), L, h->K * sizeof(float), h->K * sizeof(float),
                         static_cast<size_t>(h->N), hipMemcpyHostToDevice));
  HIP_TRY(h, hipMemcpy2D(h->ring + h->N * h->Kp, h->Kp * sizeof(float), R, h->K * sizeof(float),
                         h->K * sizeof(float), static_cast<size_t>(h->M), hipMemcpyHostToDevice));
  HIP_TRY(h, hipDeviceSynchronize());
  h->clock = 0;
  h->vlog.clear();
  h->has_factors = true;
  return PS_MF_OK;
}

int ps_mf_clock(ps_mf_t *h, int32_t n) {
  if (!h || n < 0) return PS_MF_EINVAL;
  if (!h->loaded || !h->has_factors) return fail(h, PS_MF_ESTATE, "load ratings and set factors before clocking");
  int r = ensure_device(h);
  if (r) return r;
  for (int32_t q = 0; q < n; ++q)
    if ((r = one_clock(h))) return r;
  return PS_MF_OK;
}

int ps_mf_loss(ps_mf_t *h, double *out) {
  if (!h || !out) return PS_MF_EINVAL;
  if (!h->loaded || !h->has_factors) return fail(h, PS_MF_ESTATE, "load ratings and set factors before the loss");
  int r = ensure_device(h);
  if (r) return r;
  const int64_t slot_stride = (h->N + h->M) * h->Kp;
  const int32_t sl = static_cast<int32_t>(h->clock % (h->s + 1));
  const float *L = h->ring + sl * slot_stride;
  const float *R = L + h->N * h->Kp;
  const int G = shape_for(h->Kp).G;
  int64_t off = 0;
  for (int b = 0; b < h->B; ++b) {
    const DeviceBlock &d = h->dblocks[b];
    if (d.nseg == 0) continue;
    HIP_TRY(h, dispatch<LaunchLoss>(h->Kp, d.seg_user, d.seg_beg, d.seg_len, d.nseg, d.col, d.val, L, R,
                                     h->loss_partial + off, h->stream));
    off += (d.nseg + kBlock / G - 1) / (kBlock / G);
  }
  if (off == 0) {
    *out = 0.0;
    return PS_MF_OK;
  }
  hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(kBlock), 0, h->stream, h->loss_partial, off, h->loss_out);
  HIP_TRY(h, hipGetLastError());
  double v = 0;
  HIP_TRY(h, hipMemcpyAsync(&v, h->loss_out, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  *out = v;
  return PS_MF_OK;
}

int ps_mf_get_version(ps_mf_t *h, int64_t v, float *L, float *R) {
  if (!h || !L || !R) return PS_MF_EINVAL;
  if (!h->has_factors) return fail(h, PS_MF_ESTATE, "no factors set");
  if (v < 0 || v > h->clock || v < h->clock - h->s)
    return fail(h, PS_MF_EINVAL, "version %lld is not in the ring", (long long)v);
  int r = ensure_device(h);
  if (r) return r;
  const int64_t slot_stride = (h->N + h->M) * h->Kp;
  const float *base = h->ring + (v % (h->s + 1)) * slot_stride;
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  HIP_TRY(h, hipMemcpy2D(L, h->K * sizeof(float), base, h->Kp * sizeof(float), h->K * sizeof(float),
                         static_cast<size_t>(h->N), hipMemcpyDeviceToHost));
  HIP_TRY(h, hipMemcpy2D(R, h->K * sizeof(float), base + h->N * h->Kp, h->Kp * sizeof(float),
                         h->K * sizeof(float), static_cast<size_t>(h->M), hipMemcpyDeviceToHost));
  return PS_MF_OK;
}

int ps_mf_get_factors(ps_mf_t *h, float *L, float *R) {
  if (!h) return PS_MF_EINVAL;
  return ps_mf_get_version(h, h->clock, L, R);
}

int ps_mf_get_clock(ps_mf_t *h, int64_t *clock) {
  if (!h || !clock) return PS_MF_EINVAL;
  *clock = h->clock;
  return PS_MF_OK;
}

int ps_mf_export_index(ps_mf_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len) {
  if (!h || !len) return PS_MF_EINVAL;
  if (kind != PS_MF_IDX_OWNER && kind != PS_MF_IDX_VERSION_LOG) {
    if (!h->loaded) return fail(h, PS_MF_ESTATE, "no ratings loaded");
    if (block < 0 || block >= h->B) return fail(h, PS_MF_EINVAL, "block %d out of range", block);
  }
  if (kind == PS_MF_IDX_OWNER && h->owner.empty()) {
    h->owner.resize(static_cast<size_t>(h->N));
    for (int64_t i = 0; i < h->N; ++i) h->owner[i] = static_cast<int32_t>(i % h->P);
  }
  const void *src = nullptr;
  size_t esz = 0;
  int64_t n = 0;
  switch (kind) {
    case PS_MF_IDX_OWNER: src = h->owner.data(); esz = 4; n = h->N; break;
    case PS_MF_IDX_ROW_PTR: src = h->layout[block].row_ptr.data(); esz = 8; n = h->N + 1; break;
    case PS_MF_IDX_COL: src = h->layout[block].col.data(); esz = 4; n = h->layout[block].nnz; break;
    case PS_MF_IDX_PERM: src = h->layout[block].perm.data(); esz = 8; n = h->layout[block].nnz; break;
    case PS_MF_IDX_USER_COUNT: src = h->layout[block].ucount.data(); esz = 4; n = h->N; break;
    case PS_MF_IDX_ITEM_COUNT: src = h->layout[block].icount.data(); esz = 4; n = h->M; break;
    case PS_MF_IDX_VERSION_LOG: src = h->vlog.data(); esz = 8; n = static_cast<int64_t>(h->vlog.size()); break;
    default: return fail(h, PS_MF_EINVAL, "unknown index kind %d", kind);
  }
  *len = n;
  if (!buf) return PS_MF_OK;
  if (cap < n) return fail(h, PS_MF_EINVAL, "buffer holds %lld elements, %lld needed", (long long)cap, (long long)n);
  if (n > 0) std::memcpy(buf, src, static_cast<size_t>(n) * esz);
  return PS_MF_OK;
}

int ps_mf_kernel_time(ps_mf_t *h, int32_t kernel, double *ms, int64_t *count) {
  if (!h || !ms || !count || kernel < 0 || kernel > 1) return PS_MF_EINVAL;
  if (h->stream) HIP_TRY(h, hipStreamSynchronize(h->stream));
  for (auto &ev : h->events) {
    float t = 0;
    HIP_TRY(h, hipEventElapsedTime(&t, ev.a, ev.b));
    h->kernel_ms[ev.kernel] += t;
    h->kernel_count[ev.kernel] += 1;
    (void)hipEventDestroy(ev.a);
    (void)hipEventDestroy(ev.b);
  }
  h->events.clear();
  *ms = h->kernel_ms[kernel];
  *count = h->kernel_count[kernel];
  return PS_MF_OK;
}

const char *ps_mf_last_error(const ps_mf_t *h) {
  if (!h) return "null handle";
  return h->err.c_str();
}

void ps_mf_destroy(ps_mf_t *h) {
  if (!h) return;
  if (h->stream) (void)hipStreamSynchronize(h->stream);
  for (auto &ev : h->events) {
    (void)hipEventDestroy(ev.a);
    (void)hipEventDestroy(ev.b);
  }
  for (void *p : h->allocations) (void)hipFree(p);
  if (h->own_stream && h->stream) (void)hipStreamDestroy(h->stream);
  delete h;
}

}  // extern "C"
