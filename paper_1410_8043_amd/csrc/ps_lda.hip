// LDA by collapsed Gibbs sampling under clocked SSP / ESSP (arXiv 1410.8043, Section 5's
// topic-modeling workload) on one gfx950 GPU: P logical workers, one wavefront each.
//
// Design:
//   - the shared state is a ring of s+2 committed versions of the (V+1) x K int32 counts
//     (word-topic rows, then the topic totals); after the sampling kernel, a commit kernel
//     writes the version of clock c+1 into its own slot: version c plus every worker's
//     changes of the clock (integer sums: exact and order-free);
//   - one wavefront per worker, lanes over topics (lane l holds ceil(K/64) consecutive
//     topics): the collapsed conditional's K weights are computed in fp64 and quantised to
//     integers on a scale set by the largest of them (its exponent from a DPP wave max),
//     their prefix sums come from per-lane sums and one DPP wave scan, and the drawn topic
//     from one ballot;
//   - a worker reads its view plus its own changes of the clock: these live in a private
//     dense delta table (words x K) whose rows carry the clock that last wrote them, so a row
//     from an older clock reads as zero and nothing is cleared between clocks; the worker's
//     topic-total changes stay in registers and go to its row of a P x K table at its end,
//     which the commit adds with the tagged own-change rows;
//   - the doc-topic row of the current document stays in registers while the worker's tokens
//     of that document run (tokens are in (document, load index) order).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <stdexcept>
#include <string>
#include <type_traits>
#include <utility>
#include <vector>

#include "ps_lda.h"

namespace {

constexpr int kWave = 64;
constexpr int kMaxTopicsPerLane = 8;  // K <= 512
constexpr uint64_t kDrawSalt = 0x5851F42D4C957F2DULL;
constexpr int kLoglikBlocks = 1024;
constexpr int kLoglikThreads = 256;

// one step of SplitMix64 (Steele, Lea and Flood 2014) from state x
__host__ __device__ inline uint64_t splitmix64(uint64_t x) {
  uint64_t z = x + 0x9E3779B97F4A7C15ULL;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

// the staleness of worker p's view at clock c under each policy
__host__ __device__ inline int64_t view_of(int policy, int64_t s, int64_t p, int64_t c) {
  int64_t d;
  if (policy == PS_LDA_SSP_LAZY) d = (c + p % (s + 1)) % (s + 1);
  else if (policy == PS_LDA_SSP_WORST) d = s;
  else d = s < 1 ? s : 1;
  return c - d < 0 ? 0 : c - d;
}

struct SweepArgs {
  const int4 *rec;      // per block position: {word, document, load index, 0}
  int32_t *z;           // per block position: current topic
  int32_t *ndk;         // D x K
  int32_t *ring;        // nslots x (V+1) x K
  int32_t *delta;       // P x V x K, rows valid where tag == tagc
  int32_t *tag;         // P x V
  int32_t *tot;         // P x K: each worker's topic-total changes of the clock
  const int64_t *wbeg;  // P+1 block positions of this clock's block
  int64_t slot_stride;  // (V+1) * K
  int64_t V, D;
  int64_t c;
  double alpha, beta, Vbeta;
  uint64_t seed;
  int32_t K, s, policy, nslots, tagc;
  int32_t shift0;       // 62 - ceil(log2 K): the largest weight lies in [2^shift0, 2^(shift0+1))
};

__device__ __forceinline__ uint64_t readlane_u64(uint64_t x, int lane) {
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x)), lane));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<uint32_t>(x >> 32)), lane));
  return (static_cast<uint64_t>(hi) << 32) | lo;
}

// the high 64 bits of the 128-bit product a * b, on the vector unit: four 32 x 32 + 64
// multiply-adds (the operands are first moved into vector registers, where the scalar
// unit's form of the same product takes about fifteen instructions)
__device__ __forceinline__ uint64_t umulhi64_vec(uint64_t a, uint64_t b) {
  uint32_t a0 = static_cast<uint32_t>(a), a1 = static_cast<uint32_t>(a >> 32);
  asm("" : "+v"(a0), "+v"(a1));
  const uint32_t b0 = static_cast<uint32_t>(b), b1 = static_cast<uint32_t>(b >> 32);
  const uint64_t t = static_cast<uint64_t>(a0) * b0;
  const uint64_t u = static_cast<uint64_t>(a1) * b0 + (t >> 32);
  const uint64_t w = static_cast<uint64_t>(a0) * b1 + static_cast<uint32_t>(u);
  return static_cast<uint64_t>(a1) * b1 + (u >> 32) + (w >> 32);
}

// inclusive prefix sum of a 64-bit value over the wavefront (all 64 lanes active):
// Hillis-Steele inside each row of 16 lanes (DPP row shifts 1, 2, 4, 8; a lane without a
// source adds 0), then row_bcast:15 adds the last lane of rows 0 and 2 into rows 1 and 3,
// and row_bcast:31 the last lane of row 1 (by then the sum of rows 0-1) into rows 2 and 3
// (rows the mask leaves out keep their value); *total gets lane 63's sum.  Each step is one
// add of the low halves with the carry into VCC and one add of the high halves with that
// carry, both reading the shifted operand through DPP.  A DPP read needs two wait states
// after the write of its operand: s_nop 1 before the first step (the input's write), and
// between steps one s_nop 0 plus the other half's add; the s_nop 0 at the end is the wait
// state that a lane read of the result needs after its write.
__device__ __forceinline__ uint64_t wave_scan(uint64_t x, uint64_t *total) {
  uint32_t lo = static_cast<uint32_t>(x), hi = static_cast<uint32_t>(x >> 32);
#define PS_LDA_SCAN_STEP(DPP)                                          \
  "v_add_co_u32_dpp %0, vcc, %0, %0 " DPP "\n\t"                        \
  "v_addc_co_u32_dpp %1, vcc, %1, %1, vcc " DPP "\n\t"
  asm volatile("s_nop 1\n\t"
               PS_LDA_SCAN_STEP("row_shr:1 row_mask:0xf bank_mask:0xf bound_ctrl:1") "s_nop 0\n\t"
               PS_LDA_SCAN_STEP("row_shr:2 row_mask:0xf bank_mask:0xf bound_ctrl:1") "s_nop 0\n\t"
               PS_LDA_SCAN_STEP("row_shr:4 row_mask:0xf bank_mask:0xf bound_ctrl:1") "s_nop 0\n\t"
               PS_LDA_SCAN_STEP("row_shr:8 row_mask:0xf bank_mask:0xf bound_ctrl:1") "s_nop 0\n\t"
               PS_LDA_SCAN_STEP("row_bcast:15 row_mask:0xa bank_mask:0xf") "s_nop 0\n\t"
               PS_LDA_SCAN_STEP("row_bcast:31 row_mask:0xc bank_mask:0xf") "s_nop 0"
               : "+v"(lo), "+v"(hi)
               :
               : "vcc");
#undef PS_LDA_SCAN_STEP
  x = (static_cast<uint64_t>(hi) << 32) | lo;
  *total = readlane_u64(x, 63);
  return x;
}

// One step of a wavefront maximum: x = max(x, x of the lane that CTRL names), by one DPP
// instruction (lanes that the row mask leaves out keep x).  A DPP read needs two wait
// states after the write of its operand: WAIT is the number of instructions the caller
// places between the write and the step (0, 1 or 2 and more), and the step adds s_nop 1,
// s_nop 0 or nothing.  Four steps (quad_perm [1,0,3,2], quad_perm [2,3,0,1], row_half_mirror,
// row_mirror) give each lane its 16-lane row's maximum (every source lane lies inside the
// row), then row_bcast:15 (rows 1 and 3) and row_bcast:31 (rows 2 and 3) carry the rows'
// maxima into row 3, so lane 63 holds the wavefront's.
#define PS_LDA_MAX_STEP(x, WAIT, CTRL)                                                  \
  do {                                                                                  \
    if constexpr ((WAIT) >= 2) asm volatile("v_max_i32_dpp %0, %0, %0 " CTRL : "+v"(x)); \
    else if constexpr ((WAIT) == 1)                                                     \
      asm volatile("s_nop 0\n\tv_max_i32_dpp %0, %0, %0 " CTRL : "+v"(x));              \
    else                                                                                \
      asm volatile("s_nop 1\n\tv_max_i32_dpp %0, %0, %0 " CTRL : "+v"(x));              \
  } while (0)

// what one token reads before it can be sampled: its view row and own-change row of the
// word, the row's clock tag, and its current topic
template <int KPL>
struct TokenRows {
  int nw[KPL], dw[KPL];
  int tag, z;
};

// A table of int32 counts read and written at (row offset + lane offset) bytes.  The buffer
// form (Buf = true) goes through a buffer resource (CDNA word 3 0x00020000: raw, untyped
// dword access): a 32-bit lane offset (the topic) plus a 32-bit uniform offset (the row), so
// that a row's address costs one scalar multiply; the host picks it when every such table
// is under 2^31 bytes.  The flat form takes 64-bit row offsets for larger tables.
template <bool Buf>
struct Table;

template <>
struct Table<true> {
  using Off = uint32_t;
  __amdgpu_buffer_rsrc_t rs;
  __device__ __forceinline__ Table(const int32_t *base, int64_t num_bytes)
      : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t *>(base), static_cast<short>(0),
                                             static_cast<int>(static_cast<uint32_t>(num_bytes)), 0x00020000)) {}
  __device__ __forceinline__ int ld(uint32_t lane_off, Off row_off) const {
    return static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(rs, static_cast<int>(lane_off), static_cast<int>(row_off), 0));
  }
  __device__ __forceinline__ int ld(Off row_off) const {
    return static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(rs, 0, static_cast<int>(row_off), 0));
  }
  __device__ __forceinline__ void st(int v, uint32_t lane_off, Off row_off) const {
    __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(v), rs, static_cast<int>(lane_off), static_cast<int>(row_off), 0);
  }
  __device__ __forceinline__ void st(int v, Off row_off) const {
    __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(v), rs, 0, static_cast<int>(row_off), 0);
  }
  // a store that the hardware drops unless keep, without a branch: the dropped lanes' offset
  // is 2^31 + row_off, past every table of this form (each is under 2^31 bytes, and so is
  // row_off, so the sum does not wrap), and a buffer store outside its resource is discarded
  __device__ __forceinline__ void st_if(bool keep, int v, uint32_t lane_off, Off row_off) const {
    st(v, keep ? lane_off : 0x80000000u, row_off);
  }
};

template <>
struct Table<false> {
  using Off = uint64_t;
  char *base;
  __device__ __forceinline__ Table(const int32_t *b, int64_t) : base(reinterpret_cast<char *>(const_cast<int32_t *>(b))) {}
  __device__ __forceinline__ int ld(uint32_t lane_off, Off row_off) const {
    return *reinterpret_cast<const int32_t *>(base + row_off + lane_off);
  }
  __device__ __forceinline__ int ld(Off row_off) const { return *reinterpret_cast<const int32_t *>(base + row_off); }
  __device__ __forceinline__ void st(int v, uint32_t lane_off, Off row_off) const {
    *reinterpret_cast<int32_t *>(base + row_off + lane_off) = v;
  }
  __device__ __forceinline__ void st(int v, Off row_off) const { *reinterpret_cast<int32_t *>(base + row_off) = v; }
  __device__ __forceinline__ void st_if(bool keep, int v, uint32_t lane_off, Off row_off) const {
    if (keep) st(v, lane_off, row_off);
  }
};

// koff[j]: the byte offset of this lane's topic j in a row (lanes past the last topic
// re-read topic K-1: every load is issued on every path, so the waits before a use count
// exactly; their values are masked); rb: the word's row offset in bytes
template <int KPL, bool Buf>
__device__ __forceinline__ void fetch_rows(const Table<Buf> &view, const Table<Buf> &mydelta, const Table<Buf> &mytag,
                                           const Table<Buf> &z, const uint32_t (&koff)[KPL],
                                           typename Table<Buf>::Off rb, int w, int i, TokenRows<KPL> &o) {
  using Off = typename Table<Buf>::Off;
  o.tag = mytag.ld(Off{4} * static_cast<uint32_t>(w));
  o.z = z.ld(Off{4} * static_cast<uint32_t>(i));
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    o.nw[j] = view.ld(koff[j], rb);
    o.dw[j] = mydelta.ld(koff[j], rb);
  }
}

// step(integral_constant<int, I>, q + I) for I = I0 .. N-1 while q + I < q1
template <int I0, int N, class F>
__device__ __forceinline__ void seq_steps(F &f, int q, int q1, bool &more) {
  if (q + I0 >= q1) {
    more = false;
    return;
  }
  f(std::integral_constant<int, I0>{}, q + I0);
  if constexpr (I0 + 1 < N) seq_steps<I0 + 1, N>(f, q, q1, more);
}

// Lane l holds topics l*KPL .. l*KPL+KPL-1 (consecutive, so one wave scan of the lanes'
// sums orders every topic).  Tokens run in a rotation of kDist+1 steps whose buffer indices
// are fixed at compile time: at the end of step q, after its own stores, the rows of token
// q+kDist are fetched.  The fetch of token t sees every store up to token t-kDist; the
// stores of the kDist-1 tokens after that come later, so the updated own-change rows of
// those tokens stay in registers, and a token whose word matches one of them takes the
// latest such row instead of its fetched one.  Fetches past the last token read the
// last token's word (the record block repeats it) and topic entries past it (the topic
// array has kDist entries of padding) and are never used, which keeps every fetch
// unconditional (so the waits before a use count exactly the newer loads).
//
// The token records come in blocks of 64, one per lane (a vector load), read with lane
// reads: the block at base holds tokens base .. base+63 and serves the tokens base ..
// base+kRecStep-1 and the fetches up to kDist tokens further; the next block is loaded
// when this one starts, kRecStep tokens before its first use.  (Records loaded one at a
// time by scalar loads, a token ahead of their fetch, put the scalar load's latency into
// every token: a wait for a scalar load waits for all of them.)
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kDist = 3;
constexpr int kRecStep = (64 - kDist) / (kDist + 1) * (kDist + 1);  // a multiple of the rotation, at most 64 - kDist

template <int KPL, bool Buf>
__global__ __launch_bounds__(kWave) void k_lda_sweep(SweepArgs a) {
  using Off = typename Table<Buf>::Off;
  constexpr int R = kDist + 1;  // ring entries
  constexpr int F = kDist - 1;  // forwarded rows
  const int lane = threadIdx.x;
  const int64_t p = blockIdx.x;
  const int64_t q0 = a.wbeg[p], q1 = a.wbeg[p + 1];
  const int K = a.K;
  if (q0 >= q1) {  // no tokens this clock: no topic-total changes
    for (int k = lane; k < K; k += kWave) a.tot[p * K + k] = 0;
    return;
  }
  const int64_t V = a.V, c = a.c;
  const int64_t v = view_of(a.policy, a.s, p, c);
  const int32_t *view_p = a.ring + (v % a.nslots) * a.slot_stride;
  const Table<Buf> view(view_p, a.slot_stride * 4);
  const Table<Buf> mydelta(a.delta + p * V * K, V * K * 4);
  const Table<Buf> mytag(a.tag + p * V, V * 4);
  const Table<Buf> ndk(a.ndk, a.D * K * 4);
  // this worker's tokens of the block, indexed from 0 (a worker has fewer than 2^31)
  const i32x4 *rec = reinterpret_cast<const i32x4 *>(a.rec) + q0;
  const int n = static_cast<int>(q1 - q0), last = n - 1;
  const Table<Buf> z(a.z + q0, (static_cast<int64_t>(n) + kDist) * 4);
  const Off rowb = Off{4} * static_cast<uint32_t>(K);  // bytes per row
  const uint64_t rbase = a.seed ^ kDrawSalt ^ (static_cast<uint64_t>(c) << 40);
  uint32_t koff[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j) koff[j] = 4u * static_cast<uint32_t>(min(lane * KPL + j, K - 1));

  // alpha per topic slot, 0 past the last topic: there the document count is 0 as well, so
  // the weight's numerator and the weight are 0 (the denominator is at least V beta)
  double alpha_k[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j) alpha_k[j] = lane * KPL + j < K ? a.alpha : 0.0;
  // topic totals: the view's, and the current ones (the view's plus this worker's changes)
  int vk[KPL], nk[KPL], nd[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int k = lane * KPL + j;
    vk[j] = k < K ? view_p[V * K + k] : 0;
    nk[j] = vk[j];
    nd[j] = 0;
  }
  int cur_doc = -1;
  TokenRows<KPL> rows[R];
  // token records: the current block and the next one; rnd holds the draw's random value of
  // each token of the current block (SplitMix64 of its load index, computed once per block)
  int base = 0;
  i32x4 rv = rec[min(base + lane, last)];
  i32x4 rv_next = rec[min(base + kRecStep + lane, last)];
  uint64_t rnd = splitmix64(rbase ^ static_cast<uint64_t>(static_cast<uint32_t>(rv[2])));
  auto field = [&](int i, int f) { return __builtin_amdgcn_readlane(rv[f], i - base); };
#pragma unroll
  for (int i = 0; i < kDist; ++i) {
    const int wi = field(i, 0);
    fetch_rows<KPL, Buf>(view, mydelta, mytag, z, koff, rowb * static_cast<Off>(wi), wi, i, rows[i]);
    __builtin_amdgcn_sched_barrier(0);
  }
  // the last F tokens' words (-1: none), row validity and updated own-change rows, latest first
  int fw[F > 0 ? F : 1];
  int fvalid[F > 0 ? F : 1];
  int fdw[F > 0 ? F : 1][KPL];
#pragma unroll
  for (int i = 0; i < F; ++i) {
    fw[i] = -1;
    fvalid[i] = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) fdw[i][j] = 0;
  }

  auto step = [&](auto phase, int i) {
    constexpr int C = decltype(phase)::value;
    const int w = field(i, 0), d = field(i, 1);
    // read early (a value from a lane read wants wait states before a load or a vector
    // instruction uses it): the word of the token whose rows this step fetches, and this
    // token's draw value
    const int wf = field(i + kDist, 0);
    const uint64_t ru = readlane_u64(rnd, i - base);
    const int k0 = __builtin_amdgcn_readfirstlane(rows[C].z);
    // 1 when the fetched own-change row is of this clock, formed on the scalar unit (the
    // compiler would turn the compare's flag into an integer on the vector unit)
    int valid;
    asm("s_cmp_eq_u32 %1, %2\n\ts_cselect_b32 %0, 1, 0"
        : "=s"(valid)
        : "s"(__builtin_amdgcn_readfirstlane(rows[C].tag)), "s"(a.tagc)
        : "scc");
    int dw[KPL];
#pragma unroll
    for (int j = 0; j < KPL; ++j) dw[j] = rows[C].dw[j];
    // the latest of the last F tokens with this word, if any, overrides the fetched row (a
    // branch on the rare repeat, so that the common token runs no selects; the product of
    // the differences is 0 on a repeat, and on a wrap to 0 the branch only checks for
    // nothing)
    uint32_t differ = 1;
#pragma unroll
    for (int f = 0; f < F; ++f) differ *= static_cast<uint32_t>(fw[f] ^ w);
    if (__builtin_expect(differ == 0, 0)) {
#pragma unroll
      for (int f = F - 1; f >= 0; --f) {
        if (fw[f] == w) {
          valid = fvalid[f];
#pragma unroll
          for (int j = 0; j < KPL; ++j) dw[j] = fdw[f][j];
        }
      }
    }
    // an own-change row from an older clock reads as zero (an and with a uniform mask keeps
    // the validity an integer rather than a lane mask)
    const int vmask = -valid;
#pragma unroll
    for (int j = 0; j < KPL; ++j) dw[j] &= vmask;
    if (d != cur_doc) {
      if (cur_doc >= 0) {
#pragma unroll
        for (int j = 0; j < KPL; ++j)
          if (lane * KPL + j < K) ndk.st(nd[j], koff[j], rowb * static_cast<Off>(cur_doc));
      }
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        const int x = ndk.ld(koff[j], rowb * static_cast<Off>(d));
        nd[j] = lane * KPL + j < K ? x : 0;
      }
      cur_doc = d;
    }
    // the collapsed conditional's weights p_k = num_k / den_k in fp64 and the exponent of
    // the largest (computed on every lane, without a branch: lanes past the last topic hold
    // topic K-1's rows, a zero document count and alpha = 0, so their weights are 0, and
    // their exponents are masked).
    // * The exponent is found without waiting for the divisions: with frexp exponents (x =
    //   m 2^e, m in [0.5, 1)) num / den lies in [2^(e_num - e_den - 1), 2^(e_num - e_den + 1))
    //   and never rounds up to the upper end, so the largest weight's frexp exponent is the
    //   wavefront maximum E of e_num - e_den + 1 over the topics, or E - 1; it is E exactly
    //   when some weight reaches 2^(E - 1).
    // * The divisions are the hardware reciprocal, two Newton steps, the product and one
    //   correction: the instructions the compiler emits for a correctly rounded fp64
    //   division, without its range scaling (v_div_scale) and special-case fixup
    //   (v_div_fixup). Those leave their operands unchanged when num, den and num / den
    //   are normal with exponents well inside +-768 (no scaling, no overflow, no
    //   denormal), which the load guarantees: every num, den and p lies in
    //   [2^-700, 2^700].  So each p_k is the correctly rounded quotient, as the oracle's.
    // * The maximum's six DPP steps are interleaved with the Newton steps of the KPL
    //   divisions, pinned by scheduling barriers: the two instructions between steps are
    //   the wait states a DPP read needs.
    double num[KPL], den[KPL], rcp[KPL], err[KPL], pk[KPL];
    int ex = -4096;  // the lane's largest e_num - e_den; below every exponent past the last topic
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const int k = lane * KPL + j;
      const int self = k == k0;
      const int ndx = nd[j] - self;
      const int nwx = max(rows[C].nw[j] + dw[j] - self, 0);
      const int nkx = max(nk[j] - self, 0);
      num[j] = (static_cast<double>(ndx) + alpha_k[j]) * (static_cast<double>(nwx) + a.beta);
      den[j] = static_cast<double>(nkx) + a.Vbeta;
      const int e = __builtin_amdgcn_frexp_exp(num[j]) - __builtin_amdgcn_frexp_exp(den[j]);
      if (j == 0) ex = k < K ? e : -4096;
      else if (k < K) ex = max(ex, e);
      rcp[j] = __builtin_amdgcn_rcp(den[j]);
    }
    // between two steps: the KPL operations of one Newton step
#define PS_LDA_GAP KPL
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, 0, "quad_perm:[1,0,3,2] row_mask:0xf bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) err[j] = fma(-den[j], rcp[j], 1.0);
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, PS_LDA_GAP, "quad_perm:[2,3,0,1] row_mask:0xf bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) rcp[j] = fma(rcp[j], err[j], rcp[j]);
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, PS_LDA_GAP, "row_half_mirror row_mask:0xf bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) err[j] = fma(-den[j], rcp[j], 1.0);
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, PS_LDA_GAP, "row_mirror row_mask:0xf bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) rcp[j] = fma(rcp[j], err[j], rcp[j]);
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, PS_LDA_GAP, "row_bcast:15 row_mask:0xa bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) pk[j] = num[j] * rcp[j];
    __builtin_amdgcn_sched_barrier(0);
    PS_LDA_MAX_STEP(ex, PS_LDA_GAP, "row_bcast:31 row_mask:0xc bank_mask:0xf");
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < KPL; ++j) err[j] = fma(-den[j], pk[j], num[j]);
    __builtin_amdgcn_sched_barrier(0);
#undef PS_LDA_GAP
    const int ehi = __builtin_amdgcn_readlane(ex, 63) + 1;  // the KPL corrections before it: its wait state
    int top = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      pk[j] = fma(err[j], rcp[j], pk[j]);  // 0 past the last topic
      top |= pk[j] >= ldexp(1.0, ehi - 1);
    }
    // the largest p_k lies in [2^emax, 2^(emax + 1))
    const int emax = (__ballot(top) != 0 ? ehi : ehi - 1) - 1;
    // integer weights floor(p_k 2^(shift0 - emax)) (the scaling is exact), prefix sums in
    // topic order
    const int shift = a.shift0 - emax;
    uint64_t loc[KPL];
    uint64_t acc = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      acc += static_cast<uint64_t>(floor(ldexp(pk[j], shift)));  // pk = 0 past the last topic
      loc[j] = acc;
    }
    uint64_t total;
    const uint64_t excl = wave_scan(acc, &total) - acc;
    int k1 = k0;
    if (total != 0) {  // always: the largest weight is at least 2^shift0
      const uint64_t target = umulhi64_vec(ru, total);
      const uint64_t m = __ballot(excl + acc > target);
      const int L = __ffsll(static_cast<unsigned long long>(m)) - 1;  // m != 0: the last lane's sum is the total
      int jj = KPL - 1;
#pragma unroll
      for (int j = KPL - 1; j >= 0; --j)
        if (excl + loc[j] > target) jj = j;
      k1 = __builtin_amdgcn_readlane(lane * KPL + jj, L);
    }
    const bool changed = k1 != k0;
    if (changed) {
      const Off rb = rowb * static_cast<Off>(w);
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        const int k = lane * KPL + j;
        const int dl = (k == k1) - (k == k0);
        nd[j] += dl;
        nk[j] += dl;
        dw[j] += dl;
        mydelta.st_if(k < K && (!valid || dl != 0), dw[j], koff[j], rb);
      }
      // lane 0 stores the new topic, and the row's clock tag when the row was of an older clock
      z.st_if(lane == 0, k1, 0u, Off{4} * static_cast<uint32_t>(i));
      mytag.st_if(lane == 0 && !valid, a.tagc, 0u, Off{4} * static_cast<uint32_t>(w));
    }
    // this token becomes the latest forwarded row
#pragma unroll
    for (int f = F - 1; f > 0; --f) {
      fw[f] = fw[f - 1];
      fvalid[f] = fvalid[f - 1];
#pragma unroll
      for (int j = 0; j < KPL; ++j) fdw[f][j] = fdw[f - 1][j];
    }
    if constexpr (F > 0) {
      fw[0] = w;
      fvalid[0] = valid | static_cast<int>(changed);
#pragma unroll
      for (int j = 0; j < KPL; ++j) fdw[0][j] = dw[j];
    }
    constexpr int NF = (C + kDist) % R;
    fetch_rows<KPL, Buf>(view, mydelta, mytag, z, koff, rowb * static_cast<Off>(wf), wf, i + kDist, rows[NF]);
  };
  // whole rotations without an exit inside (an exit path would join the loop's back edge
  // with its latest fetch still in flight, and the wait at the top of the loop would then
  // drain every fetch), then the last tokens
  int i = 0;
  for (;;) {
    const int lim = min(base + kRecStep, n);
    for (; i + R <= lim; i += R) {
      bool more = true;
      seq_steps<0, R>(step, i, n, more);
    }
    if (n <= base + kRecStep) break;
    // i = base + kRecStep: the next block of records
    base = i;
    rv = rv_next;
    rv_next = rec[min(base + kRecStep + lane, last)];
    rnd = splitmix64(rbase ^ static_cast<uint64_t>(static_cast<uint32_t>(rv[2])));
  }
  if (i < n) {
    bool more = true;
    seq_steps<0, R - 1>(step, i, n, more);
  }
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int k = lane * KPL + j;
    if (k < K) {
      ndk.st(nd[j], koff[j], rowb * static_cast<Off>(cur_doc));
      a.tot[p * K + k] = nk[j] - vk[j];
    }
  }
}

// version c+1 = version c + every worker's changes of clock c.  One wavefront per word row
// (lanes over topics as in the sweep): the workers' row tags are read 64 at a time, and the
// own-change rows of the workers that wrote this word in this clock are added, several
// loads in flight (a popular word has a writer in nearly every worker); the last row
// (topic totals) adds the workers' topic-total changes.  Every sum is integer, so the
// result does not depend on the order.
template <int KPL>
__global__ __launch_bounds__(kWave) void k_lda_commit(const int32_t *cur, int32_t *next, const int32_t *delta,
                                                      const int32_t *tag, const int32_t *tot, int64_t V, int32_t K,
                                                      int32_t P, int32_t tagc) {
  const int lane = threadIdx.x;
  const int64_t w = blockIdx.x;
  int acc[KPL];
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int k = lane * KPL + j;
    acc[j] = k < K ? cur[w * K + k] : 0;
  }
  if (w < V) {
    for (int p0 = 0; p0 < P; p0 += kWave) {
      const int pl = p0 + lane;
      const bool hit = pl < P && tag[static_cast<int64_t>(pl) * V + w] == tagc;
      uint64_t m = __ballot(hit);
      // the writers' rows, 8 in flight at a time; a slot past the last writer re-reads
      // worker p0's row (in bounds) and is not added
      constexpr int U = 8;
      while (m != 0) {
        int pp[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          ok[u] = m != 0;
          pp[u] = p0 + (ok[u] ? __ffsll(static_cast<unsigned long long>(m)) - 1 : 0);
          if (ok[u]) m &= m - 1;
        }
        int t[U][KPL];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int32_t *row = delta + (static_cast<int64_t>(pp[u]) * V + w) * K;
#pragma unroll
          for (int j = 0; j < KPL; ++j) {
            const int k = lane * KPL + j;
            t[u][j] = k < K ? row[k] : 0;
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
#pragma unroll
          for (int j = 0; j < KPL; ++j)
            if (ok[u]) acc[j] += t[u][j];
        }
      }
    }
  } else {
    // the topic-total rows, 16 workers' rows in flight at a time
    constexpr int U = 16;
    for (int p0 = 0; p0 < P; p0 += U) {
      int t[U][KPL];
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int j = 0; j < KPL; ++j) {
          const int k = lane * KPL + j;
          t[u][j] = (p0 + u < P && k < K) ? tot[static_cast<int64_t>(p0 + u) * K + k] : 0;
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
#pragma unroll
        for (int j = 0; j < KPL; ++j) acc[j] += t[u][j];
      }
    }
  }
#pragma unroll
  for (int j = 0; j < KPL; ++j) {
    const int k = lane * KPL + j;
    if (k < K) next[w * K + k] = acc[j];
  }
}

// collapsed log p(w, z): per-thread terms over (word, topic) counts, topic totals and
// documents, a fixed-order block reduction into one partial per block
__global__ __launch_bounds__(kLoglikThreads) void k_lda_loglik(const int32_t *n, const int32_t *ndk, int64_t V,
                                                               int32_t K, int64_t D, double alpha, double beta,
                                                               double Vbeta, double *partial) {
  __shared__ double red[kLoglikThreads];
  const int64_t VK = V * K, total = VK + K + D;
  const double lg_beta = lgamma(beta), lg_alpha = lgamma(alpha), Ka = K * alpha;
  double acc = 0.0;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
    if (i < VK) {
      const int32_t x = n[i];
      if (x > 0) acc += lgamma(x + beta) - lg_beta;
    } else if (i < VK + K) {
      acc += lgamma(Vbeta) - lgamma(n[i] + Vbeta);
    } else {
      const int32_t *row = ndk + (i - VK - K) * K;
      int64_t len = 0;
      double t = 0.0;
      for (int k = 0; k < K; ++k) {
        const int32_t x = row[k];
        len += x;
        if (x > 0) t += lgamma(x + alpha) - lg_alpha;
      }
      acc += t + lgamma(Ka) - lgamma(static_cast<double>(len) + Ka);
    }
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = kLoglikThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(kLoglikThreads) void k_lda_sum(const double *partial, int n, double *out) {
  __shared__ double red[kLoglikThreads];
  double acc = 0.0;
  for (int i = threadIdx.x; i < n; i += kLoglikThreads) acc += partial[i];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = kLoglikThreads / 2; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

}  // namespace

struct ps_lda {
  int64_t D = 0, V = 0;
  int32_t K = 0, P = 0, s = 0;
  double alpha = 0, beta = 0, Vbeta = 0;
  int32_t policy = PS_LDA_ESSP, B = 2;
  uint64_t seed = 0;
  bool host_only = false, timing = false, loaded = false;
  bool flat = false;  // 64-bit addresses in the sampling kernel even where the buffer form fits
  int64_t clock = 0, ntok = 0;
  int device = -1;
  hipStream_t stream = nullptr, user_stream = nullptr;
  bool own_stream = false;
  std::string err;
  std::vector<void *> allocations;
  std::vector<int64_t> wbeg;   // B x (P+1) block positions
  std::vector<int64_t> order;  // load index at every block position
  std::vector<int64_t> vlog;
  int4 *rec = nullptr;
  int32_t *z = nullptr, *ndk = nullptr, *ring = nullptr, *delta = nullptr, *tag = nullptr, *tot = nullptr;
  int64_t *wbeg_dev = nullptr;
  double *partial = nullptr;
  struct Ev {
    hipEvent_t a, b;
  };
  std::vector<Ev> events;
  double kernel_ms = 0;
  int64_t kernel_count = 0;
};

namespace {

int lda_fail(ps_lda_t *h, int code, const char *fmt, ...) {
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

#define LDA_TRY(h, expr)                                                                                       \
  do {                                                                                                        \
    hipError_t e_ = (expr);                                                                                   \
    if (e_ != hipSuccess) {                                                                                   \
      if (e_ == hipErrorOutOfMemory) return lda_fail(h, PS_LDA_ENOMEM, "%s: %s", #expr, hipGetErrorString(e_)); \
      return lda_fail(h, PS_LDA_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_));                             \
    }                                                                                                         \
  } while (0)

int lda_alloc(ps_lda_t *h, void **p, size_t bytes) {
  *p = nullptr;
  if (bytes == 0) bytes = 256;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    (void)hipGetLastError();
    if (e == hipErrorOutOfMemory) return lda_fail(h, PS_LDA_ENOMEM, "hipMalloc(%zu bytes): out of memory", bytes);
    return lda_fail(h, PS_LDA_EDEVICE, "hipMalloc(%zu bytes): %s", bytes, hipGetErrorString(e));
  }
  h->allocations.push_back(*p);
  return PS_LDA_OK;
}

int lda_device(ps_lda_t *h) {
  if (h->device < 0) {
    int dev = 0;
    LDA_TRY(h, hipGetDevice(&dev));
    h->device = dev;
  }
  LDA_TRY(h, hipSetDevice(h->device));
  if (!h->stream) {
    if (h->user_stream) {
      h->stream = h->user_stream;
    } else {
      LDA_TRY(h, hipStreamCreateWithFlags(&h->stream, hipStreamNonBlocking));
      h->own_stream = true;
    }
  }
  return PS_LDA_OK;
}

int64_t slot_stride(const ps_lda_t *h) { return (h->V + 1) * h->K; }

template <int KPL>
void launch_sweep(const SweepArgs &a, int P, bool flat, hipStream_t st) {
  if (flat) hipLaunchKernelGGL((k_lda_sweep<KPL, false>), dim3(P), dim3(kWave), 0, st, a);
  else hipLaunchKernelGGL((k_lda_sweep<KPL, true>), dim3(P), dim3(kWave), 0, st, a);
}

template <int KPL>
void launch_commit(const ps_lda_t *h, const int32_t *cur, int32_t *nxt, int32_t tagc) {
  hipLaunchKernelGGL(k_lda_commit<KPL>, dim3(static_cast<unsigned>(h->V + 1)), dim3(kWave), 0, h->stream, cur, nxt,
                     h->delta, h->tag, h->tot, h->V, h->K, h->P, tagc);
}

int sweep(ps_lda_t *h) {
  const int64_t c = h->clock, b = c % h->B, ns = h->s + 2, stride = slot_stride(h);
  const int32_t *cur = h->ring + (c % ns) * stride;
  int32_t *nxt = h->ring + ((c + 1) % ns) * stride;
  SweepArgs a;
  a.rec = h->rec;
  a.z = h->z;
  a.ndk = h->ndk;
  a.ring = h->ring;
  a.delta = h->delta;
  a.tag = h->tag;
  a.tot = h->tot;
  a.wbeg = h->wbeg_dev + b * (h->P + 1);
  a.slot_stride = stride;
  a.V = h->V;
  a.D = h->D;
  a.c = c;
  a.alpha = h->alpha;
  a.beta = h->beta;
  a.Vbeta = h->Vbeta;
  a.seed = h->seed;
  a.K = h->K;
  a.s = h->s;
  a.policy = h->policy;
  a.nslots = static_cast<int32_t>(ns);
  int clog2k = 0;
  while ((int64_t{1} << clog2k) < h->K) ++clog2k;
  a.shift0 = 62 - clog2k;
  a.tagc = static_cast<int32_t>(c + 1);
  // the buffer form of the sampling kernel's tables needs each under 2^31 bytes: the ring
  // slot, a worker's own-change rows and row tags, the doc-topic rows and a worker's topics
  const int64_t big = std::max({stride, h->V * h->K, h->D * h->K, h->ntok + kDist}) * 4;
  const bool flat = h->flat || big >= (int64_t{1} << 31);
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (h->timing) {
    LDA_TRY(h, hipEventCreate(&e0));
    LDA_TRY(h, hipEventRecord(e0, h->stream));
  }
  switch ((h->K + kWave - 1) / kWave) {
    case 1: launch_sweep<1>(a, h->P, flat, h->stream); break;
    case 2: launch_sweep<2>(a, h->P, flat, h->stream); break;
    case 3: launch_sweep<3>(a, h->P, flat, h->stream); break;
    case 4: launch_sweep<4>(a, h->P, flat, h->stream); break;
    case 5: launch_sweep<5>(a, h->P, flat, h->stream); break;
    case 6: launch_sweep<6>(a, h->P, flat, h->stream); break;
    case 7: launch_sweep<7>(a, h->P, flat, h->stream); break;
    default: launch_sweep<8>(a, h->P, flat, h->stream); break;
  }
  LDA_TRY(h, hipGetLastError());
  if (h->timing) {
    LDA_TRY(h, hipEventCreate(&e1));
    LDA_TRY(h, hipEventRecord(e1, h->stream));
    h->events.push_back({e0, e1});
  }
  switch ((h->K + kWave - 1) / kWave) {
    case 1: launch_commit<1>(h, cur, nxt, a.tagc); break;
    case 2: launch_commit<2>(h, cur, nxt, a.tagc); break;
    case 3: launch_commit<3>(h, cur, nxt, a.tagc); break;
    case 4: launch_commit<4>(h, cur, nxt, a.tagc); break;
    case 5: launch_commit<5>(h, cur, nxt, a.tagc); break;
    case 6: launch_commit<6>(h, cur, nxt, a.tagc); break;
    case 7: launch_commit<7>(h, cur, nxt, a.tagc); break;
    default: launch_commit<8>(h, cur, nxt, a.tagc); break;
  }
  LDA_TRY(h, hipGetLastError());
  for (int64_t p = 0; p < h->P; ++p) h->vlog.push_back(view_of(h->policy, h->s, p, c));
  h->clock = c + 1;
  return PS_LDA_OK;
}

}  // namespace

extern "C" {

int ps_lda_create(int64_t D, int64_t V, int32_t K, int32_t P, int32_t s, double alpha, double beta,
                  ps_lda_t **out) {
  if (!out) return PS_LDA_EINVAL;
  *out = nullptr;
  if (D < 1 || V < 1 || D > 0x7fffffff || V > 0x7fffffff) return PS_LDA_EINVAL;
  if (K < 1 || K > kWave * kMaxTopicsPerLane || P < 1 || P > 65536 || s < 0 || s > 1024) return PS_LDA_EINVAL;
  if (!(alpha > 0) || !(beta > 0) || !std::isfinite(alpha) || !std::isfinite(beta)) return PS_LDA_EINVAL;
  ps_lda_t *h = new (std::nothrow) ps_lda_t();
  if (!h) return PS_LDA_ENOMEM;
  h->D = D;
  h->V = V;
  h->K = K;
  h->P = P;
  h->s = s;
  h->alpha = alpha;
  h->beta = beta;
  h->Vbeta = static_cast<double>(V) * beta;
  *out = h;
  return PS_LDA_OK;
}

int ps_lda_set_option(ps_lda_t *h, int32_t key, int64_t value) {
  if (!h) return PS_LDA_EINVAL;
  if (h->loaded) return lda_fail(h, PS_LDA_ESTATE, "options must be set before ps_lda_load");
  switch (key) {
    case PS_LDA_OPT_POLICY:
      if (value < PS_LDA_SSP_LAZY || value > PS_LDA_ESSP) return lda_fail(h, PS_LDA_EINVAL, "unknown policy %lld", (long long)value);
      h->policy = static_cast<int32_t>(value);
      return PS_LDA_OK;
    case PS_LDA_OPT_MB_BLOCKS:
      if (value < 1 || value > 65536) return lda_fail(h, PS_LDA_EINVAL, "blocks must be in [1, 65536]");
      h->B = static_cast<int32_t>(value);
      return PS_LDA_OK;
    case PS_LDA_OPT_SEED:
      h->seed = static_cast<uint64_t>(value);
      return PS_LDA_OK;
    case PS_LDA_OPT_HOST_ONLY:
      h->host_only = value != 0;
      return PS_LDA_OK;
    case PS_LDA_OPT_TIMING:
      h->timing = value != 0;
      return PS_LDA_OK;
    case PS_LDA_OPT_FLAT_ADDRESSING:
      h->flat = value != 0;
      return PS_LDA_OK;
    default:
      return lda_fail(h, PS_LDA_EINVAL, "unknown option %d", key);
  }
}

int ps_lda_set_stream(ps_lda_t *h, void *hip_stream) {
  if (!h) return PS_LDA_EINVAL;
  if (h->stream) (void)hipStreamSynchronize(h->stream);
  if (h->stream && h->own_stream) {
    (void)hipStreamDestroy(h->stream);
    h->own_stream = false;
  }
  h->stream = nullptr;
  h->user_stream = static_cast<hipStream_t>(hip_stream);
  if (h->loaded && !h->host_only) return lda_device(h);
  return PS_LDA_OK;
}

namespace {
int load_tokens(ps_lda_t *h, const int32_t *doc, const int32_t *word, const int32_t *z0, int64_t n);
}

int ps_lda_load(ps_lda_t *h, const int32_t *doc, const int32_t *word, const int32_t *z0, int64_t n) {
  if (!h) return PS_LDA_EINVAL;
  try {
    return load_tokens(h, doc, word, z0, n);
  } catch (const std::bad_alloc &) {
    return lda_fail(h, PS_LDA_ENOMEM, "host memory for the token layout of %lld tokens", (long long)n);
  }
}

}  // extern "C"

namespace {
int load_tokens(ps_lda_t *h, const int32_t *doc, const int32_t *word, const int32_t *z0, int64_t n) {
  if (h->loaded) return lda_fail(h, PS_LDA_ESTATE, "tokens already loaded");
  if (n < 0 || n > 0x7fffffff) return lda_fail(h, PS_LDA_EINVAL, "token count %lld out of range", (long long)n);
  if (n > 0 && (!doc || !word || !z0)) return lda_fail(h, PS_LDA_EINVAL, "null token array");
  for (int64_t t = 0; t < n; ++t) {
    if (doc[t] < 0 || doc[t] >= h->D) return lda_fail(h, PS_LDA_EINVAL, "token %lld: document out of range", (long long)t);
    if (word[t] < 0 || word[t] >= h->V) return lda_fail(h, PS_LDA_EINVAL, "token %lld: word out of range", (long long)t);
    if (z0[t] < 0 || z0[t] >= h->K) return lda_fail(h, PS_LDA_EINVAL, "token %lld: topic out of range", (long long)t);
  }
  const int64_t P = h->P, B = h->B, K = h->K, V = h->V;
  {
    // every weight p_k = num / den of the sampler, its numerator (n_dk + alpha)(n_wk + beta)
    // and its denominator n_k + V beta must lie in [2^-700, 2^700]: then p_k is a normal fp64
    // number (its exponent sets the weights' scale) and the sampler's short division (no
    // range scaling, no special cases) is exact.  num lies between alpha beta and (longest
    // document + alpha)(tokens + beta), den between V beta and tokens + V beta, and p_k
    // between alpha beta / (tokens + V beta) and (longest document + alpha)(tokens + beta) /
    // (V beta)
    std::vector<int64_t> len(static_cast<size_t>(h->D), 0);
    int64_t lmax = 0;
    for (int64_t t = 0; t < n; ++t) lmax = std::max(lmax, ++len[doc[t]]);
    const double num_hi = (static_cast<double>(lmax) + h->alpha) * (static_cast<double>(n) + h->beta);
    const double num_lo = h->alpha * h->beta;
    const double den_hi = static_cast<double>(n) + h->Vbeta, den_lo = h->Vbeta;
    const double lo = num_lo / den_hi, hi = num_hi / den_lo;
    const double top = std::ldexp(1.0, 700), bottom = std::ldexp(1.0, -700);
    for (const double x : {num_lo, num_hi, den_lo, den_hi, lo, hi})
      if (!(x >= bottom && x <= top))
        return lda_fail(h, PS_LDA_EINVAL,
                        "topic weights, their numerators or denominators leave [2^-700, 2^700]: weights from "
                        "%.3g to %.3g, numerators from %.3g to %.3g, denominators from %.3g to %.3g",
                        lo, hi, num_lo, num_hi, den_lo, den_hi);
  }
  // processing order: block, worker (document mod P), document, load index
  std::vector<std::pair<uint64_t, int64_t>> key(static_cast<size_t>(n));
  std::vector<int64_t> count(static_cast<size_t>(B * P) + 1, 0);
  for (int64_t t = 0; t < n; ++t) {
    const uint64_t b = B == 1 ? 0 : splitmix64(h->seed ^ static_cast<uint64_t>(t)) % static_cast<uint64_t>(B);
    const uint64_t bucket = b * static_cast<uint64_t>(P) + static_cast<uint64_t>(doc[t] % P);
    key[t] = {(bucket << 32) | static_cast<uint32_t>(doc[t]), t};
    count[bucket + 1] += 1;
  }
  std::sort(key.begin(), key.end());
  for (int64_t i = 0; i < B * P; ++i) count[i + 1] += count[i];
  h->wbeg.assign(static_cast<size_t>(B * (P + 1)), 0);
  for (int64_t b = 0; b < B; ++b)
    for (int64_t p = 0; p <= P; ++p) h->wbeg[b * (P + 1) + p] = count[b * P + p];
  h->order.resize(static_cast<size_t>(n));
  for (int64_t q = 0; q < n; ++q) h->order[q] = key[q].second;
  h->ntok = n;
  if (h->host_only) {
    h->loaded = true;
    return PS_LDA_OK;
  }
  int rc = lda_device(h);
  if (rc) return rc;
  std::vector<int4> rec(static_cast<size_t>(n));
  std::vector<int32_t> zq(static_cast<size_t>(n));
  std::vector<int32_t> ndk(static_cast<size_t>(h->D * K), 0);
  std::vector<int32_t> n0(static_cast<size_t>((V + 1) * K), 0);
  for (int64_t q = 0; q < n; ++q) {
    const int64_t t = h->order[q];
    rec[q] = make_int4(word[t], doc[t], static_cast<int>(t), 0);
    zq[q] = z0[t];
    ndk[static_cast<int64_t>(doc[t]) * K + z0[t]] += 1;
    n0[static_cast<int64_t>(word[t]) * K + z0[t]] += 1;
    n0[V * K + z0[t]] += 1;
  }
  const int64_t stride = slot_stride(h), ns = h->s + 2;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->rec), sizeof(int4) * n))) return rc;
  // kDist entries past the end: a worker's fetches past its last token read them (unused)
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->z), sizeof(int32_t) * (n + kDist)))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->ndk), sizeof(int32_t) * h->D * K))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->ring), sizeof(int32_t) * stride * ns))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->delta), sizeof(int32_t) * P * V * K))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->tag), sizeof(int32_t) * P * V))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->tot), sizeof(int32_t) * P * K))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->wbeg_dev), sizeof(int64_t) * h->wbeg.size()))) return rc;
  if ((rc = lda_alloc(h, reinterpret_cast<void **>(&h->partial), sizeof(double) * (kLoglikBlocks + 1)))) return rc;
  if (n > 0) {
    LDA_TRY(h, hipMemcpy(h->rec, rec.data(), sizeof(int4) * n, hipMemcpyHostToDevice));
    LDA_TRY(h, hipMemcpy(h->z, zq.data(), sizeof(int32_t) * n, hipMemcpyHostToDevice));
  }
  LDA_TRY(h, hipMemcpy(h->ndk, ndk.data(), sizeof(int32_t) * ndk.size(), hipMemcpyHostToDevice));
  LDA_TRY(h, hipMemset(h->ring, 0, sizeof(int32_t) * stride * ns));
  LDA_TRY(h, hipMemcpy(h->ring, n0.data(), sizeof(int32_t) * n0.size(), hipMemcpyHostToDevice));
  LDA_TRY(h, hipMemset(h->tag, 0, sizeof(int32_t) * P * V));
  LDA_TRY(h, hipMemcpy(h->wbeg_dev, h->wbeg.data(), sizeof(int64_t) * h->wbeg.size(), hipMemcpyHostToDevice));
  LDA_TRY(h, hipDeviceSynchronize());
  h->loaded = true;
  return PS_LDA_OK;
}
}  // namespace

extern "C" {

int ps_lda_clock(ps_lda_t *h, int32_t n) {
  if (!h || n < 0) return PS_LDA_EINVAL;
  if (!h->loaded) return lda_fail(h, PS_LDA_ESTATE, "ps_lda_clock before ps_lda_load");
  if (h->host_only) return lda_fail(h, PS_LDA_ESTATE, "host-only handle: no device work");
  if (h->clock + n >= 0x7fffffff) return lda_fail(h, PS_LDA_EINVAL, "clock count overflows");
  int rc = lda_device(h);
  if (rc) return rc;
  for (int32_t i = 0; i < n; ++i)
    if ((rc = sweep(h))) return rc;
  return PS_LDA_OK;
}

int ps_lda_loglik(ps_lda_t *h, double *out) {
  if (!h || !out) return PS_LDA_EINVAL;
  if (!h->loaded || h->host_only) return lda_fail(h, PS_LDA_ESTATE, "no device state");
  int rc = lda_device(h);
  if (rc) return rc;
  const int32_t *n = h->ring + (h->clock % (h->s + 2)) * slot_stride(h);
  hipLaunchKernelGGL(k_lda_loglik, dim3(kLoglikBlocks), dim3(kLoglikThreads), 0, h->stream, n, h->ndk, h->V, h->K,
                     h->D, h->alpha, h->beta, h->Vbeta, h->partial);
  hipLaunchKernelGGL(k_lda_sum, dim3(1), dim3(kLoglikThreads), 0, h->stream, h->partial, kLoglikBlocks,
                     h->partial + kLoglikBlocks);
  LDA_TRY(h, hipGetLastError());
  LDA_TRY(h, hipMemcpyAsync(out, h->partial + kLoglikBlocks, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  LDA_TRY(h, hipStreamSynchronize(h->stream));
  return PS_LDA_OK;
}

int ps_lda_get_clock(ps_lda_t *h, int64_t *clock) {
  if (!h || !clock) return PS_LDA_EINVAL;
  *clock = h->clock;
  return PS_LDA_OK;
}

}  // extern "C"

namespace {
int export_state(ps_lda_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len);
}

extern "C" {

int ps_lda_export(ps_lda_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len) {
  if (!h || !len) return PS_LDA_EINVAL;
  try {
    return export_state(h, kind, block, buf, cap, len);
  } catch (const std::bad_alloc &) {
    return lda_fail(h, PS_LDA_ENOMEM, "host staging memory for export %d", kind);
  }
}

}  // extern "C"

namespace {
int export_state(ps_lda_t *h, int32_t kind, int32_t block, void *buf, int64_t cap, int64_t *len) {
  if (!h->loaded && kind != PS_LDA_X_VERSION_LOG) return lda_fail(h, PS_LDA_ESTATE, "nothing loaded");
  const bool device_kind = kind == PS_LDA_X_Z || kind == PS_LDA_X_NDK || kind == PS_LDA_X_NWK;
  if (device_kind && h->host_only) return lda_fail(h, PS_LDA_ESTATE, "host-only handle: no device state");
  int64_t n;
  switch (kind) {
    case PS_LDA_X_Z: n = h->ntok; break;
    case PS_LDA_X_NDK: n = h->D * h->K; break;
    case PS_LDA_X_NWK: n = slot_stride(h); break;
    case PS_LDA_X_VERSION_LOG: n = static_cast<int64_t>(h->vlog.size()); break;
    case PS_LDA_X_BLOCK_ORDER:
      if (block < 0 || block >= h->B) return lda_fail(h, PS_LDA_EINVAL, "block %d out of range", block);
      n = h->wbeg[block * (h->P + 1) + h->P] - h->wbeg[block * (h->P + 1)];
      break;
    default: return lda_fail(h, PS_LDA_EINVAL, "unknown export %d", kind);
  }
  *len = n;
  if (!buf) return PS_LDA_OK;
  if (cap < n) return lda_fail(h, PS_LDA_EINVAL, "buffer holds %lld, needs %lld", (long long)cap, (long long)n);
  if (n == 0) return PS_LDA_OK;
  if (device_kind) {
    int rc = lda_device(h);
    if (rc) return rc;
    LDA_TRY(h, hipStreamSynchronize(h->stream));
  }
  switch (kind) {
    case PS_LDA_X_Z: {
      std::vector<int32_t> zq(static_cast<size_t>(n));
      LDA_TRY(h, hipMemcpy(zq.data(), h->z, sizeof(int32_t) * n, hipMemcpyDeviceToHost));
      int32_t *o = static_cast<int32_t *>(buf);
      for (int64_t q = 0; q < n; ++q) o[h->order[q]] = zq[q];
      break;
    }
    case PS_LDA_X_NDK: LDA_TRY(h, hipMemcpy(buf, h->ndk, sizeof(int32_t) * n, hipMemcpyDeviceToHost)); break;
    case PS_LDA_X_NWK:
      LDA_TRY(h, hipMemcpy(buf, h->ring + (h->clock % (h->s + 2)) * slot_stride(h), sizeof(int32_t) * n,
                           hipMemcpyDeviceToHost));
      break;
    case PS_LDA_X_VERSION_LOG: std::memcpy(buf, h->vlog.data(), sizeof(int64_t) * n); break;
    case PS_LDA_X_BLOCK_ORDER:
      std::memcpy(buf, h->order.data() + h->wbeg[block * (h->P + 1)], sizeof(int64_t) * n);
      break;
  }
  return PS_LDA_OK;
}

}  // namespace

extern "C" {

int ps_lda_kernel_time(ps_lda_t *h, double *ms, int64_t *count) {
  if (!h || !ms || !count) return PS_LDA_EINVAL;
  if (h->stream) LDA_TRY(h, hipStreamSynchronize(h->stream));
  for (auto &ev : h->events) {
    float t = 0;
    LDA_TRY(h, hipEventElapsedTime(&t, ev.a, ev.b));
    h->kernel_ms += t;
    h->kernel_count += 1;
    (void)hipEventDestroy(ev.a);
    (void)hipEventDestroy(ev.b);
  }
  h->events.clear();
  *ms = h->kernel_ms;
  *count = h->kernel_count;
  return PS_LDA_OK;
}

const char *ps_lda_last_error(const ps_lda_t *h) {
  if (!h) return "null handle";
  return h->err.c_str();
}

void ps_lda_destroy(ps_lda_t *h) {
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
