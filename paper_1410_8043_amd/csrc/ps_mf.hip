// ps_mf: clocked SSP / ESSP matrix-factorization SGD, P logical workers on one MI355X.
// C-ABI entry points are declared in include/ps_mf.h; this file holds the gfx950 kernels
// and the host orchestration around them.
//
// Device state (HBM):
//   ring      : (s+1) slots, each [L: users x Kp | R: items x Kp] fp32 row-major; version v
//               lives in slot v mod (s+1); Kp = K rounded up to a power of two >= 8, the
//               padding columns are kept at zero in every slot.
//   per block : the ratings twice, as work units of the user-major and of the item-major
//               sweep (see layout.h), user and item rating counts (items also per worker
//               class).
//   partial_u : [units, Kp] one row of sum_j e_ij R^v_j per user-major unit;
//   partial_i : [units, Kp] one row of sum_i e_ij L^v_i per item-major unit.
//   slot table: for clock c, the ring slot each worker class reads (Section 3.2 view).
//
// One clock c (Section 3.1 update, Section 3.2 SSP view, Section 4 coalesced commit).
// Neither sweep uses atomics: a unit keeps one row (the stationary side) in registers,
// gathers the other side's rows from a tile that stays in one XCD's L2, recomputes the
// residual e = D_ij - L^v_i . R^v_j and writes one partial row.
//   sweep    : the item-major and the user-major units in one launch;
//   commit   : in one launch, L^{c+1}_i = L^c_i + scale_i (sum of i's partial rows -
//              n_i lambda L^v_i) (users without a rating in the block keep L^c_i) and
//              R^{c+1}_j = R^c_j + scale_j (sum of j's partial rows - lambda sum_class
//              n_j^(class) R^{v(class)}_j).
// Both sweeps read versions <= c only; finalize and commit write version c+1 into the
// slot that held version c-s, after both sweeps are done with it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <type_traits>
#include <vector>

#include "../../include/ps_mf.h"
#include "layout.h"

// The fp64 partial sums of the loss for callers that cannot allocate (ps_mf_loss_noalloc):
// a fixed array in every GPU's memory, held until the process ends.  Entries
// [0, kNoAllocPartials) take the per-workgroup partials, the last one the final sum.  Host
// code never passes the array's name to a kernel (on the host it is a stand-in, not a
// device address): each device's address comes from hipGetSymbolAddress.
constexpr int64_t kNoAllocPartials = int64_t{1} << 18;  // 2 MiB of partials
static __device__ __align__(256) double scratch[kNoAllocPartials + 1];

namespace {

constexpr int kBlock = 256;       // threads per workgroup of the small kernels (4 wavefronts)
#ifndef PS_MF_CELL_THREADS
#define PS_MF_CELL_THREADS 1024
#endif
#ifndef PS_MF_CELL_TILE_FLOATS
#define PS_MF_CELL_TILE_FLOATS 40960
#endif
constexpr int kSweepBlock = PS_MF_CELL_THREADS;     // threads per cell workgroup (1024: 16 wavefronts)
constexpr int kTileFloats = PS_MF_CELL_TILE_FLOATS; // LDS sub-tile of a cell (40960: 160 KiB = ts rows of Kp floats)
static_assert(kSweepBlock % 256 == 0 && kSweepBlock <= 1024, "cell workgroups hold whole 256-thread quarters");
static_assert(kTileFloats % 512 == 0 && kTileFloats * 4 <= 160 * 1024, "a cell sub-tile holds whole 512-wide rows in LDS");
constexpr int kLossSegment = 512;  // ratings per lane group of the loss
// automatic threshold of the dense (MFMA) tiles: ratings per 64 x 64 tile
#ifndef PS_MF_DENSE_AUTO
#define PS_MF_DENSE_AUTO 800
#endif
constexpr int kDenseAuto = PS_MF_DENSE_AUTO;
// ratings per minibatch block from which the automatic split uses dense tiles and LDS cells
constexpr int64_t kSplitMinRatings = int64_t{1} << 24;
// dense cells per direction the layout aims at (more cells: shorter runs and a shorter tail,
// but one partial row per cell and row)
#ifndef PS_MF_DENSE_CELLS
#define PS_MF_DENSE_CELLS 1024
#endif
constexpr int kMaxKp = 512;
// 1: the LDS cells run on a third internal stream beside the dense tiles and the units
#ifndef PS_MF_CELL_STREAM
#define PS_MF_CELL_STREAM 1
#endif
constexpr int kXcds = psmf::kXcds;
#ifndef PS_MF_ROWS_IN_FLIGHT
#define PS_MF_ROWS_IN_FLIGHT 4
#endif
constexpr int kRowsInFlight = PS_MF_ROWS_IN_FLIGHT;  // gathered rows loaded before their use (divides 8)
// rows in flight for E floats per lane: the 512-wide rows keep one (registers are capped
// at 128 per lane with 16 wavefronts per CU); narrow rows (E <= 8 floats per lane) keep
// PS_MF_NARROW_ROWS_IN_FLIGHT, so that enough bytes are in flight per CU to cover the L2
// latency
#ifndef PS_MF_NARROW_ROWS_IN_FLIGHT
#define PS_MF_NARROW_ROWS_IN_FLIGHT 8
#endif
template <int E>
constexpr int rows_in_flight() { return E >= 32 ? 1 : E >= 16 ? kRowsInFlight : PS_MF_NARROW_ROWS_IN_FLIGHT; }
// the cells also hold the next 8 (row, value) pairs: two rows in flight from 16 floats on
template <int E>
constexpr int cell_rows_in_flight() { return E >= 32 ? 1 : E >= 16 ? 2 : kRowsInFlight; }

// ------------------------------------------------------------------ device helpers
// A factor row of Kp = G*E floats is spread over a lane group of G lanes: lane g holds the
// float4 chunks q*G + g (q = 0 .. E/4-1), so each float4 load of the group reads 16*G
// contiguous bytes.
template <int G, int E>
__device__ __forceinline__ void load_row(float (&d)[E], const float *__restrict__ row, int g) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q) {
    const float4 t = *reinterpret_cast<const float4 *>(row + 4 * (q * G + g));
    d[4 * q] = t.x; d[4 * q + 1] = t.y; d[4 * q + 2] = t.z; d[4 * q + 3] = t.w;
  }
}

template <int G, int E>
__device__ __forceinline__ void store_row(float *__restrict__ row, const float (&d)[E], int g) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q)
    *reinterpret_cast<float4 *>(row + 4 * (q * G + g)) = make_float4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
}

// LDS rows of a cell: with G = 8 lanes per group, the two groups of a 16-lane LDS access
// would read the same 32 of the 64 banks (rows are multiples of 512 bytes apart); odd
// groups therefore hold their chunks in the order 1,0,3,2,... (register chunk h is row
// chunk h ^ 1) and the pair reads different halves.  The stationary row and the partial
// row of such a group use the same order.
template <int G, int E>
constexpr bool swizzled() { return G == 8 && E >= 8; }

template <int G, int E>
__device__ __forceinline__ void load_row_sw(float (&d)[E], const float *__restrict__ row, int g, int rot) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q) {
    const float4 t = *reinterpret_cast<const float4 *>(row + 4 * ((q ^ rot) * G + g));
    d[4 * q] = t.x; d[4 * q + 1] = t.y; d[4 * q + 2] = t.z; d[4 * q + 3] = t.w;
  }
}

template <int G, int E>
__device__ __forceinline__ void store_row_sw(float *__restrict__ row, const float (&d)[E], int g, int rot) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q)
    *reinterpret_cast<float4 *>(row + 4 * ((q ^ rot) * G + g)) =
        make_float4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

// Data that a clock touches once -- rating streams, stationary rows, partial rows, dense
// values and residuals -- may be loaded and stored non-temporally, so that it does not
// evict from L2 the gathered rows that other work units reuse.  Which of the three
// streams are non-temporal is a build choice (PS_MF_NT_LOADS: the sweeps' once-read
// data; PS_MF_NT_STORES: partial rows and residuals; PS_MF_NT_COMMIT: the commit's
// partial-row reads).
#ifndef PS_MF_NT_LOADS
#define PS_MF_NT_LOADS 0
#endif
#ifndef PS_MF_NT_STORES
#define PS_MF_NT_STORES 1
#endif
#ifndef PS_MF_NT_COMMIT
#define PS_MF_NT_COMMIT 1
#endif
template <class T>
__device__ __forceinline__ T ld_once(const T *p) {
  if constexpr (PS_MF_NT_LOADS != 0) return __builtin_nontemporal_load(p);
  else return *p;
}
template <class T>
__device__ __forceinline__ void st_once(T *p, T v) {
  if constexpr (PS_MF_NT_STORES != 0) __builtin_nontemporal_store(v, p);
  else *p = v;
}
template <class T>
__device__ __forceinline__ T ld_partial(const T *p) {
  if constexpr (PS_MF_NT_COMMIT != 0) return __builtin_nontemporal_load(p);
  else return *p;
}

template <int G, int E>
__device__ __forceinline__ void load_row_once(float (&d)[E], const float *__restrict__ row, int g) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q) {
    const f32x4 t = ld_once(reinterpret_cast<const f32x4 *>(row + 4 * (q * G + g)));
    d[4 * q] = t[0]; d[4 * q + 1] = t[1]; d[4 * q + 2] = t[2]; d[4 * q + 3] = t[3];
  }
}

template <int G, int E>
__device__ __forceinline__ void store_row_once(float *__restrict__ row, const float (&d)[E], int g, int rot = 0) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q)
    st_once(reinterpret_cast<f32x4 *>(row + 4 * ((q ^ rot) * G + g)), f32x4{d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]});
}

template <int G, int E>
__device__ __forceinline__ void load_row_sw_once(float (&d)[E], const float *__restrict__ row, int g, int rot) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q) {
    const f32x4 t = ld_once(reinterpret_cast<const f32x4 *>(row + 4 * ((q ^ rot) * G + g)));
    d[4 * q] = t[0]; d[4 * q + 1] = t[1]; d[4 * q + 2] = t[2]; d[4 * q + 3] = t[3];
  }
}

// Sum over the G lanes of an aligned lane group with DPP moves inside a 16-lane row:
// quad_perm [1,0,3,2] (xor 1), quad_perm [2,3,0,1] (xor 2), row_half_mirror (the other
// quad of the 8), row_mirror (the other 8 of the 16).  Every lane gets the total.
template <int G>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(G == 2 || G == 4 || G == 8 || G == 16, "lane groups live inside one DPP row");
  // every source lane of these patterns lies inside the row, so bound_ctrl (zero for an
  // invalid source) never applies; with it the compiler folds each move into v_add_f32_dpp
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));
  if constexpr (G >= 4) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
  if constexpr (G >= 8) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, true));
  if constexpr (G >= 16) v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, true));
  return v;
}

// residual e = r - x . y of one rating (x stationary, y gathered)
template <int G, int E>
__device__ __forceinline__ float residual(const float (&x)[E], const float (&y)[E], float r) {
  float p = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) p = fmaf(x[e], y[e], p);
  return r - group_sum<G>(p);
}

struct UnitArgs {
  const int32_t *unit_x, *unit_cls, *unit_len, *unit_out;
  const int64_t *unit_beg;
  const int64_t *xcd_off;   // [kXcds + 1]
  const int32_t *y;         // gathered row of each rating
  const float *val;
  const int32_t *cls_slot;  // ring slot read by each worker class at this clock
  const float *ring;
  int64_t slot_stride;      // floats per slot
  int64_t x_off, y_off;     // offsets of the stationary and the gathered table in a slot
  int64_t y_bytes;          // bytes of the gathered table (< 2^32)
  float *partial;           // [units, Kp]
  // per-row policies: the ring slot of every stationary / gathered row (null: the class
  // slot), tables of rows_per_class entries per worker class (0: one entry per row)
  const int32_t *rs_x, *rs_y;
  int64_t rs_x_cls, rs_y_cls;
  // user-major units: sole[x] = 1 where x's only partial row is one unit's.  Such a unit
  // writes x's new version itself (as the commit would) when x's view is not the new
  // version's slot: no one reads x's row of that slot during the sweep.  Null: never.
  const uint8_t *sole;
  const int32_t *xcount;    // [x] ratings of x in the block
  int32_t slot_c, slot_n;
  const float *base_rows;   // the x table of version c (slot_c)
  float *new_rows;          // the x table of version c + 1 (slot_n)
  float eta, lambda;
  int32_t rowmean;
};

// one element of a committed row: base + scale (sum of partial rows - n lambda view)
__device__ __forceinline__ float commit_elem(float base, float sc, float d, float nl, float view) {
  return fmaf(sc, fmaf(-nl, view, d), base);
}

// The unit processed by lane group `grp` of workgroup `block` (counted within its sweep;
// the first sweep's grid is a multiple of 8, so workgroup b of either sweep runs on XCD
// b mod 8) takes the units of that XCD's chunk; -1 if there is none.
__device__ __forceinline__ int64_t unit_of(const UnitArgs &a, int block, int grp, int groups_per_wg) {
  const int xcd = block % kXcds;
  const int64_t local = static_cast<int64_t>(block / kXcds) * groups_per_wg + grp;
  const int64_t first = a.xcd_off[xcd];
  return local < a.xcd_off[xcd + 1] - first ? first + local : -1;
}

// 32-bit-offset loads from one factor table through a buffer resource (CDNA word 3
// 0x00020000: raw, untyped dword access); offsets past num_bytes read as zero.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t table_rsrc(const float *base, int64_t num_bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(base), static_cast<short>(0),
                                           static_cast<int>(static_cast<uint32_t>(num_bytes)), 0x00020000);
}

template <int G, int E>
__device__ __forceinline__ void load_row_rsrc(float (&d)[E], __amdgpu_buffer_rsrc_t rs, uint32_t row_bytes, int g) {
#pragma unroll
  for (int q = 0; q < E / 4; ++q) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(row_bytes + 16u * (q * G + g)), 0, 0);
    d[4 * q] = __uint_as_float(t[0]);
    d[4 * q + 1] = __uint_as_float(t[1]);
    d[4 * q + 2] = __uint_as_float(t[2]);
    d[4 * q + 3] = __uint_as_float(t[3]);
  }
}

// One lane group per work unit: acc = sum_t (val_t - x . Y_{y_t}) Y_{y_t} over the unit's
// ratings, x the unit's stationary row; acc -> the unit's partial row.  The unit's
// (row, value) pairs are read 8 at a time with one 32-byte load per lane group (a unit
// starts at a multiple of 8 entries and is padded to one); kRowsInFlight gathered rows
// are loaded before they are used.
template <int G, int E, bool PerRow>
__device__ __forceinline__ void run_unit(const UnitArgs &a, int64_t unit, int g) {
  constexpr int Kp = G * E;
  constexpr int RF = rows_in_flight<E>();
  // every unit of a wavefront reads the same class (the layout pads class changes to whole
  // wavefronts), so the class slot and the buffer resource are wave-uniform; under the
  // per-row policies each row has its own slot instead and the rows are read through
  // 64-bit addresses
  const int cls = __builtin_amdgcn_readfirstlane(a.unit_cls[unit]);
  const int sv = PerRow ? 0 : __builtin_amdgcn_readfirstlane(a.cls_slot[cls]);
  const float *__restrict__ V = a.ring + sv * a.slot_stride;
  const __amdgpu_buffer_rsrc_t ys = table_rsrc(V + a.y_off, a.y_bytes);
  const int32_t *__restrict__ rs_y = PerRow ? a.rs_y + cls * a.rs_y_cls : nullptr;
  const int64_t beg = a.unit_beg[unit];
  const int n = a.unit_len[unit];
  const i32x4 *__restrict__ yi = reinterpret_cast<const i32x4 *>(a.y + beg);
  const f32x4 *__restrict__ vr = reinterpret_cast<const f32x4 *>(a.val + beg);
  float x[E], acc[E];
  const int32_t xr = a.unit_x[unit];
  const int64_t xs = PerRow ? a.rs_x[cls * a.rs_x_cls + xr] : sv;
  load_row_once<G, E>(x, a.ring + xs * a.slot_stride + a.x_off + static_cast<int64_t>(xr) * Kp, g);
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  // the next 8 (row, value) pairs are loaded while the current 8 are swept
  i32x4 ni0 = {0, 0, 0, 0}, ni1 = {0, 0, 0, 0};
  f32x4 nv0 = {0.f, 0.f, 0.f, 0.f}, nv1 = {0.f, 0.f, 0.f, 0.f};
  if (n > 0) { ni0 = ld_once(yi); ni1 = ld_once(yi + 1); nv0 = ld_once(vr); nv1 = ld_once(vr + 1); }
  for (int t0 = 0; t0 < n; t0 += 8) {
    const i32x4 i0 = ni0, i1 = ni1;
    const f32x4 v0 = nv0, v1 = nv1;
    if (t0 + 8 < n) {
      ni0 = ld_once(yi + t0 / 4 + 2); ni1 = ld_once(yi + t0 / 4 + 3);
      nv0 = ld_once(vr + t0 / 4 + 2); nv1 = ld_once(vr + t0 / 4 + 3);
    }
    const int idx[8] = {i0[0], i0[1], i0[2], i0[3], i1[0], i1[1], i1[2], i1[3]};
    const float val[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
    for (int q = 0; q < 8; q += RF) {
      if (t0 + q >= n) break;  // only padding left
      float y[RF][E];
#pragma unroll
      for (int w = 0; w < RF; ++w) {
        if constexpr (PerRow) {
          const int32_t r = idx[q + w];
          load_row<G, E>(y[w], a.ring + static_cast<int64_t>(rs_y[r]) * a.slot_stride + a.y_off +
                                   static_cast<int64_t>(r) * Kp, g);
        } else {
          load_row_rsrc<G, E>(y[w], ys, static_cast<uint32_t>(idx[q + w]) * (Kp * 4u), g);
        }
      }
#pragma unroll
      for (int w = 0; w < RF; ++w) {
        // padding entries (row 0, value 0, past the unit's n ratings) contribute nothing
        const float e_all = residual<G, E>(x, y[w], val[q + w]);
        const float err = (t0 + q + w < n) ? e_all : 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e) acc[e] = fmaf(err, y[w][e], acc[e]);
      }
    }
  }
  if (a.sole && n > 0 && a.sole[xr] && xs != a.slot_n) {
    // x's new version, exactly as the commit forms it from one partial row
    float base[E];
    if (xs == a.slot_c) {
#pragma unroll
      for (int e = 0; e < E; ++e) base[e] = x[e];
    } else {
      load_row_once<G, E>(base, a.base_rows + static_cast<int64_t>(xr) * Kp, g);
    }
    const int cnt = a.xcount[xr];
    const float sc = a.rowmean ? a.eta / static_cast<float>(cnt) : a.eta;
    const float nl = static_cast<float>(cnt) * a.lambda;
#pragma unroll
    for (int e = 0; e < E; ++e) base[e] = commit_elem(base[e], sc, acc[e] + 0.f, nl, x[e]);
    store_row_once<G, E>(a.new_rows + static_cast<int64_t>(xr) * Kp, base, g);
  } else {
    store_row_once<G, E>(a.partial + static_cast<int64_t>(a.unit_out[unit]) * Kp, acc, g);
  }
}

struct CellArgs {
  const int32_t *step_rows;      // [nsteps * ts]
  const int32_t *cell_x, *cell_cls, *cell_step_ptr, *cell_steps, *run_beg, *run_len, *cell_out;
  const uint16_t *ly;
  const float *lv;
  const int32_t *cls_slot;
  const float *ring;
  int64_t slot_stride, x_off, y_off;
  int32_t ts;
  float *partial;
  const float *zero;           // Kp zeros: the source of empty staged rows
  const int32_t *rs_x, *rs_y;  // per-row policies (see UnitArgs)
  int64_t rs_x_cls, rs_y_cls;
};

// One cell per workgroup: lane group q keeps the stationary row x_q in registers; for each
// step the workgroup copies the step's ts gathered rows into LDS, then every lane group
// sweeps its row's ratings inside the sub-tile (rows read from LDS).  The partial row of
// each used group is written at the end.
template <int G, int E>
__device__ __forceinline__ void run_cell(const CellArgs &c, int64_t cell, float4 *tile) {
  constexpr int Kp = G * E;
  constexpr int RF = cell_rows_in_flight<E>();
  constexpr int NG = kSweepBlock / G;
  constexpr int Q4 = Kp / 4;  // float4 per row
  const int g = threadIdx.x & (G - 1);
  const int grp = threadIdx.x / G;
  const int cls = c.cell_cls[cell];  // one class per cell: uniform
  const bool per_row = c.rs_x != nullptr;
  const int sv = per_row ? 0 : c.cls_slot[cls];
  const float *__restrict__ V = c.ring + sv * c.slot_stride;
  const int32_t xr = c.cell_x[cell * NG + grp];
  const int rot = swizzled<G, E>() ? (grp & 1) : 0;
  const uint32_t lane_bytes = static_cast<uint32_t>(rot * G + g) * 16u;  // < 32 * G: below a row's size
  const char *tile_bytes = reinterpret_cast<const char *>(tile);
  float x[E], acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) { x[e] = 0.f; acc[e] = 0.f; }
  if (xr >= 0) {
    const int64_t xs = per_row ? c.rs_x[cls * c.rs_x_cls + xr] : sv;
    load_row_sw_once<G, E>(x, c.ring + xs * c.slot_stride + c.x_off + static_cast<int64_t>(xr) * Kp, g, rot);
  }
  const int32_t k0 = c.cell_step_ptr[cell], k1 = c.cell_step_ptr[cell + 1];
  // the sub-tile holds ts * Q4 = kTileFloats / 4 chunks of 16 bytes: NIT per thread, chunk
  // idx = it * kSweepBlock + threadIdx.x (row idx / Q4, column chunk idx % Q4)
  constexpr int NIT = kTileFloats / 4 / kSweepBlock;
  static_assert(NIT * kSweepBlock * 4 == kTileFloats, "whole chunks per thread");
  const int wave = static_cast<int>(threadIdx.x) >> 6;
  // the row numbers of this thread's chunks of step k (independent loads); they are loaded
  // one step ahead, during the previous step's sweep, and the step ids two steps ahead
  int32_t rr[NIT];
  auto load_rows = [&](int32_t step_id) {
    const int32_t *rows = c.step_rows + static_cast<int64_t>(step_id) * c.ts;
#pragma unroll
    for (int it = 0; it < NIT; ++it) rr[it] = rows[(it * kSweepBlock + static_cast<int>(threadIdx.x)) / Q4];
  };
  int32_t next_id = 0;
  if (k0 < k1) {
    load_rows(c.cell_steps[k0]);
    if (k0 + 1 < k1) next_id = c.cell_steps[k0 + 1];
  }
  for (int32_t k = k0; k < k1; ++k) {
    // the direct global-to-LDS loads back to back: a wavefront's load of iteration it
    // writes the 64 consecutive chunks it * kSweepBlock + 64 * wave + lane of the tile
    const float *base[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      base[it] = V + c.y_off;
      if (per_row && rr[it] >= 0)
        base[it] = c.ring + static_cast<int64_t>(c.rs_y[cls * c.rs_y_cls + rr[it]]) * c.slot_stride + c.y_off;
    }
    __syncthreads();  // the previous sub-tile is no longer read
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int idx = it * kSweepBlock + static_cast<int>(threadIdx.x);
      const float *src = (rr[it] >= 0 ? base[it] + static_cast<int64_t>(rr[it]) * Kp : c.zero) + 4 * (idx % Q4);
      lds_char *dst = (lds_char *)(tile) + 16 * (it * kSweepBlock + 64 * wave);  // generic -> LDS address space
      __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
    }
    const int32_t beg = c.run_beg[static_cast<int64_t>(k) * NG + grp];
    const int n = c.run_len[static_cast<int64_t>(k) * NG + grp];
    const uint16_t *__restrict__ li = c.ly + beg;
    const float *__restrict__ lv = c.lv + beg;
    // the first 8 (row, value) pairs are loaded before the barrier, then always the next 8
    // while the current 8 are swept
    u32x4 ni = {0u, 0u, 0u, 0u};
    f32x4 nv0 = {0.f, 0.f, 0.f, 0.f}, nv1 = {0.f, 0.f, 0.f, 0.f};
    if (n > 0) {
      ni = ld_once(reinterpret_cast<const u32x4 *>(li));
      nv0 = ld_once(reinterpret_cast<const f32x4 *>(lv));
      nv1 = ld_once(reinterpret_cast<const f32x4 *>(lv + 4));
    }
    __builtin_amdgcn_s_waitcnt(0);  // this thread's chunks have landed in LDS
    __syncthreads();
    if (k + 1 < k1) {  // the next step's row numbers, while this one is swept
      load_rows(next_id);
      if (k + 2 < k1) next_id = c.cell_steps[k + 2];
    }
    for (int t0 = 0; t0 < n; t0 += 8) {
      if constexpr (E >= 32) {  // 512-wide rows: no registers to spare for the prefetch
        if (t0 > 0) {
          ni = ld_once(reinterpret_cast<const u32x4 *>(li + t0));
          nv0 = ld_once(reinterpret_cast<const f32x4 *>(lv + t0));
          nv1 = ld_once(reinterpret_cast<const f32x4 *>(lv + t0 + 4));
        }
      }
      const u32x4 i8 = ni;  // 8 x uint16
      const f32x4 v0 = nv0, v1 = nv1;
      if (E < 32 && t0 + 8 < n) {
        ni = ld_once(reinterpret_cast<const u32x4 *>(li + t0 + 8));
        nv0 = ld_once(reinterpret_cast<const f32x4 *>(lv + t0 + 8));
        nv1 = ld_once(reinterpret_cast<const f32x4 *>(lv + t0 + 12));
      }
      const int idx[8] = {static_cast<int>(i8[0] & 0xffff), static_cast<int>(i8[0] >> 16),
                          static_cast<int>(i8[1] & 0xffff), static_cast<int>(i8[1] >> 16),
                          static_cast<int>(i8[2] & 0xffff), static_cast<int>(i8[2] >> 16),
                          static_cast<int>(i8[3] & 0xffff), static_cast<int>(i8[3] >> 16)};
      const float val[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
#pragma unroll
      for (int q = 0; q < 8; q += RF) {
        if (t0 + q >= n) break;
        float y[RF][E];
#pragma unroll
        for (int w = 0; w < RF; ++w) {
          // byte address of register chunk 0 (even chunks) and chunk 1 (odd chunks) of the row
          const uint32_t b0 = (static_cast<uint32_t>(idx[q + w]) * (Kp * 4u)) | lane_bytes;
          const uint32_t b1 = swizzled<G, E>() ? (b0 ^ (G * 16u)) : (b0 + G * 16u);
#pragma unroll
          for (int h = 0; h < E / 4; ++h) {
            const float4 tt = *reinterpret_cast<const float4 *>(tile_bytes + ((h & 1) ? b1 : b0) + (h & ~1) * G * 16);
            y[w][4 * h] = tt.x; y[w][4 * h + 1] = tt.y; y[w][4 * h + 2] = tt.z; y[w][4 * h + 3] = tt.w;
          }
        }
#pragma unroll
        for (int w = 0; w < RF; ++w) {
          // padding entries (row 0, value 0, past the run's n ratings) contribute nothing
          const float e_all = residual<G, E>(x, y[w], val[q + w]);
          const float err = (t0 + q + w < n) ? e_all : 0.f;
#pragma unroll
          for (int e = 0; e < E; ++e) acc[e] = fmaf(err, y[w][e], acc[e]);
        }
      }
    }
  }
  const int32_t out = c.cell_out[cell * NG + grp];
  if (out >= 0) store_row_once<G, E>(c.partial + static_cast<int64_t>(out) * Kp, acc, g, rot);
}

// The LDS-staged cells of both sweep directions in one launch (one 1024-thread workgroup
// per cell): workgroups [0, ncell_a) take set A, the rest set B.
struct CellSweepArgs {
  CellArgs ca, cb;
  int32_t ncell_a;
};

template <int G, int E>
__global__ __launch_bounds__(kSweepBlock) void k_cells(CellSweepArgs s) {
  __shared__ float4 tile[kTileFloats / 4];
  const int b = static_cast<int>(blockIdx.x);
  if (b < s.ncell_a) run_cell<G, E>(s.ca, b, tile);
  else run_cell<G, E>(s.cb, b - s.ncell_a, tile);
}

// The work units of both sweep directions in one launch: workgroups [0, grid_a) take set
// A, the rest set B (grid_a is a multiple of 8, so workgroup b of either set runs on XCD
// b mod 8).  The two directions only read the ring and write their own partial rows, so
// they may run concurrently, also with the cells.
struct UnitSweepArgs {
  UnitArgs ua, ub;
  int32_t grid_a;
};

template <int G, int E, bool PerRow>
__global__ __launch_bounds__(kBlock) void k_units(UnitSweepArgs s) {
  const int b = static_cast<int>(blockIdx.x);
  const bool first = b < s.grid_a;
  const UnitArgs &a = first ? s.ua : s.ub;
  const int64_t unit = unit_of(a, first ? b : b - s.grid_a, threadIdx.x / G, kBlock / G);
  if (unit < 0) return;  // whole groups leave together
  run_unit<G, E, PerRow>(a, unit, threadIdx.x & (G - 1));
}

// ------------------------------------------------------------------ dense (MFMA) cells
// A dense cell sweeps one 64-row x tile (users or items, one worker class) against a run
// of 64-row y tiles whose ratings are stored as dense 64 x 64 blocks (NaN = no rating).
// Wavefront w keeps x rows 16w .. 16w+15 in registers; per step the workgroup stages the
// 64 y rows in LDS and each wavefront, for every 16-row slice of them, computes with
// v_mfma_f32_16x16x4_f32
//   S^T = Y_s X_w^T                (16 y x 16 x, contraction over the rank),
//   E^T = D^T - S^T where rated, 0 elsewhere (the residuals, Section 3.1),
//   acc += E Y_s                   (16 x rows x Kp, contraction over the 16 y rows),
// so each rated (x, y) adds e_xy Y_y to acc_x exactly as the per-rating sweeps do.  The
// user-major pass also stores E in the item-major pass's fragment order, and the
// item-major pass (FromE) starts from those residuals: it skips GEMM 1 (a quarter of the
// dense products) and reads E where the user-major pass reads D.  Fragment
// layouts of the 16x16x4 fp32 MFMA (lane l, i = l % 16, g = l / 16): A operand A[i][g],
// B operand B[g][i], C/D holds D[4g + v][i] in register v.
//   GEMM 1: A[i][g] = Y[16 ys + i][k], B[g][i] = X[16 w + i][k] with the rank index
//           k = 16 q + 4 g + j for the j-th product of chunk q (any order of k sums the same);
//   GEMM 2: A[i][g] = E[16 w + i][16 ys + 4 g + r] is register r of S^T's fragment, B[g][i]
//           = Y[16 ys + 4 g + r][col(c, i)]; output block c holds the columns
//           col(c, i) = 16 C4 (c / C4) + C4 i + c % C4, so each lane reads and stores C4
//           consecutive floats (C4 = 4 from Kp = 64 on).
constexpr int kDenseThreads = 256;  // 4 wavefronts x 16 x rows
constexpr int kDenseRowsDev = psmf::kDenseRows;
static_assert(kDenseThreads / 64 * 16 == kDenseRowsDev, "one wavefront per 16 x rows");

struct DenseArgs {
  const int32_t *cell_x, *cell_cls, *cell_step_ptr, *step_rows, *cell_out;
  const float *dval;        // D (user-major) or the stored residuals E (item-major), fragment order
  float *eout;              // user-major: E in the item-major fragment order
  const int32_t *step_twin; // user-major: the item-major step of the same tile
  const float *zero;        // Kp zeros: the source of staged rows past the end of a ragged tile
  const int32_t *cls_slot;
  const float *ring;
  int64_t slot_stride, x_off, y_off;
  float *partial;
  const int32_t *rs_x, *rs_y;  // per-row policies (see UnitArgs)
  int64_t rs_x_cls, rs_y_cls;
};

// float4 chunk h of staged row y in LDS: chunks are XOR-swizzled by the row so that the
// 8 lanes of one ds_read_b128 pass (8 rows, same chunk; or one row, 8 chunks) hit
// different banks
template <int Kp>
__device__ __forceinline__ int dense_lds_chunk(int y, int h) {
  constexpr int H = Kp / 4;
  constexpr int SW = H < 16 ? H : 16;
  return y * H + (h ^ (y & (SW - 1)));
}

template <int C4>
struct VecOf;
template <>
struct VecOf<1> { typedef float T; };
template <>
struct VecOf<2> { typedef float2 T; };
template <>
struct VecOf<4> { typedef float4 T; };

template <int C4>
__device__ __forceinline__ float vec_at(const typename VecOf<C4>::T &v, int c) {
  if constexpr (C4 == 1) return v;
  else if constexpr (C4 == 2) return c == 0 ? v.x : v.y;
  else return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
}

// 4 x 4 transpose across the four lanes of a DPP quad: lane b of the quad holds row b in
// x[0..3] and returns column b (element r from lane r).  Two exchange stages: partners
// b ^ 1 swap the off-diagonal entries of each 2 x 2 block, then partners b ^ 2 swap the
// off-diagonal 2 x 2 blocks.  Every lane of the wavefront must be active.
__device__ __forceinline__ float dpp_quad_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, true));
}
__device__ __forceinline__ float dpp_quad_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, true));
}
__device__ __forceinline__ f32x4 quad_transpose(f32x4 x, int b) {
  const bool odd = (b & 1) != 0, hi = (b & 2) != 0;
  const float p0 = dpp_quad_xor1(odd ? x[0] : x[1]);
  const float p1 = dpp_quad_xor1(odd ? x[2] : x[3]);
  if (odd) { x[0] = p0; x[2] = p1; } else { x[1] = p0; x[3] = p1; }
  const float q0 = dpp_quad_xor2(hi ? x[0] : x[2]);
  const float q1 = dpp_quad_xor2(hi ? x[1] : x[3]);
  if (hi) { x[0] = q0; x[1] = q1; } else { x[2] = q0; x[3] = q1; }
  return x;
}

// Stage the 64 y rows of step k into an LDS buffer with direct global-to-LDS loads
// (global_load_lds_dwordx4): the loads of one wavefront write 64 consecutive 16-byte
// chunks starting at a wave-uniform LDS address, so lane l fetches the row chunk that the
// swizzle places at physical chunk p = 256 m + 64 w + l.  Rows -1 (past the end of a
// ragged tile) read a zero row.  Completion is waited for (vmcnt) before the barrier that
// hands the buffer to the readers.
// The staged row number of each of this thread's chunks of step k (independent loads).
template <int Kp>
__device__ __forceinline__ void dense_rows(const DenseArgs &a, int64_t k, int32_t (&r)[Kp / 16]) {
  constexpr int H = Kp / 4;
  const int32_t *rows = a.step_rows + k * kDenseRowsDev;
  const int lane = static_cast<int>(threadIdx.x) & 63, w = static_cast<int>(threadIdx.x) >> 6;
#pragma unroll
  for (int m = 0; m < Kp / 16; ++m) r[m] = rows[(kDenseThreads * m + 64 * w + lane) / H];
}

template <int Kp>
__device__ __forceinline__ void dense_stage(const DenseArgs &a, const float *__restrict__ Y, int cls,
                                            const int32_t (&r)[Kp / 16], float4 *lds_buf) {
  constexpr int H = Kp / 4;
  constexpr int SW = H < 16 ? H : 16;
  constexpr int NM = Kp / 16;
  const int lane = static_cast<int>(threadIdx.x) & 63, w = static_cast<int>(threadIdx.x) >> 6;
  // the loads into LDS back to back (the row numbers were loaded beforehand)
  const float *base[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    base[m] = Y;
    if (a.rs_y && r[m] >= 0) base[m] = a.ring + static_cast<int64_t>(a.rs_y[cls * a.rs_y_cls + r[m]]) * a.slot_stride + a.y_off;
  }
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    const int p = kDenseThreads * m + 64 * w + lane;
    const int y = p / H, h = (p % H) ^ (y & (SW - 1));
    const float *src = (r[m] >= 0 ? base[m] + static_cast<int64_t>(r[m]) * Kp : a.zero) + 4 * h;
    lds_char *dst = (lds_char *)(lds_buf) + 16 * (kDenseThreads * m + 64 * w);  // generic -> LDS address space
    __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
  }
}

// The two staging buffers are separate LDS variables and the step loop alternates them
// statically: the compiler then knows that the DMA into one buffer does not alias the
// reads of the other and does not wait for the DMA before those reads.
template <int Kp, bool FromE>
__device__ __forceinline__ void run_dense(const DenseArgs &a, int64_t cell, float4 *lds0, float4 *lds1) {
  constexpr int NQ = Kp / 16;             // rank chunks of 16 (GEMM 1) = output blocks of 16 columns (GEMM 2)
  constexpr int C4 = NQ < 4 ? NQ : 4;     // output blocks read / stored together
  constexpr int NB = 4 * (NQ / C4);       // GEMM 2 operand reads per 16-row slice
  typedef typename VecOf<C4>::T VecT;
  const int lane = static_cast<int>(threadIdx.x) & 63, w = static_cast<int>(threadIdx.x) >> 6;
  const int i = lane & 15, g = lane >> 4;
  const int cls = a.cell_cls[cell];  // one class per cell: uniform
  const int sv = a.rs_x ? 0 : a.cls_slot[cls];
  const float *__restrict__ V = a.ring + sv * a.slot_stride;
  const float *__restrict__ X = V + a.x_off;
  const float *__restrict__ Y = V + a.y_off;
  const int64_t k0 = a.cell_step_ptr[cell], k1 = a.cell_step_ptr[cell + 1];
  // row numbers of the next step to stage (loaded a step ahead of their staging)
  int32_t rnext[NQ];
  if (k0 < k1) {
    dense_rows<Kp>(a, k0, rnext);
    dense_stage<Kp>(a, Y, cls, rnext, lds0);
    if (k0 + 1 < k1) dense_rows<Kp>(a, k0 + 1, rnext);
  }
  // stationary rows in the B-operand layout of GEMM 1: xb[q] = X[16w + i][16q + 4g .. +3]
  f32x4 xb[NQ];
  if constexpr (!FromE) {
    const int32_t xr = a.cell_x[cell * kDenseRowsDev + 16 * w + i];
    const float *Xr = X;
    if (a.rs_x && xr >= 0) Xr = a.ring + static_cast<int64_t>(a.rs_x[cls * a.rs_x_cls + xr]) * a.slot_stride + a.x_off;
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      xb[q] = xr >= 0 ? ld_once(reinterpret_cast<const f32x4 *>(Xr + static_cast<int64_t>(xr) * Kp + 16 * q + 4 * g))
                      : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  f32x4 acc[NQ];
#pragma unroll
  for (int c = 0; c < NQ; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  const f32x4 *__restrict__ dv = reinterpret_cast<const f32x4 *>(a.dval);
  f32x4 dcur[4], dnext[4];
  if (k0 < k1) {
#pragma unroll
    for (int yb = 0; yb < 4; ++yb) dcur[yb] = ld_once(dv + (k0 * 16 + w * 4 + yb) * 64 + lane);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // one step: sweep the rows staged in T4 while the next step's rows go to `nextbuf`
  auto step = [&](int64_t k, const float4 *T4, float4 *nextbuf) {
    const bool more = k + 1 < k1;
    if (more) {  // the next step's rows (into the other buffer) and values
      dense_stage<Kp>(a, Y, cls, rnext, nextbuf);
      if (k + 2 < k1) dense_rows<Kp>(a, k + 2, rnext);
#pragma unroll
      for (int yb = 0; yb < 4; ++yb) dnext[yb] = ld_once(dv + ((k + 1) * 16 + w * 4 + yb) * 64 + lane);
    }
    const char *Tb = reinterpret_cast<const char *>(T4);
#pragma unroll
    for (int y2 = 0; y2 < 4; y2 += 2) {
      float e[2][4];
      if constexpr (FromE) {
        // the residuals of the user-major pass (0 where there is no rating)
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int v = 0; v < 4; ++v) e[h][v] = dcur[y2 + h][v];
      } else {
        // GEMM 1 for two 16-row slices at once (two independent accumulation chains); the
        // operands of chunk q+1 are read from LDS before the products of chunk q
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
        float4 a0n = T4[dense_lds_chunk<Kp>(16 * y2 + i, g)];
        float4 a1n = T4[dense_lds_chunk<Kp>(16 * y2 + 16 + i, g)];
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
          const float4 a0 = a0n, a1 = a1n;
          if (q + 1 < NQ) {
            a0n = T4[dense_lds_chunk<Kp>(16 * y2 + i, 4 * (q + 1) + g)];
            a1n = T4[dense_lds_chunk<Kp>(16 * y2 + 16 + i, 4 * (q + 1) + g)];
          }
          // keep the reads of chunk q+1 ahead of the products of chunk q (the scheduler
          // would otherwise sink them to their use and wait for them there)
          __builtin_amdgcn_sched_barrier(0);
          s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.x, xb[q][0], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.x, xb[q][0], s1, 0, 0, 0);
          s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.y, xb[q][1], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.y, xb[q][1], s1, 0, 0, 0);
          s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.z, xb[q][2], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.z, xb[q][2], s1, 0, 0, 0);
          s0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.w, xb[q][3], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.w, xb[q][3], s1, 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
        // residuals where rated (D is NaN elsewhere): the A operands of GEMM 2; stored for
        // the item-major pass at its fragment position of (x = item, y = user).  Lane
        // (i, g) holds E[item 16 ys + 4 g + v][user 16 w + i] in register v; after a 4 x 4
        // transpose inside each quad of lanes (i = 4 q + b) it holds E[item 16 ys + 4 g + b]
        // [user 16 w + 4 q + r] in register r, which is the float4 of lane 4 g + b + 16 q of
        // the item-major fragment block (ys, w): one contiguous 1 KiB store per wavefront
        f32x4 *eo = reinterpret_cast<f32x4 *>(a.eout + static_cast<int64_t>(a.step_twin[k]) * psmf::kDenseTile);
        const int elane = 4 * g + (i & 3) + 16 * (i >> 2);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const f32x4 sv4 = h ? s1 : s0;
          const f32x4 d = dcur[y2 + h];
          f32x4 et;
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            e[h][v] = d[v] == d[v] ? d[v] - sv4[v] : 0.f;
            et[v] = e[h][v];
          }
          st_once(eo + ((y2 + h) * 4 + w) * 64 + elane, quad_transpose(et, i & 3));
        }
      }
      // GEMM 2 over both slices; operand read t = (h, r, cg), the next one read first
      auto boff = [&](int t) {
        const int h = t / NB, r = (t % NB) / (NQ / C4), cg = t % (NQ / C4);
        const int f = 16 * C4 * cg + C4 * i;  // first float of this lane's columns
        return 16 * dense_lds_chunk<Kp>(16 * (y2 + h) + 4 * g + r, f >> 2) + 4 * (f & 3);
      };
      VecT bn = *reinterpret_cast<const VecT *>(Tb + boff(0));
#pragma unroll
      for (int t = 0; t < 2 * NB; ++t) {
        const VecT b = bn;
        if (t + 1 < 2 * NB) bn = *reinterpret_cast<const VecT *>(Tb + boff(t + 1));
        // keep each read ahead of the products before it (the scheduler would otherwise
        // sink it to its use and wait for it there)
        __builtin_amdgcn_sched_barrier(0);
        const int h = t / NB, r = (t % NB) / (NQ / C4), cg = t % (NQ / C4);
#pragma unroll
        for (int cc = 0; cc < C4; ++cc)
          acc[C4 * cg + cc] = __builtin_amdgcn_mfma_f32_16x16x4f32(e[h][r], vec_at<C4>(b, cc), acc[C4 * cg + cc], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    if (more) {
#pragma unroll
      for (int yb = 0; yb < 4; ++yb) dcur[yb] = dnext[yb];
    }
    __builtin_amdgcn_s_waitcnt(0);  // the staged rows of step k+1 have landed
    __syncthreads();
  };
  for (int64_t k = k0; k < k1; k += 2) {
    step(k, lds0, lds1);
    if (k + 1 < k1) step(k + 1, lds1, lds0);
  }
  // acc[c][v] = dX[16w + 4g + v][col(c, i)]
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    const int32_t out = a.cell_out[cell * kDenseRowsDev + 16 * w + 4 * g + v];
    if (out < 0) continue;
    float *dst = a.partial + static_cast<int64_t>(out) * Kp;
#pragma unroll
    for (int cg = 0; cg < NQ / C4; ++cg) {
      const int f = 16 * C4 * cg + C4 * i;
      if constexpr (C4 == 4) {
        st_once(reinterpret_cast<f32x4 *>(dst + f),
                f32x4{acc[4 * cg][v], acc[4 * cg + 1][v], acc[4 * cg + 2][v], acc[4 * cg + 3][v]});
      } else if constexpr (C4 == 2) {
        *reinterpret_cast<float2 *>(dst + f) = make_float2(acc[2 * cg][v], acc[2 * cg + 1][v]);
      } else {
        dst[f] = acc[cg][v];
      }
    }
  }
}

// The dense cells of both sweep directions in one launch: workgroups [0, ncell_a) take set
// A, the rest set B.
// One workgroup per dense cell of one direction: the user-major cells (residuals from D,
// stored as E), then, in a second launch, the item-major cells (FromE).  Up to Kp = 128 two
// workgroups share a CU (64 KiB of LDS each); at Kp = 256 the two staging buffers take
// 128 KiB, one workgroup fills a CU and its four wavefronts may use 512 registers each.
template <int Kp>
constexpr int dense_waves_per_simd() { return Kp <= 128 ? 2 : 1; }

template <int Kp, bool FromE>
__global__ __launch_bounds__(kDenseThreads, dense_waves_per_simd<Kp>()) void k_dense(DenseArgs a) {
  __shared__ float4 lds0[kDenseRowsDev * Kp / 4];
  __shared__ float4 lds1[kDenseRowsDev * Kp / 4];
  run_dense<Kp, FromE>(a, static_cast<int64_t>(blockIdx.x), lds0, lds1);
}

// Squared loss over the canonical CSR of a block at one ring slot: one lane group per
// segment (a user's ratings, cut at kLossSegment), e in fp32, e^2 accumulated in fp64,
// one partial per workgroup (fixed order, so the result is deterministic).
template <int G, int E>
__global__ __launch_bounds__(kBlock) void k_loss(const int32_t *__restrict__ seg_user,
                                                 const int64_t *__restrict__ seg_beg, int64_t nseg,
                                                 const int32_t *__restrict__ col, const float *__restrict__ val,
                                                 const float *__restrict__ L, const float *__restrict__ R,
                                                 double *__restrict__ out) {
  constexpr int Kp = G * E;
  constexpr int NG = kBlock / G;
  __shared__ double acc_sh[NG];
  const int g = threadIdx.x & (G - 1);
  const int grp = threadIdx.x / G;
  const int64_t sg = static_cast<int64_t>(blockIdx.x) * NG + grp;
  double acc = 0.0;
  if (sg < nseg) {
    float x[E];
    load_row<G, E>(x, L + static_cast<int64_t>(seg_user[sg]) * Kp, g);
    for (int64_t t = seg_beg[sg]; t < seg_beg[sg + 1]; ++t) {
      float y[E];
      load_row<G, E>(y, R + static_cast<int64_t>(col[t]) * Kp, g);
      const float e = residual<G, E>(x, y, val[t]);
      acc += static_cast<double>(e) * static_cast<double>(e);
    }
  }
  if (g == 0) acc_sh[grp] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int h = 0; h < NG; ++h) s += acc_sh[h];
    out[blockIdx.x] = s;
  }
}

// fixed-order final sum of the loss partials (deterministic for a given layout)
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

struct FinalArgs {
  float *ring;
  int64_t slot_stride;
  int64_t users;
  int32_t Kp;
  int32_t slot_c, slot_n;
  const int32_t *ucount;   // [users]
  const int32_t *ucls;     // [users]
  const int32_t *cls_slot; // [nclass]
  const float *partial;    // user-major partial rows
  const int64_t *user_pp;  // [users + 1]
  float eta, lambda;
  int32_t rowmean;
  const int32_t *rs_u;     // per-row policies: ring slot of each user row's view (null: class slot)
  const uint8_t *sole;     // users whose unit writes the new version (when its view slot is not slot_n)
};

// L^{c+1}_i = L^c_i + scale_i (sum of i's partial rows - n_i lambda L^v_i): the lambda term
// of each of the n_i ratings is hoisted; scale = eta (SUM) or eta / n_i (ROWMEAN).  Users
// without a rating in the block keep L^c_i (copied when the new slot differs).  One
// thread per 4 columns.
__device__ __forceinline__ void finalize_users(const FinalArgs &a, int64_t idx) {
  const int64_t q4 = a.Kp / 4;
  if (idx >= a.users * q4) return;
  const int64_t i = idx / q4;
  float4 *ring4 = reinterpret_cast<float4 *>(a.ring);
  const int64_t ss4 = a.slot_stride / 4;
  // what depends on i alone is loaded at once, so that the row's chain of dependent loads
  // is the view slot, then the partial rows and the view row
  const int n = a.ucount[i];
  const int32_t vs = a.rs_u ? a.rs_u[i] : a.ucls[i];  // the row's view slot, or its class
  const int64_t p0 = a.user_pp[i], p1 = a.user_pp[i + 1];
  const bool sole = a.sole && a.sole[i];
  const float4 lc = ring4[a.slot_c * ss4 + idx];
  if (n == 0) {
    if (a.slot_n != a.slot_c) ring4[a.slot_n * ss4 + idx] = lc;
    return;
  }
  const int32_t sv = a.rs_u ? vs : a.cls_slot[vs];
  if (sole && sv != a.slot_n) return;  // its unit wrote the new version
  const f32x4 *part4 = reinterpret_cast<const f32x4 *>(a.partial);
  const int64_t k4 = idx - i * q4;
  const float4 lv = ring4[sv * ss4 + idx];
  float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 4
  for (int64_t p = p0; p < p1; ++p) {
    const f32x4 t = ld_partial(part4 + p * q4 + k4);
    d.x += t[0]; d.y += t[1]; d.z += t[2]; d.w += t[3];
  }
  const float sc = a.rowmean ? a.eta / static_cast<float>(n) : a.eta;
  const float nl = static_cast<float>(n) * a.lambda;
  ring4[a.slot_n * ss4 + idx] = make_float4(commit_elem(lc.x, sc, d.x, nl, lv.x), commit_elem(lc.y, sc, d.y, nl, lv.y),
                                            commit_elem(lc.z, sc, d.z, nl, lv.z), commit_elem(lc.w, sc, d.w, nl, lv.w));
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
  const float *partial;       // item-major partial rows
  const int64_t *item_pp;     // [items + 1]
  float eta, lambda;
  int32_t rowmean;
  const int32_t *rs_i;        // per-row policies: [nclass * items] ring slot of each class's view of an item row
};

// R^{c+1}_j = R^c_j + scale_j (sum of j's partial rows - lambda sum_class n_j^(class) R^{v(class)}_j).
// One workgroup per item: thread t sums the float4 column t mod (Kp/4) of every
// (kBlock / (Kp/4))-th partial row, starting at row t / (Kp/4); the column sums are then
// added in row-lane order through LDS (popular items own thousands of partial rows).
__device__ __forceinline__ void commit_item(const CommitArgs &a, int64_t j, float4 *red) {
  const int q4 = a.Kp / 4;
  const int lanes = kBlock / q4;  // row lanes: Kp is a power of two in [8, 512], so 2..128
  const int k4 = static_cast<int>(threadIdx.x) % q4, lane = static_cast<int>(threadIdx.x) / q4;
  float4 *R4 = reinterpret_cast<float4 *>(a.ring + a.r_off);
  const int64_t ss4 = a.slot_stride / 4;
  const int64_t idx = j * q4 + k4;
  const int n = a.icount[j];
  const int64_t p0 = a.item_pp[j], p1 = a.item_pp[j + 1];
  float4 rc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (lane == 0) rc = R4[a.slot_c * ss4 + idx];  // loaded before the partial rows
  if (n == 0) {  // uniform over the workgroup
    if (lane == 0) R4[a.slot_n * ss4 + idx] = rc;
    return;
  }
  float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
  const f32x4 *part4 = reinterpret_cast<const f32x4 *>(a.partial);
#pragma unroll 4
  for (int64_t p = p0 + lane; p < p1; p += lanes) {
    const f32x4 t = ld_partial(part4 + p * q4 + k4);
    d.x += t[0]; d.y += t[1]; d.z += t[2]; d.w += t[3];
  }
  red[threadIdx.x] = d;
  __syncthreads();
  if (lane != 0) return;
  for (int l = 1; l < lanes; ++l) {
    const float4 t = red[l * q4 + k4];
    d.x += t.x; d.y += t.y; d.z += t.z; d.w += t.w;
  }
  // the classes' view rows, four classes' loads at a time (a class without a rating of the
  // item reads the current row instead and adds nothing), summed in class order
  float4 lam = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int q0 = 0; q0 < a.nclass; q0 += 4) {
    int cnt[4];
    float4 r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) cnt[u] = q0 + u < a.nclass ? a.icount_cls[j * a.nclass + q0 + u] : 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t slot = cnt[u] ? (a.rs_i ? a.rs_i[(q0 + u) * a.items + j] : a.cls_slot[q0 + u]) : a.slot_c;
      r[u] = R4[slot * ss4 + idx];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (cnt[u]) {
        const float c = static_cast<float>(cnt[u]);
        lam = make_float4(fmaf(c, r[u].x, lam.x), fmaf(c, r[u].y, lam.y), fmaf(c, r[u].z, lam.z),
                          fmaf(c, r[u].w, lam.w));
      }
    }
  }
  const float sc = a.rowmean ? a.eta / static_cast<float>(n) : a.eta;
  R4[a.slot_n * ss4 + idx] = make_float4(rc.x + sc * (d.x - a.lambda * lam.x), rc.y + sc * (d.y - a.lambda * lam.y),
                                         rc.z + sc * (d.z - a.lambda * lam.z), rc.w + sc * (d.w - a.lambda * lam.w));
}

// ------------------------------------------------------------------ per-row views
// Per-row policies (Section 4: each client caches rows; a row is served only while its
// version is >= c - s): one thread per cached row, the user rows (read by their owner's
// client when the user has a rating in the block) and the (client, item) rows (read when a
// worker of the client has a rating of the item in the block).  A row read at clock c
// takes the version the cache serves -- SSP_ROW: fetched at c when not cached or older
// than c - s, else kept; ESSP_ROW: fetched at c on the first read, then the push of
// version c - min(s, 1) -- and its slot in the ring.  Each read row adds its reads (one per
// rating) to the staleness profile at delay c - v.
constexpr int kMaxStaleBins = 1025;  // s <= 1024
struct RowViewArgs {
  int32_t *ver_u, *slot_u;          // [users]
  int32_t *ver_i, *slot_i;          // [nclass * items], client-major
  const int32_t *ucount;            // [users] ratings in the block
  const int32_t *icount_cls;        // [items * nclass] ratings in the block per client
  int64_t users, items, clock;
  int32_t nclass, s, essp;
  unsigned long long *stale;        // [s + 1]
};

__global__ __launch_bounds__(kBlock) void k_row_views(RowViewArgs a) {
  __shared__ unsigned long long hist[kMaxStaleBins];
  for (int t = static_cast<int>(threadIdx.x); t <= a.s; t += kBlock) hist[t] = 0ull;
  __syncthreads();
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx < a.users + static_cast<int64_t>(a.nclass) * a.items) {
    int32_t *ver, *slot;
    int64_t reads;
    if (idx < a.users) {
      ver = a.ver_u + idx;
      slot = a.slot_u + idx;
      reads = a.ucount[idx];
    } else {
      const int64_t x = idx - a.users, m = x / a.items, j = x - m * a.items;
      ver = a.ver_i + x;
      slot = a.slot_i + x;
      reads = a.icount_cls[j * a.nclass + m];
    }
    if (reads > 0) {
      const int64_t old = *ver, c = a.clock;
      int64_t v;
      if (a.essp) v = old < 0 ? c : c - (a.s < 1 ? a.s : 1);
      else v = (old < 0 || old < c - a.s) ? c : old;
      *ver = static_cast<int32_t>(v);
      *slot = static_cast<int32_t>(v % (a.s + 1));
      atomicAdd(&hist[c - v], static_cast<unsigned long long>(reads));
    }
  }
  __syncthreads();
  for (int t = static_cast<int>(threadIdx.x); t <= a.s; t += kBlock)
    if (hist[t]) atomicAdd(a.stale + t, hist[t]);
}

// Version c+1 of both factors in one launch: workgroups [0, grid_users) finalize L (one
// thread per 4 columns of a user), the rest commit R (one workgroup per item).  They write
// different rows of the new slot and read only partial rows and versions <= c.
__global__ __launch_bounds__(kBlock) void k_commit(FinalArgs fa, CommitArgs ca, int32_t grid_users) {
  __shared__ float4 red[kBlock];
  if (static_cast<int32_t>(blockIdx.x) < grid_users)
    finalize_users(fa, static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x);
  else
    commit_item(ca, static_cast<int64_t>(blockIdx.x) - grid_users, red);
}

// Debug check of the commit (PS_MF_OPT_POISON): before the commit of clock c, every row of
// the new version's slot that the commit will not read is set to NaN (but the user rows the
// work units wrote in the sweep), so that a row the commit fails to write stays NaN.  The
// commit reads the new slot (which held version c-s) where a view is version c-s: a user
// row with ratings whose view slot is the new slot, an item row with a rating by a worker
// class whose view slot is the new slot.  One thread per float4 of the slot.
__global__ __launch_bounds__(kBlock) void k_poison(FinalArgs fa, CommitArgs ca) {
  const int64_t q4 = fa.Kp / 4;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  if (idx >= (fa.users + ca.items) * q4) return;
  const int64_t row = idx / q4;
  bool read = false;
  if (row < fa.users) {
    const int64_t i = row;
    const int32_t sv = fa.rs_u ? fa.rs_u[i] : fa.cls_slot[fa.ucls[i]];
    read = fa.ucount[i] > 0 && sv == fa.slot_n;
    if (fa.sole && fa.ucount[i] > 0 && fa.sole[i] && sv != fa.slot_n) return;  // its unit wrote the new row
  } else {
    const int64_t j = row - fa.users;
    if (ca.icount[j] > 0)
      for (int q = 0; q < ca.nclass; ++q)
        if (ca.icount_cls[j * ca.nclass + q] > 0 &&
            (ca.rs_i ? ca.rs_i[q * ca.items + j] : ca.cls_slot[q]) == fa.slot_n)
          read = true;
  }
  if (!read) {
    const float nan = __int_as_float(0x7fc00000);
    reinterpret_cast<float4 *>(fa.ring)[fa.slot_n * (fa.slot_stride / 4) + idx] = make_float4(nan, nan, nan, nan);
  }
}

// ------------------------------------------------------------------ value-bounded views
// VAP (Section 3's condition on in-transit updates): at clock c every worker reads the
// stalest version v = c - d, d <= min(c, s), with |x_c - x_v|_inf <= v0 / sqrt(c + 1).
// k_vap_norms reduces, for d = 1 .. dmax, the max of the fp32 differences between the
// slots of versions c and c - d (padding columns are zero in every slot) into this
// clock's entry of the norm log (float bits, atomicMax over non-negative floats; NaN is
// ignored): one pass reads every slot once, with the dmax running maxima in registers
// (dmax <= kVapFused; beyond, one pass per d).  k_vap_pick then writes the slot the sweeps
// read and the version log entry.
constexpr int kVapFused = 16;
struct VapArgs {
  const float *ring;
  int64_t slot_stride;
  int64_t n4;          // float4s of one slot
  int64_t c;
  int32_t S1, dmax;
  unsigned *norms;     // [S1] this clock's norms
};

__device__ __forceinline__ float f4_absdiff_max(const float4 x, const float4 y) {
  return fmaxf(fmaxf(fabsf(x.x - y.x), fabsf(x.y - y.y)), fmaxf(fabsf(x.z - y.z), fabsf(x.w - y.w)));
}

// block max of m (every thread passes its value), added to *out by atomicMax
__device__ __forceinline__ void vap_block_max(float m, float *red, unsigned *out) {
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x / 64] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = red[0];
    for (int w = 1; w < kBlock / 64; ++w) t = fmaxf(t, red[w]);
    atomicMax(out, __float_as_uint(t));
  }
  __syncthreads();
}

__global__ __launch_bounds__(kBlock) void k_vap_norms(VapArgs a) {
  __shared__ float red[kBlock / 64];
  const float4 *r4 = reinterpret_cast<const float4 *>(a.ring);
  const int64_t ss4 = a.slot_stride / 4;
  const int32_t slot_c = static_cast<int32_t>(a.c % a.S1);
  if (a.dmax <= kVapFused) {
    float m[kVapFused];
    int32_t sd[kVapFused];
#pragma unroll
    for (int d = 0; d < kVapFused; ++d) {
      m[d] = 0.f;
      sd[d] = static_cast<int32_t>((a.c - d - 1 + (a.c < d + 1 ? a.S1 : 0)) % a.S1);  // used for d < dmax only
    }
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < a.n4;
         i += static_cast<int64_t>(gridDim.x) * kBlock) {
      const float4 x = r4[slot_c * ss4 + i];
#pragma unroll
      for (int d = 0; d < kVapFused; ++d)
        if (d < a.dmax) m[d] = fmaxf(m[d], f4_absdiff_max(x, r4[sd[d] * ss4 + i]));
    }
#pragma unroll
    for (int d = 0; d < kVapFused; ++d)
      if (d < a.dmax) vap_block_max(m[d], red, a.norms + d + 1);
    return;
  }
  for (int d = 1; d <= a.dmax; ++d) {
    const int32_t sd = static_cast<int32_t>((a.c - d) % a.S1);
    float m = 0.f;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < a.n4;
         i += static_cast<int64_t>(gridDim.x) * kBlock) {
      m = fmaxf(m, f4_absdiff_max(r4[slot_c * ss4 + i], r4[sd * ss4 + i]));
    }
    vap_block_max(m, red, a.norms + d);
  }
}

__global__ void k_vap_pick(const unsigned *norms, int32_t dmax, double bound, int64_t c, int32_t S1, int32_t *slot,
                           int64_t *vlog) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  int32_t d = 0;
  for (int32_t k = 1; k <= dmax; ++k)
    if (static_cast<double>(__uint_as_float(norms[k])) <= bound) d = k;
  slot[0] = static_cast<int32_t>((c - d) % S1);
  vlog[c] = c - d;
}

// ------------------------------------------------------------------ sequential step
// Under STEP_SEQ every worker applies the Section 3.1 rule rating by rating to its own
// copies of the rows.  A chain (one stratum: sub-epoch, worker, user group) is one
// wavefront; the chains of one sub-epoch share no row and run side by side in one launch,
// the sub-epochs one launch after another.  Lane l holds elements [l*E, (l+1)*E) of a row
// (E = Kp/64, at least 1), so the chain's control -- rating records, flags, branches -- is
// uniform over the wavefront, the records come through scalar loads, and a dot product is
// a 16-lane DPP sum plus the four row sums.  Inside a chain the current user's row stays in
// registers for the user's run and leaves it into the work copy; each rating updates its
// item row in the worker's copy (read from the view on the worker's first rating of the
// item in the clock).  Every rating depends on the rows the previous ones wrote, so the
// records are fetched 2*kSeqAhead ratings ahead and the item rows (and, at a run start, the
// user row) kSeqAhead ahead, in register rings whose slots are fixed at compile time.  A
// rating whose item occurs among the kSeqAhead ratings before it takes the row the latest
// of them wrote from a ring of the last kSeqAhead written rows (its prefetched copy may
// predate that store), so no rating waits on its own chain's stores.
typedef const __attribute__((address_space(4))) i32x4 *const_rec_ptr;  // read-only during the sweep
struct SeqArgs {
  const int64_t *chain_beg;
  const int32_t *chain_worker;
  const i32x4 *rec;                // [nnz] (user, item, value bits, flags) in application order
  const int32_t *wcls, *cls_slot;  // worker class, ring slot of each class's view
  const int32_t *rs_u, *rs_i;      // per-row policies: ring slot of each user row, of each
                                   // (class, item) row ([nclass * items], class-major)
  const float *ring;
  int64_t slot_stride, r_off, items;
  float *lwork;                    // [users, Kp] the user rows between their runs
  float *rwork;                    // [P, items, Kp] each worker's copy of the item rows
  int64_t rwork_stride;            // items * Kp
  int32_t Kp;
  float eta, lambda;
};

// a row of Kp = 64*E floats (Kp < 64: E = 1 and lanes >= Kp hold zeros)
template <int E>
__device__ __forceinline__ void wave_load_row(float (&d)[E], const float *__restrict__ row, int lane, int Kp) {
  if constexpr (E == 1) {
    d[0] = lane < Kp ? row[lane] : 0.f;
  } else if constexpr (E == 2) {
    const float2 t = *reinterpret_cast<const float2 *>(row + 2 * lane);
    d[0] = t.x; d[1] = t.y;
  } else {
#pragma unroll
    for (int q = 0; q < E / 4; ++q) {
      const float4 t = *reinterpret_cast<const float4 *>(row + E * lane + 4 * q);
      d[4 * q] = t.x; d[4 * q + 1] = t.y; d[4 * q + 2] = t.z; d[4 * q + 3] = t.w;
    }
  }
}

template <int E>
__device__ __forceinline__ void wave_store_row(float *__restrict__ row, const float (&d)[E], int lane, int Kp) {
  if constexpr (E == 1) {
    if (lane < Kp) row[lane] = d[0];
  } else if constexpr (E == 2) {
    *reinterpret_cast<float2 *>(row + 2 * lane) = make_float2(d[0], d[1]);
  } else {
#pragma unroll
    for (int q = 0; q < E / 4; ++q)
      *reinterpret_cast<float4 *>(row + E * lane + 4 * q) = make_float4(d[4 * q], d[4 * q + 1], d[4 * q + 2], d[4 * q + 3]);
  }
}

// sum over the 64 lanes: the 16-lane row sums, then the four rows through scalar registers
__device__ __forceinline__ float wave_sum(float v) {
  v = group_sum<16>(v);
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (r0 + r1) + (r2 + r3);
}

// f(integral_constant<int, K>, base + K) for K = K0 .. N-1 while f returns true
template <int K0, int N, class F>
__device__ __forceinline__ void seq_unrolled(F &f, int64_t base) {
  if (!f(std::integral_constant<int, K0>{}, base + K0)) return;
  if constexpr (K0 + 1 < N) seq_unrolled<K0 + 1, N>(f, base);
}

template <int E, bool PerRow>
__global__ __launch_bounds__(kBlock) void k_seq(SeqArgs a, int64_t c0, int64_t c1) {
  constexpr int D = psmf::kSeqAhead, D2 = 2 * psmf::kSeqAhead;
  const int lane = static_cast<int>(threadIdx.x) % 64, Kp = a.Kp;
  const int64_t ch = c0 + static_cast<int64_t>(blockIdx.x) * (kBlock / 64) +
                     __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x) / 64);
  if (ch >= c1) return;  // uniform over the wavefront
  const int64_t beg = a.chain_beg[ch], end = a.chain_beg[ch + 1];
  const int32_t p = a.chain_worker[ch];
  const int32_t cls = a.wcls[p];
  const float *Lv = a.ring + a.cls_slot[cls] * a.slot_stride;
  const float *Rv = Lv + a.r_off;
  float *Rw = a.rwork + static_cast<int64_t>(p) * a.rwork_stride;
  const const_rec_ptr rec = (const_rec_ptr)(a.rec);
  // the view of a row: the worker's whole view, or the row's own cached version
  auto view_L = [&](int32_t i) {
    return (PerRow ? a.ring + a.rs_u[i] * a.slot_stride : Lv) + static_cast<int64_t>(i) * Kp;
  };
  auto view_R = [&](int32_t j) {
    return (PerRow ? a.ring + a.rs_i[cls * a.items + j] * a.slot_stride + a.r_off : Rv) + static_cast<int64_t>(j) * Kp;
  };
  i32x4 meta[D2];
  float yq[D][E], lq[D][E], wq[D][E];
  auto fetch = [&](const i32x4 &m, float (&y)[E], float (&x)[E]) {
    wave_load_row<E>(y, (m[3] & psmf::kSeqFirstR) ? view_R(m[1]) : Rw + static_cast<int64_t>(m[1]) * Kp, lane, Kp);
    if (m[3] & psmf::kSeqRunStart)
      wave_load_row<E>(x, (m[3] & psmf::kSeqFirstL) ? view_L(m[0]) : a.lwork + static_cast<int64_t>(m[0]) * Kp,
                       lane, Kp);
  };
#pragma unroll
  for (int k = 0; k < D2; ++k)
    if (beg + k < end) meta[k] = rec[beg + k];
#pragma unroll
  for (int k = 0; k < D; ++k)
    if (beg + k < end) fetch(meta[k], yq[k], lq[k]);
  float x[E];
  int32_t cur = -1;
  // one rating; K is the ring position (a compile-time constant, so the rings stay in
  // registers); false once the chain is done
  auto step = [&](auto kc, int64_t n) -> bool {
    constexpr int K = decltype(kc)::value;
    if (n >= end) return false;
    const i32x4 m = meta[K];
    const int32_t flags = m[3];
    if (flags & psmf::kSeqRunStart) {
      if (cur >= 0) wave_store_row<E>(a.lwork + static_cast<int64_t>(cur) * Kp, x, lane, Kp);
#pragma unroll
      for (int e = 0; e < E; ++e) x[e] = lq[K % D][e];
      cur = m[0];
    }
    float y[E];
#pragma unroll
    for (int e = 0; e < E; ++e) y[e] = yq[K % D][e];
    const int dist = flags >> psmf::kSeqDistShift;
    if (dist) {  // the row rating n - dist wrote
#pragma unroll
      for (int q = 1; q <= D; ++q)
        if (dist == q) {
#pragma unroll
          for (int e = 0; e < E; ++e) y[e] = wq[(K - q + D2) % D][e];
        }
    }
    float dot = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) dot = fmaf(x[e], y[e], dot);
    const float err = __int_as_float(m[2]) - wave_sum(dot);
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float xl = x[e], yl = y[e];
      x[e] = fmaf(a.eta, fmaf(err, yl, -a.lambda * xl), xl);
      y[e] = fmaf(a.eta, fmaf(err, xl, -a.lambda * yl), yl);
    }
    wave_store_row<E>(Rw + static_cast<int64_t>(m[1]) * Kp, y, lane, Kp);
#pragma unroll
    for (int e = 0; e < E; ++e) wq[K % D][e] = y[e];
    if (n + D < end) fetch(meta[(K + D) % D2], yq[K % D], lq[K % D]);
    if (n + D2 < end) meta[K] = rec[n + D2];
    return true;
  };
  for (int64_t base = beg; base < end; base += D2) seq_unrolled<0, D2>(step, base);
  if (cur >= 0) wave_store_row<E>(a.lwork + static_cast<int64_t>(cur) * Kp, x, lane, Kp);
}

struct SeqCommitArgs {
  float *ring;
  int64_t slot_stride, r_off;
  int64_t users, items;
  int32_t Kp;
  int32_t slot_c, slot_n;
  const int32_t *ucount;       // [users] ratings in the block
  const int32_t *ucls;         // [users] class of the user's worker
  const int32_t *rs_u, *rs_i;  // per-row policies: the rows' own view slots (else null)
  const float *lwork;
  const int64_t *item_wptr;    // [items + 1]
  const int32_t *item_workers; // the workers with a rating of each item
  const int32_t *wcls, *cls_slot;
  const float *rwork;
  int64_t rwork_stride;
};

// One thread per float4 of a row: L^{c+1}_i = L^c_i + (copy - L^v_i) for the users with a
// rating in the block, the others keep L^c_i (copied when the new slot differs);
// R^{c+1}_j = R^c_j + sum over the workers with a rating of j of (copy - R^{v(p)}_j).
__global__ __launch_bounds__(kBlock) void k_seq_commit(SeqCommitArgs a) {
  const int64_t q4 = a.Kp / 4;
  int64_t idx = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  float4 *ring4 = reinterpret_cast<float4 *>(a.ring);
  const int64_t ss4 = a.slot_stride / 4;
  if (idx < a.users * q4) {
    const int64_t i = idx / q4;
    if (a.ucount[i] == 0) {
      if (a.slot_n != a.slot_c) ring4[a.slot_n * ss4 + idx] = ring4[a.slot_c * ss4 + idx];
      return;
    }
    const float4 loc = reinterpret_cast<const float4 *>(a.lwork)[idx];
    const float4 v = ring4[(a.rs_u ? a.rs_u[i] : a.cls_slot[a.ucls[i]]) * ss4 + idx];
    const float4 lc = ring4[a.slot_c * ss4 + idx];
    ring4[a.slot_n * ss4 + idx] = make_float4(lc.x + (loc.x - v.x), lc.y + (loc.y - v.y), lc.z + (loc.z - v.z),
                                              lc.w + (loc.w - v.w));
    return;
  }
  idx -= a.users * q4;
  if (idx >= a.items * q4) return;
  const int64_t j = idx / q4, r4 = a.r_off / 4 + idx;
  float4 d = make_float4(0.f, 0.f, 0.f, 0.f);
  const float4 *rw4 = reinterpret_cast<const float4 *>(a.rwork);
  for (int64_t q = a.item_wptr[j]; q < a.item_wptr[j + 1]; ++q) {
    const int32_t w = a.item_workers[q];
    const float4 loc = rw4[w * (a.rwork_stride / 4) + idx];
    const float4 v = ring4[(a.rs_i ? a.rs_i[a.wcls[w] * a.items + j] : a.cls_slot[a.wcls[w]]) * ss4 + r4];
    d.x += loc.x - v.x; d.y += loc.y - v.y; d.z += loc.z - v.z; d.w += loc.w - v.w;
  }
  const float4 rc = ring4[a.slot_c * ss4 + r4];
  ring4[a.slot_n * ss4 + r4] = make_float4(rc.x + d.x, rc.y + d.y, rc.z + d.z, rc.w + d.w);
}

// ------------------------------------------------------------------ kernel dispatch on Kp
// lane-group shape per padded rank: G lanes x E floats, G <= 16 so that a group sits in
// one DPP row, E a multiple of 4 for float4 access
struct Shape {
  int G, E;
};
Shape shape_for(int Kp) {
  switch (Kp) {
    case 8: return {2, 4};
    case 16: return {4, 4};
    case 32: return {8, 4};
    case 64: return {8, 8};
    case 128: return {8, 16};
    case 256: return {16, 16};
    default: return {16, 32};  // 512
  }
}
int padded_k(int K) {
  int Kp = 8;
  while (Kp < K) Kp *= 2;
  return Kp;
}

// lane-group shape of the work units: PS_MF_UNIT_WIDE = 1 spreads a row over 16 lanes
// (fewer registers and memory instructions per row, one more DPP step per dot product)
#ifndef PS_MF_UNIT_WIDE
#define PS_MF_UNIT_WIDE 0
#endif
Shape unit_shape_for(int Kp) {
  Shape sh = shape_for(Kp);
  if (PS_MF_UNIT_WIDE && sh.G < 16 && Kp / 16 >= 4) sh = {16, Kp / 16};
  return sh;
}

template <template <int, int> class F, class... Args>
hipError_t dispatch_units(int Kp, Args &&...args) {
  if (PS_MF_UNIT_WIDE) {
    switch (Kp) {
      case 64: return F<16, 4>::run(args...);
      case 128: return F<16, 8>::run(args...);
      default: break;
    }
  }
  switch (Kp) {
    case 8: return F<2, 4>::run(args...);
    case 16: return F<4, 4>::run(args...);
    case 32: return F<8, 4>::run(args...);
    case 64: return F<8, 8>::run(args...);
    case 128: return F<8, 16>::run(args...);
    case 256: return F<16, 16>::run(args...);
    default: return F<16, 32>::run(args...);
  }
}

template <template <int, int> class F, class... Args>
hipError_t dispatch(int Kp, Args &&...args) {
  switch (Kp) {
    case 8: return F<2, 4>::run(args...);
    case 16: return F<4, 4>::run(args...);
    case 32: return F<8, 4>::run(args...);
    case 64: return F<8, 8>::run(args...);
    case 128: return F<8, 16>::run(args...);
    case 256: return F<16, 16>::run(args...);
    default: return F<16, 32>::run(args...);
  }
}

template <int G, int E>
struct LaunchCells {
  static hipError_t run(const CellSweepArgs &a, int64_t grid, hipStream_t st) {
    hipLaunchKernelGGL((k_cells<G, E>), dim3(static_cast<unsigned>(grid)), dim3(kSweepBlock), 0, st, a);
    return hipGetLastError();
  }
};
template <int G, int E>
struct LaunchUnits {
  static hipError_t run(const UnitSweepArgs &a, int64_t grid, hipStream_t st) {
    if (a.ua.rs_x) hipLaunchKernelGGL((k_units<G, E, true>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, a);
    else hipLaunchKernelGGL((k_units<G, E, false>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, a);
    return hipGetLastError();
  }
};
// padded ranks with a dense (MFMA) cell kernel
bool dense_supported(int Kp) { return Kp >= 16 && Kp <= 256; }

template <int E>
hipError_t launch_seq(const SeqArgs &a, int64_t c0, int64_t c1, hipStream_t st) {
  const int64_t waves = kBlock / 64, grid = (c1 - c0 + waves - 1) / waves;
  if (a.rs_u) hipLaunchKernelGGL((k_seq<E, true>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, a, c0, c1);
  else hipLaunchKernelGGL((k_seq<E, false>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, a, c0, c1);
  return hipGetLastError();
}
// one chain per wavefront: E = Kp / 64 floats per lane (at least one)
hipError_t dispatch_seq(int Kp, const SeqArgs &a, int64_t c0, int64_t c1, hipStream_t st) {
  switch (Kp) {
    case 128: return launch_seq<2>(a, c0, c1, st);
    case 256: return launch_seq<4>(a, c0, c1, st);
    case 512: return launch_seq<8>(a, c0, c1, st);
    default: return launch_seq<1>(a, c0, c1, st);  // 8 .. 64
  }
}

template <bool FromE>
hipError_t launch_dense(int Kp, const DenseArgs &a, int64_t grid, hipStream_t st) {
  const dim3 gd(static_cast<unsigned>(grid)), bd(kDenseThreads);
  switch (Kp) {
    case 16: hipLaunchKernelGGL((k_dense<16, FromE>), gd, bd, 0, st, a); break;
    case 32: hipLaunchKernelGGL((k_dense<32, FromE>), gd, bd, 0, st, a); break;
    case 64: hipLaunchKernelGGL((k_dense<64, FromE>), gd, bd, 0, st, a); break;
    case 128: hipLaunchKernelGGL((k_dense<128, FromE>), gd, bd, 0, st, a); break;
    case 256: hipLaunchKernelGGL((k_dense<256, FromE>), gd, bd, 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int G, int E>
struct LaunchLoss {
  static hipError_t run(const int32_t *seg_user, const int64_t *seg_beg, int64_t nseg, const int32_t *col,
                        const float *val, const float *L, const float *R, int64_t grid, double *out, hipStream_t st) {
    hipLaunchKernelGGL((k_loss<G, E>), dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, st, seg_user, seg_beg,
                       nseg, col, val, L, R, out);
    return hipGetLastError();
  }
};

}  // namespace

// ------------------------------------------------------------------ handle
struct DeviceUnits {
  int64_t nunits = 0;  // units with ratings (the padding units come after them in the chunks)
  int64_t grid = 0;    // workgroups of a launch: kXcds x the largest chunk
  int32_t *y = nullptr;
  float *val = nullptr;
  int32_t *unit_x = nullptr, *unit_cls = nullptr, *unit_len = nullptr, *unit_out = nullptr;
  int64_t *unit_beg = nullptr, *xcd_off = nullptr, *x_pp = nullptr;
  uint8_t *sole = nullptr;  // user-major set: rows whose only partial row is one unit's
};

struct DeviceCells {
  int64_t ncells = 0, padded = 0;  // cells with work; launch slots (a multiple of 8)
  int32_t ts = 0;
  int32_t *step_rows = nullptr, *cell_x = nullptr, *cell_cls = nullptr, *cell_step_ptr = nullptr,
          *cell_steps = nullptr, *run_beg = nullptr, *run_len = nullptr, *cell_out = nullptr;
  uint16_t *ly = nullptr;
  float *lv = nullptr;
};

struct DeviceDense {
  int64_t ncells = 0;
  int32_t *cell_x = nullptr, *cell_cls = nullptr, *cell_step_ptr = nullptr, *step_rows = nullptr,
          *cell_out = nullptr, *step_twin = nullptr;
  float *dval = nullptr;
  float *eval = nullptr;  // item-major set: the residuals the user-major pass stores each clock
};

struct DeviceSeq {
  std::vector<int64_t> epoch_chain;  // host copy: the chains of each sub-epoch
  int64_t *chain_beg = nullptr, *item_wptr = nullptr;
  int32_t *chain_worker = nullptr, *item_workers = nullptr;
  int32_t *rec = nullptr;            // [nnz * 4] (user, item, value bits, flags)
};

struct DeviceBlock {
  int64_t nnz = 0, loss_grid = 0;
  int32_t *ucount = nullptr, *icount = nullptr, *icount_cls = nullptr;
  int64_t nseg = 0;            // the canonical CSR cut into loss segments
  int32_t *seg_user = nullptr;
  int64_t *seg_beg = nullptr;  // [nseg + 1]
  int32_t *col = nullptr;
  float *val = nullptr;
  DeviceUnits by_user, by_item;
  DeviceCells cells_user, cells_item;
  DeviceDense dense_user, dense_item;
  DeviceSeq seq;
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
  int64_t tile_bytes = 6 << 20;  // rows per L2 tile of the item-major sweep, in bytes
  int64_t item_tile_bytes = -1;  // rows per L2 tile of the user-major sweep (-1: 4 x tile_bytes)
  bool poison = false;           // debug: NaN in the rows of the new slot the commit does not read
  int32_t unit_max = 256;
  bool cells = true;             // stage the dense part (heavy users) through LDS
  int64_t heavy_min = -1;        // ratings from which a user goes to the cells (-1: automatic)
  int32_t dense_min = -1;        // ratings from which a 64 x 64 tile goes to the MFMA cells (-1: automatic, 0: none)
  int32_t seq_groups = 256;      // sub-epochs of the sequential step
  double v0 = INFINITY;          // value bound of the VAP policy
  bool eta_decay = false;        // step eta / sqrt(c + 1) at clock c
  bool seq_graphs = true;        // replay each clock's sub-epoch launches from a captured HIP graph
  std::vector<hipGraphExec_t> seq_exec;  // per (block, slot-table row)
  bool sweep_graphs = false;     // replay each clock's sweep launches from a captured HIP graph
  bool unit_commit = true;       // a user's only unit writes its new version (see UnitArgs::sole)
  std::vector<hipGraphExec_t> sweep_exec;  // per (block, slot-table row)
  std::vector<int32_t> owner;
  // host state
  bool loaded = false, has_factors = false;
  int64_t clock = 0;
  std::vector<int64_t> vlog;
  std::vector<int64_t> worker_ratings;  // [B * P]: ratings of each worker in each block
  std::vector<psmf::BlockLayout> layout;
  int32_t nclass = 1;
  std::vector<int32_t> cls_of_worker;
  std::string err;
  // device state
  int device = -1;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  hipStream_t user_stream = nullptr;
  hipStream_t side_stream = nullptr;  // runs the work units beside the cells (default priority)
  hipEvent_t fork = nullptr, join = nullptr;
  hipStream_t cell_stream = nullptr;  // runs the LDS cells beside the dense tiles (three streams)
  hipEvent_t join_cells = nullptr;
  bool two_streams = true;
  int32_t hot_steps = -1;  // LDS sub-tiles of hot items whose light-user ratings go to cells (-1: auto)
  float *ring = nullptr;
  float *partial_u = nullptr, *partial_i = nullptr;
  float *zero_row = nullptr;  // Kp zeros (staging source of empty dense rows)
  // per-row policies: cached version and ring slot of every user row and (client, item)
  // row, and the staleness profile of the clocks run
  int32_t *ver_u = nullptr, *slot_u = nullptr, *ver_i = nullptr, *slot_i = nullptr;
  unsigned long long *stale = nullptr;
  int32_t *ucls = nullptr;
  int32_t *slot_table = nullptr;  // [(2s+1) * nclass]
  int32_t *wcls = nullptr;        // [P] class of each worker
  float *lwork = nullptr, *rwork = nullptr;  // sequential step: user rows between runs, workers' item rows
  // VAP: the slot of the current clock's view, the version read and the norms of every clock
  int32_t *vap_slot = nullptr;
  int64_t *vap_v = nullptr;
  unsigned *vap_norms = nullptr;
  int64_t vap_cap = 0;
  double *loss_partial = nullptr;
  int64_t loss_partial_len = 0;
  int64_t loss_parts = 0;  // partial sums one loss takes (all blocks)
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

#define HIP_TRY(h, expr)                                                                                  \
  do {                                                                                                   \
    hipError_t e_ = (expr);                                                                              \
    if (e_ != hipSuccess) {                                                                              \
      if (e_ == hipErrorOutOfMemory) return fail(h, PS_MF_ENOMEM, "%s: %s", #expr, hipGetErrorString(e_)); \
      return fail(h, PS_MF_EDEVICE, "%s: %s", #expr, hipGetErrorString(e_));                             \
    }                                                                                                    \
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

int upload_units(ps_mf_t *h, DeviceUnits &d, const psmf::UnitSet &u) {
  int r;
  if ((r = upload(h, &d.y, u.y)) || (r = upload(h, &d.val, u.val)) || (r = upload(h, &d.unit_x, u.unit_x)) ||
      (r = upload(h, &d.unit_cls, u.unit_cls)) || (r = upload(h, &d.unit_len, u.unit_len)) ||
      (r = upload(h, &d.unit_out, u.unit_out)) || (r = upload(h, &d.unit_beg, u.unit_beg)) ||
      (r = upload(h, &d.xcd_off, u.xcd_off)) || (r = upload(h, &d.x_pp, u.x_pp)))
    return r;
  d.nunits = u.nreal;
  int64_t most = 0;
  for (int x = 0; x < kXcds; ++x) most = std::max<int64_t>(most, u.xcd_off[x + 1] - u.xcd_off[x]);
  const int groups = kBlock / unit_shape_for(h->Kp).G;
  d.grid = kXcds * ((most + groups - 1) / groups);
  return PS_MF_OK;
}

int upload_cells(ps_mf_t *h, DeviceCells &d, const psmf::CellSet &c) {
  int r;
  if ((r = upload(h, &d.step_rows, c.step_rows)) || (r = upload(h, &d.cell_x, c.cell_x)) ||
      (r = upload(h, &d.cell_cls, c.cell_cls)) || (r = upload(h, &d.cell_step_ptr, c.cell_step_ptr)) ||
      (r = upload(h, &d.cell_steps, c.cell_steps)) || (r = upload(h, &d.run_beg, c.run_beg)) ||
      (r = upload(h, &d.run_len, c.run_len)) || (r = upload(h, &d.cell_out, c.cell_out)) ||
      (r = upload(h, &d.ly, c.ly)) || (r = upload(h, &d.lv, c.lv)))
    return r;
  d.ncells = static_cast<int64_t>(c.cell_cls.size());
  d.padded = (d.ncells + kXcds - 1) / kXcds * kXcds;
  d.ts = c.ts;
  return PS_MF_OK;
}

// the user-major set keeps D and the map to the item-major steps; the item-major set
// keeps a residual buffer of its steps instead of its own copy of D
int upload_dense(ps_mf_t *h, DeviceDense &d, const psmf::DenseSet &D, bool user_major) {
  int r;
  if ((r = upload(h, &d.cell_x, D.cell_x)) || (r = upload(h, &d.cell_cls, D.cell_cls)) ||
      (r = upload(h, &d.cell_step_ptr, D.cell_step_ptr)) || (r = upload(h, &d.step_rows, D.step_rows)) ||
      (r = upload(h, &d.cell_out, D.cell_out)))
    return r;
  if (user_major) {
    if ((r = upload(h, &d.dval, D.dval)) || (r = upload(h, &d.step_twin, D.step_twin))) return r;
  } else {
    if ((r = dev_alloc(h, reinterpret_cast<void **>(&d.eval), D.dval.size() * sizeof(float)))) return r;
  }
  d.ncells = static_cast<int64_t>(D.cell_cls.size());
  return PS_MF_OK;
}

DenseArgs dense_args(const ps_mf_t *h, const DeviceDense &d, float *partial, int64_t x_off, int64_t y_off,
                     const int32_t *cls_slot, const DeviceDense &twin) {
  DenseArgs a{};
  a.cell_x = d.cell_x;
  a.cell_cls = d.cell_cls;
  a.cell_step_ptr = d.cell_step_ptr;
  a.step_rows = d.step_rows;
  a.cell_out = d.cell_out;
  a.dval = d.dval ? d.dval : d.eval;
  a.eout = twin.eval;
  a.step_twin = d.step_twin;
  a.zero = h->zero_row;
  a.cls_slot = cls_slot;
  a.ring = h->ring;
  a.slot_stride = (h->N + h->M) * h->Kp;
  a.x_off = x_off;
  a.y_off = y_off;
  a.partial = partial;
  return a;
}

CellArgs cell_args(const ps_mf_t *h, const DeviceCells &d, float *partial, int64_t x_off, int64_t y_off,
                   const int32_t *cls_slot) {
  CellArgs a{};
  a.step_rows = d.step_rows;
  a.cell_x = d.cell_x;
  a.cell_cls = d.cell_cls;
  a.cell_step_ptr = d.cell_step_ptr;
  a.cell_steps = d.cell_steps;
  a.run_beg = d.run_beg;
  a.run_len = d.run_len;
  a.cell_out = d.cell_out;
  a.ly = d.ly;
  a.lv = d.lv;
  a.cls_slot = cls_slot;
  a.ring = h->ring;
  a.slot_stride = (h->N + h->M) * h->Kp;
  a.x_off = x_off;
  a.y_off = y_off;
  a.ts = d.ts;
  a.partial = partial;
  a.zero = h->zero_row;
  return a;
}

UnitArgs unit_args(const ps_mf_t *h, const DeviceUnits &d, float *partial, int64_t x_off, int64_t y_off,
                   int64_t y_rows) {
  UnitArgs a{};
  a.unit_x = d.unit_x;
  a.unit_cls = d.unit_cls;
  a.unit_len = d.unit_len;
  a.unit_out = d.unit_out;
  a.unit_beg = d.unit_beg;
  a.xcd_off = d.xcd_off;
  a.y = d.y;
  a.val = d.val;
  a.ring = h->ring;
  a.slot_stride = (h->N + h->M) * h->Kp;
  a.x_off = x_off;
  a.y_off = y_off;
  a.y_bytes = y_rows * h->Kp * 4;
  a.partial = partial;
  return a;
}

bool per_row_policy(const ps_mf_t *h) { return h->policy == PS_MF_SSP_ROW || h->policy == PS_MF_ESSP_ROW; }

// per-row slot tables of one sweep direction: the user-major direction keeps users (one
// entry each) and gathers items (one entry per client and item); item-major the reverse
template <class A>
void set_row_slots(const ps_mf_t *h, A &a, bool user_major) {
  if (!per_row_policy(h)) {
    a.rs_x = a.rs_y = nullptr;
    a.rs_x_cls = a.rs_y_cls = 0;
    return;
  }
  a.rs_x = user_major ? h->slot_u : h->slot_i;
  a.rs_y = user_major ? h->slot_i : h->slot_u;
  a.rs_x_cls = user_major ? 0 : h->M;
  a.rs_y_cls = user_major ? h->M : 0;
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
  {
    const hipError_t e = hipSetDevice(h->device);
    if (e != hipSuccess) {
      (void)hipGetLastError();  // not sticky: leave no error for the caller's next HIP call
      return fail(h, PS_MF_EDEVICE, "hipSetDevice(%d): %s", h->device, hipGetErrorString(e));
    }
  }
  if (!h->stream) {
    if (h->user_stream) {
      h->stream = h->user_stream;
    } else {
      HIP_TRY(h, hipStreamCreateWithFlags(&h->stream, hipStreamNonBlocking));
      h->own_stream = true;
    }
  }
  if (h->two_streams && !h->side_stream) {
    HIP_TRY(h, hipStreamCreateWithFlags(&h->side_stream, hipStreamNonBlocking));
    HIP_TRY(h, hipEventCreateWithFlags(&h->fork, hipEventDisableTiming));
    HIP_TRY(h, hipEventCreateWithFlags(&h->join, hipEventDisableTiming));
  }
  if (h->two_streams && PS_MF_CELL_STREAM && !h->cell_stream) {
    HIP_TRY(h, hipStreamCreateWithFlags(&h->cell_stream, hipStreamNonBlocking));
    HIP_TRY(h, hipEventCreateWithFlags(&h->join_cells, hipEventDisableTiming));
  }
  return PS_MF_OK;
}

int host_threads() {
  unsigned n = std::thread::hardware_concurrency();
  if (n == 0) n = 1;
  return static_cast<int>(std::min(16u, n));
}

int record(ps_mf_t *h, hipEvent_t *a) {
  *a = nullptr;
  if (!h->timing) return PS_MF_OK;
  HIP_TRY(h, hipEventCreate(a));
  HIP_TRY(h, hipEventRecord(*a, h->stream));
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

// per-row policies: the version and ring slot each cached row is read at in clock c
int row_views(ps_mf_t *h, const DeviceBlock &db, int64_t c) {
  RowViewArgs rv{};
  rv.ver_u = h->ver_u;
  rv.slot_u = h->slot_u;
  rv.ver_i = h->ver_i;
  rv.slot_i = h->slot_i;
  rv.ucount = db.ucount;
  rv.icount_cls = db.icount_cls;
  rv.users = h->N;
  rv.items = h->M;
  rv.clock = c;
  rv.nclass = h->nclass;
  rv.s = h->s;
  rv.essp = h->policy == PS_MF_ESSP_ROW;
  rv.stale = h->stale;
  const int64_t rows = h->N + static_cast<int64_t>(h->nclass) * h->M;
  hipLaunchKernelGGL(k_row_views, dim3(static_cast<unsigned>((rows + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                     h->stream, rv);
  HIP_TRY(h, hipGetLastError());
  return PS_MF_OK;
}

float eta_at(const ps_mf_t *h, int64_t c) {
  return h->eta_decay ? static_cast<float>(static_cast<double>(h->eta) / std::sqrt(static_cast<double>(c + 1)))
                      : h->eta;
}

// room in the VAP logs for clock c (the logs double; old buffers stay allocated until the
// handle is destroyed)
int vap_reserve(ps_mf_t *h, int64_t c) {
  if (c < h->vap_cap) return PS_MF_OK;
  int64_t cap = std::max<int64_t>(1024, 2 * h->vap_cap);
  while (cap <= c) cap *= 2;
  const size_t S1 = static_cast<size_t>(h->s) + 1;
  int64_t *v = nullptr;
  unsigned *nr = nullptr;
  int r;
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&v), static_cast<size_t>(cap) * sizeof(int64_t))) ||
      (r = dev_alloc(h, reinterpret_cast<void **>(&nr), static_cast<size_t>(cap) * S1 * sizeof(unsigned))))
    return r;
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  HIP_TRY(h, hipMemset(nr, 0, static_cast<size_t>(cap) * S1 * sizeof(unsigned)));
  if (h->vap_cap > 0) {
    HIP_TRY(h, hipMemcpy(v, h->vap_v, static_cast<size_t>(h->vap_cap) * sizeof(int64_t), hipMemcpyDeviceToDevice));
    HIP_TRY(h, hipMemcpy(nr, h->vap_norms, static_cast<size_t>(h->vap_cap) * S1 * sizeof(unsigned),
                         hipMemcpyDeviceToDevice));
  }
  h->vap_v = v;
  h->vap_norms = nr;
  h->vap_cap = cap;
  return PS_MF_OK;
}

// The ring slot each worker class reads at clock c: the slot table's row, or under VAP the
// slot that k_vap_pick writes (after the norm reduction, on the handle's stream).
int clock_views(ps_mf_t *h, int64_t c, const int32_t **cls_slot) {
  if (h->policy != PS_MF_VAP) {
    *cls_slot = h->slot_table + table_row(h, c) * h->nclass;
    return PS_MF_OK;
  }
  int r = vap_reserve(h, c);
  if (r) return r;
  const int32_t S1 = h->s + 1, dmax = static_cast<int32_t>(std::min<int64_t>(c, h->s));
  unsigned *norms = h->vap_norms + c * S1;
  if (dmax > 0) {
    VapArgs a{};
    a.ring = h->ring;
    a.slot_stride = (h->N + h->M) * h->Kp;
    a.n4 = a.slot_stride / 4;
    a.c = c;
    a.S1 = S1;
    a.dmax = dmax;
    a.norms = norms;
    const int64_t grid = std::max<int64_t>(1, std::min<int64_t>(2048, (a.n4 + kBlock - 1) / kBlock));
    hipLaunchKernelGGL(k_vap_norms, dim3(static_cast<unsigned>(grid)), dim3(kBlock), 0, h->stream, a);
    HIP_TRY(h, hipGetLastError());
  }
  const double bound = h->v0 / std::sqrt(static_cast<double>(c + 1));
  hipLaunchKernelGGL(k_vap_pick, dim3(1), dim3(64), 0, h->stream, norms, dmax, bound, c, S1, h->vap_slot, h->vap_v);
  HIP_TRY(h, hipGetLastError());
  *cls_slot = h->vap_slot;
  return PS_MF_OK;
}

// the version log under VAP lives on the device: rebuild the host copy (P entries a clock)
int vap_sync_log(ps_mf_t *h) {
  if (h->policy != PS_MF_VAP) return PS_MF_OK;
  h->vlog.clear();
  if (h->clock == 0 || !h->vap_v) return PS_MF_OK;
  std::vector<int64_t> v(static_cast<size_t>(h->clock));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  HIP_TRY(h, hipMemcpy(v.data(), h->vap_v, v.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
  for (int64_t c = 0; c < h->clock; ++c)
    for (int64_t p = 0; p < h->P; ++p) h->vlog.push_back(v[c]);
  return PS_MF_OK;
}

// One clock of the sequential step: the sub-epochs one launch after another, then the
// commit of R and of the untouched user rows.
int seq_clock(ps_mf_t *h) {
  const int64_t c = h->clock;
  const int b = static_cast<int>(c % h->B);
  const int32_t S1 = h->s + 1;
  const DeviceBlock &db = h->dblocks[b];
  const DeviceSeq &q = db.seq;
  SeqArgs a{};
  a.chain_beg = q.chain_beg;
  a.chain_worker = q.chain_worker;
  a.rec = reinterpret_cast<const i32x4 *>(q.rec);
  a.wcls = h->wcls;
  int rc = clock_views(h, c, &a.cls_slot);
  if (rc) return rc;
  if (per_row_policy(h)) {
    if ((rc = row_views(h, db, c))) return rc;
    a.rs_u = h->slot_u;
    a.rs_i = h->slot_i;
  }
  a.items = h->M;
  a.ring = h->ring;
  a.slot_stride = (h->N + h->M) * h->Kp;
  a.r_off = h->N * h->Kp;
  a.lwork = h->lwork;
  a.rwork = h->rwork;
  a.rwork_stride = h->M * h->Kp;
  a.Kp = h->Kp;
  a.eta = eta_at(h, c);
  a.lambda = h->lambda;
  hipEvent_t ev = nullptr;
  if ((rc = record(h, &ev))) return rc;
  auto launch_epochs = [&]() -> hipError_t {
    for (int32_t t = 0; t < h->seq_groups; ++t) {
      const int64_t c0 = q.epoch_chain[t], c1 = q.epoch_chain[t + 1];
      if (c1 > c0) {
        const hipError_t e = dispatch_seq(h->Kp, a, c0, c1, h->stream);
        if (e != hipSuccess) return e;
      }
    }
    return hipSuccess;
  };
  // The launches of a clock depend on the block and the slot-table row only (VAP: the block;
  // a per-clock step schedule: never the same), so each combination is captured once into a
  // HIP graph and replayed: one submission instead of up to G.
  const int64_t rows = 2 * static_cast<int64_t>(h->s) + 1;
  const int64_t key = h->policy == PS_MF_VAP ? b : b * rows + table_row(h, c);
  if (h->seq_graphs && !h->eta_decay) {
    if (h->seq_exec.empty()) h->seq_exec.assign(static_cast<size_t>(h->B * rows), nullptr);
    hipGraphExec_t &ex = h->seq_exec[static_cast<size_t>(key)];
    if (!ex) {
      // a stream the caller is capturing already (the launches then go into the caller's
      // graph), or one that cannot start a capture, gets the launches one by one
      hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
      if (hipStreamIsCapturing(h->stream, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone ||
          hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
        (void)hipGetLastError();
        h->seq_graphs = false;
      } else {
        hipGraph_t graph = nullptr;
        const hipError_t le = launch_epochs();
        const hipError_t ce = hipStreamEndCapture(h->stream, &graph);
        hipError_t ie = hipSuccess;
        if (le == hipSuccess && ce == hipSuccess) ie = hipGraphInstantiate(&ex, graph, nullptr, nullptr, 0);
        if (graph) (void)hipGraphDestroy(graph);
        HIP_TRY(h, le);
        HIP_TRY(h, ce);
        HIP_TRY(h, ie);
      }
    }
  }
  if (h->seq_graphs && !h->eta_decay) {
    HIP_TRY(h, hipGraphLaunch(h->seq_exec[static_cast<size_t>(key)], h->stream));
  } else {
    HIP_TRY(h, launch_epochs());
  }
  if ((rc = record_end(h, PS_MF_KERNEL_SWEEP, ev))) return rc;
  if ((rc = record(h, &ev))) return rc;
  SeqCommitArgs ca{};
  ca.ring = h->ring;
  ca.slot_stride = a.slot_stride;
  ca.r_off = a.r_off;
  ca.users = h->N;
  ca.items = h->M;
  ca.Kp = h->Kp;
  ca.slot_c = static_cast<int32_t>(c % S1);
  ca.slot_n = static_cast<int32_t>((c + 1) % S1);
  ca.ucount = db.ucount;
  ca.ucls = h->ucls;
  ca.rs_u = a.rs_u;
  ca.rs_i = a.rs_i;
  ca.lwork = h->lwork;
  ca.item_wptr = q.item_wptr;
  ca.item_workers = q.item_workers;
  ca.wcls = h->wcls;
  ca.cls_slot = a.cls_slot;
  ca.rwork = h->rwork;
  ca.rwork_stride = a.rwork_stride;
  const int64_t threads = (h->N + h->M) * (h->Kp / 4);
  hipLaunchKernelGGL(k_seq_commit, dim3(static_cast<unsigned>((threads + kBlock - 1) / kBlock)), dim3(kBlock), 0,
                     h->stream, ca);
  HIP_TRY(h, hipGetLastError());
  if ((rc = record_end(h, PS_MF_KERNEL_COMMIT, ev))) return rc;
  if (h->policy != PS_MF_VAP && !per_row_policy(h))
    for (int64_t p = 0; p < h->P; ++p) h->vlog.push_back(view_version(h, p, c));
  h->clock = c + 1;
  return PS_MF_OK;
}

int one_clock(ps_mf_t *h) {
  if (h->step == PS_MF_STEP_SEQ) return seq_clock(h);
  const int64_t c = h->clock;
  const int b = static_cast<int>(c % h->B);
  const int32_t S1 = h->s + 1;
  const int32_t slot_c = static_cast<int32_t>(c % S1), slot_n = static_cast<int32_t>((c + 1) % S1);
  const DeviceBlock &db = h->dblocks[b];
  const int32_t *cls_slot = nullptr;
  int rc = clock_views(h, c, &cls_slot);
  if (rc) return rc;
  const int64_t slot_stride = (h->N + h->M) * h->Kp;
  const int64_t r_off = h->N * h->Kp;
  const int rowmean = h->step == PS_MF_STEP_ROWMEAN;

  // the commit's arguments (the sweep's work units take the direct-write part of them)
  FinalArgs fa{};
  fa.ring = h->ring;
  fa.slot_stride = slot_stride;
  fa.users = h->N;
  fa.Kp = h->Kp;
  fa.slot_c = slot_c;
  fa.slot_n = slot_n;
  fa.ucount = db.ucount;
  fa.ucls = h->ucls;
  fa.cls_slot = cls_slot;
  fa.partial = h->partial_u;
  fa.user_pp = db.by_user.x_pp;
  fa.eta = eta_at(h, c);
  fa.lambda = h->lambda;
  fa.rowmean = rowmean;
  fa.rs_u = per_row_policy(h) ? h->slot_u : nullptr;
  // (not inside a captured sweep graph: its launches would replay this clock's slots and eta)
  fa.sole = h->unit_commit && !h->sweep_graphs ? db.by_user.sole : nullptr;
  const int64_t nfin = h->N * h->Kp / 4;
  CommitArgs ca{};
  ca.ring = h->ring;
  ca.slot_stride = slot_stride;
  ca.r_off = r_off;
  ca.items = h->M;
  ca.Kp = h->Kp;
  ca.slot_c = slot_c;
  ca.slot_n = slot_n;
  ca.icount = db.icount;
  ca.icount_cls = db.icount_cls;
  ca.nclass = h->nclass;
  ca.cls_slot = cls_slot;
  ca.partial = h->partial_i;
  ca.item_pp = db.by_item.x_pp;
  ca.eta = eta_at(h, c);
  ca.lambda = h->lambda;
  ca.rowmean = rowmean;
  ca.rs_i = per_row_policy(h) ? h->slot_i : nullptr;
  const int64_t grid_users = (nfin + kBlock - 1) / kBlock, grid_items = h->M;
  hipEvent_t ev = nullptr;
  if ((rc = record(h, &ev))) return rc;
  if (per_row_policy(h) && (rc = row_views(h, db, c))) return rc;
  {
    // set A = user-major (x = user / L, y = item / R); set B = item-major (x = item, y = user)
    CellSweepArgs cs{};
    cs.ca = cell_args(h, db.cells_user, h->partial_u, 0, r_off, cls_slot);
    cs.cb = cell_args(h, db.cells_item, h->partial_i, r_off, 0, cls_slot);
    cs.ncell_a = static_cast<int32_t>(db.cells_user.ncells);
    set_row_slots(h, cs.ca, true);
    set_row_slots(h, cs.cb, false);
    const int64_t ncells = db.cells_user.ncells + db.cells_item.ncells;
    UnitSweepArgs us{};
    us.ua = unit_args(h, db.by_user, h->partial_u, 0, r_off, h->M);
    us.ub = unit_args(h, db.by_item, h->partial_i, r_off, 0, h->N);
    us.ua.cls_slot = cls_slot;
    us.ub.cls_slot = cls_slot;
    if (fa.sole) {
      us.ua.sole = fa.sole;
      us.ua.xcount = db.ucount;
      us.ua.slot_c = slot_c;
      us.ua.slot_n = slot_n;
      us.ua.base_rows = h->ring + slot_c * slot_stride;
      us.ua.new_rows = h->ring + slot_n * slot_stride;
      us.ua.eta = fa.eta;
      us.ua.lambda = fa.lambda;
      us.ua.rowmean = fa.rowmean;
    }
    set_row_slots(h, us.ua, true);
    set_row_slots(h, us.ub, false);
    const int64_t gu = db.by_user.nunits > 0 ? db.by_user.grid : 0;
    const int64_t gi = db.by_item.nunits > 0 ? db.by_item.grid : 0;
    us.grid_a = static_cast<int32_t>(gu);
    // dense cells: the user-major pass stores the residuals that the item-major pass reads,
    // so the two run one after the other on the handle's stream
    DenseArgs du = dense_args(h, db.dense_user, h->partial_u, 0, r_off, cls_slot, db.dense_item);
    DenseArgs di = dense_args(h, db.dense_item, h->partial_i, r_off, 0, cls_slot, db.dense_user);
    set_row_slots(h, du, true);
    set_row_slots(h, di, false);
    const int64_t ndense = db.dense_user.ncells + db.dense_item.ncells;
    auto launch_dense_pair = [&]() -> hipError_t {
      hipError_t e = hipSuccess;
      if (db.dense_user.ncells > 0 && (e = launch_dense<false>(h->Kp, du, db.dense_user.ncells, h->stream))) return e;
      if (db.dense_item.ncells > 0) e = launch_dense<true>(h->Kp, di, db.dense_item.ncells, h->stream);
      return e;
    };
    // the launches of the sweep; every error is returned (a capture in progress must end)
    auto launch_sweep = [&]() -> hipError_t {
      hipError_t e = hipSuccess;
      if (ncells + ndense > 0 && gu + gi > 0 && h->side_stream) {
        // dense cells (and cells) on the handle's stream, units on the side stream (cells on
        // a third stream when there is one), all after what precedes
        const bool third = h->cell_stream && ncells > 0 && ndense > 0;
        if ((e = hipEventRecord(h->fork, h->stream)) || (e = hipStreamWaitEvent(h->side_stream, h->fork, 0))) return e;
        if (third && (e = hipStreamWaitEvent(h->cell_stream, h->fork, 0))) return e;
        if ((e = dispatch_units<LaunchUnits>(h->Kp, us, gu + gi, h->side_stream))) return e;
        if (third && (e = dispatch<LaunchCells>(h->Kp, cs, ncells, h->cell_stream))) return e;
        if (ndense > 0 && (e = launch_dense_pair())) return e;
        if (!third && ncells > 0 && (e = dispatch<LaunchCells>(h->Kp, cs, ncells, h->stream))) return e;
        if ((e = hipEventRecord(h->join, h->side_stream)) || (e = hipStreamWaitEvent(h->stream, h->join, 0))) return e;
        if (third && ((e = hipEventRecord(h->join_cells, h->cell_stream)) ||
                      (e = hipStreamWaitEvent(h->stream, h->join_cells, 0))))
          return e;
      } else {
        if (ndense > 0 && (e = launch_dense_pair())) return e;
        if (ncells > 0 && (e = dispatch<LaunchCells>(h->Kp, cs, ncells, h->stream))) return e;
        if (gu + gi > 0 && (e = dispatch_units<LaunchUnits>(h->Kp, us, gu + gi, h->stream))) return e;
      }
      return e;
    };
    // The sweep's launches depend on the block and the slot-table row only (per-row and
    // value-bounded views: on the block; their slots are read from device tables), so each
    // combination is captured once into a HIP graph and replayed: one submission per clock.
    const int64_t rows = 2 * static_cast<int64_t>(h->s) + 1;
    const bool device_slots = per_row_policy(h) || h->policy == PS_MF_VAP;
    const int64_t key = device_slots ? b : b * rows + table_row(h, c);
    const bool graphed = h->sweep_graphs && (ncells + ndense + gu + gi > 0);
    if (graphed) {
      if (h->sweep_exec.empty()) h->sweep_exec.assign(static_cast<size_t>(h->B * rows), nullptr);
      hipGraphExec_t &ex = h->sweep_exec[static_cast<size_t>(key)];
      if (!ex) {
        // a stream the caller is capturing already (the launches then go into the caller's
        // graph), or one that cannot start a capture, gets the launches one by one
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(h->stream, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone ||
            hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
          (void)hipGetLastError();
          h->sweep_graphs = false;
        } else {
          hipGraph_t graph = nullptr;
          const hipError_t le = launch_sweep();
          const hipError_t ce = hipStreamEndCapture(h->stream, &graph);
          hipError_t ie = hipSuccess;
          if (le == hipSuccess && ce == hipSuccess) ie = hipGraphInstantiate(&ex, graph, nullptr, nullptr, 0);
          if (graph) (void)hipGraphDestroy(graph);
          HIP_TRY(h, le);
          HIP_TRY(h, ce);
          HIP_TRY(h, ie);
        }
      }
    }
    if (graphed && h->sweep_graphs) {
      HIP_TRY(h, hipGraphLaunch(h->sweep_exec[static_cast<size_t>(key)], h->stream));
    } else {
      HIP_TRY(h, launch_sweep());
    }
  }
  if ((rc = record_end(h, PS_MF_KERNEL_SWEEP, ev))) return rc;

  if ((rc = record(h, &ev))) return rc;
  if (h->poison && slot_n != slot_c) {
    const int64_t n4 = (h->N + h->M) * (h->Kp / 4);
    hipLaunchKernelGGL(k_poison, dim3(static_cast<unsigned>((n4 + kBlock - 1) / kBlock)), dim3(kBlock), 0, h->stream,
                       fa, ca);
    HIP_TRY(h, hipGetLastError());
  }
  hipLaunchKernelGGL(k_commit, dim3(static_cast<unsigned>(grid_users + grid_items)), dim3(kBlock), 0, h->stream, fa,
                     ca, static_cast<int32_t>(grid_users));
  HIP_TRY(h, hipGetLastError());
  if ((rc = record_end(h, PS_MF_KERNEL_COMMIT, ev))) return rc;

  if (!per_row_policy(h) && h->policy != PS_MF_VAP)
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
  // the sweeps address one factor table with 32-bit byte offsets
  if (users * padded_k(K) * 4 >= (int64_t(1) << 32) || items * padded_k(K) * 4 >= (int64_t(1) << 32))
    return PS_MF_EINVAL;
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
      if (value < PS_MF_SSP_LAZY || value > PS_MF_VAP) return fail(h, PS_MF_EINVAL, "unknown policy %lld", (long long)value);
      h->policy = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_STEP:
      if (value != PS_MF_STEP_ROWMEAN && value != PS_MF_STEP_SUM && value != PS_MF_STEP_SEQ)
        return fail(h, PS_MF_EINVAL, "unknown step %lld", (long long)value);
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
    case PS_MF_OPT_TILE_BYTES:
      if (value < 1) return fail(h, PS_MF_EINVAL, "tile bytes must be >= 1");
      h->tile_bytes = value;
      return PS_MF_OK;
    case PS_MF_OPT_UNIT_MAX:
      if (value < 1 || value > (1 << 30)) return fail(h, PS_MF_EINVAL, "unit size must be in [1, 2^30]");
      h->unit_max = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_CELLS:
      h->cells = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_TWO_STREAMS:
      h->two_streams = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_HOT_STEPS:
      if (value < -1 || value > 1024) return fail(h, PS_MF_EINVAL, "hot item sub-tiles must be in [-1, 1024]");
      h->hot_steps = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_HEAVY_MIN:
      if (value < -1) return fail(h, PS_MF_EINVAL, "heavy threshold must be >= -1");
      h->heavy_min = value;
      return PS_MF_OK;
    case PS_MF_OPT_DENSE_MIN:
      if (value < -1 || value > psmf::kDenseTile)
        return fail(h, PS_MF_EINVAL, "dense tile threshold must be in [-1, %d]", psmf::kDenseTile);
      h->dense_min = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_SEQ_STRATA:
      if (value < 1 || value > 4096) return fail(h, PS_MF_EINVAL, "sub-epochs must be in [1, 4096]");
      h->seq_groups = static_cast<int32_t>(value);
      return PS_MF_OK;
    case PS_MF_OPT_ETA_DECAY:
      h->eta_decay = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_SEQ_GRAPHS:
      h->seq_graphs = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_ITEM_TILE_BYTES:
      if (value < 1 && value != -1) return fail(h, PS_MF_EINVAL, "item tile bytes must be >= 1 or -1");
      h->item_tile_bytes = value;
      return PS_MF_OK;
    case PS_MF_OPT_DEVICE:
      if (value < -1 || value > 4095) return fail(h, PS_MF_EINVAL, "device ordinal must be in [-1, 4095]");
      if (h->stream) return fail(h, PS_MF_ESTATE, "the device is already in use");
      h->device = static_cast<int>(value);
      return PS_MF_OK;
    case PS_MF_OPT_POISON:
      h->poison = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_SWEEP_GRAPHS:
      h->sweep_graphs = value != 0;
      return PS_MF_OK;
    case PS_MF_OPT_UNIT_COMMIT:
      h->unit_commit = value != 0;
      return PS_MF_OK;
    default:
      return fail(h, PS_MF_EINVAL, "unknown option key %d", key);
  }
}

int ps_mf_set_value_bound(ps_mf_t *h, double v0) {
  if (!h) return PS_MF_EINVAL;
  if (h->loaded) return fail(h, PS_MF_ESTATE, "the value bound must be set before ps_mf_load_ratings");
  if (!(v0 >= 0)) return fail(h, PS_MF_EINVAL, "the value bound must be >= 0 (infinity allowed)");
  h->v0 = v0;
  return PS_MF_OK;
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

}  // extern "C"

namespace {
int load_ratings(ps_mf_t *h, const int32_t *user, const int32_t *item, const float *value, int64_t n);
}

extern "C" {

int ps_mf_load_ratings(ps_mf_t *h, const int32_t *user, const int32_t *item, const float *value, int64_t n) {
  if (!h) return PS_MF_EINVAL;
  try {
    return load_ratings(h, user, item, value, n);
  } catch (const std::bad_alloc &) {
    return fail(h, PS_MF_ENOMEM, "host memory for the layout of %lld ratings", (long long)n);
  }
}

}  // extern "C"

namespace {
int load_ratings(ps_mf_t *h, const int32_t *user, const int32_t *item, const float *value, int64_t n) {
  if (h->loaded) return fail(h, PS_MF_ESTATE, "ratings are already loaded");
  if (n < 0 || (n > 0 && (!user || !item || !value))) return fail(h, PS_MF_EINVAL, "bad rating arrays");
  if (h->poison && h->step == PS_MF_STEP_SEQ)
    return fail(h, PS_MF_EINVAL, "the poison check covers the fixed-view commit only, not PS_MF_STEP_SEQ");
  if (n > 0x7fffffffLL) return fail(h, PS_MF_EINVAL, "at most 2^31-1 ratings");
  const bool seq = h->step == PS_MF_STEP_SEQ;
  if (h->owner.empty()) {
    h->owner.resize(static_cast<size_t>(h->N));
    for (int64_t i = 0; i < h->N; ++i) h->owner[i] = static_cast<int32_t>(i % h->P);
  }
  // worker classes: workers that read the same version at every clock
  // (the per-row policies' clients are these classes: worker p on client p mod (s+1))
  const bool staggered = h->policy == PS_MF_SSP_LAZY || per_row_policy(h);
  h->nclass = staggered ? std::min<int32_t>(h->s + 1, h->P) : 1;
  h->cls_of_worker.resize(static_cast<size_t>(h->P));
  for (int32_t p = 0; p < h->P; ++p) h->cls_of_worker[p] = staggered ? p % (h->s + 1) : 0;

  psmf::LayoutParams lp;
  lp.users = h->N;
  lp.items = h->M;
  lp.B = h->B;
  lp.seed = h->seed;
  lp.nclass = h->nclass;
  lp.owner = h->owner.data();
  lp.cls_of_worker = h->cls_of_worker.data();
  lp.threads = host_threads();
  // item-major tiles of user rows are sized for one XCD's L2; the user-major sweep takes
  // 4x larger item tiles: fewer units and partial rows per light user measured faster
  lp.tile_rows_user = std::max<int64_t>(64, h->tile_bytes / (static_cast<int64_t>(h->Kp) * 4));
  lp.tile_rows_item = h->item_tile_bytes > 0
                          ? std::max<int64_t>(64, h->item_tile_bytes / (static_cast<int64_t>(h->Kp) * 4))
                          : 4 * lp.tile_rows_user;
  lp.unit_max = h->unit_max;
  // The automatic split sends ratings to dense tiles and LDS cells only when the minibatch
  // blocks are large: both pay fixed costs (a partial row per cell row, workgroups that
  // each sweep a few steps) that a small block does not amortize.  Measured on the
  // 10M-rating K = 64 workload in 4 blocks: units alone 0.196 ms per clock against 0.220 ms
  // with the split; on the 100M-rating K = 128 workload the split saves a quarter.
  const bool split_auto = n / h->B >= kSplitMinRatings;
  if (h->cells) {
    // cells: one 1024-thread workgroup per cell, a 160 KiB LDS sub-tile of ts rows; a user
    // is dense enough for them when it averages 16 or more ratings per item sub-tile
    lp.cell_rows = kTileFloats / h->Kp;
    lp.cell_groups = kSweepBlock / shape_for(h->Kp).G;
    lp.heavy_min = h->heavy_min >= 0 ? h->heavy_min
                   : split_auto      ? std::max<int64_t>(256, 16 * h->M / lp.cell_rows)
                                     : lp.heavy_min;  // no user is heavy
  }
  if (h->dense_min > 0 && !dense_supported(h->Kp))
    return fail(h, PS_MF_EINVAL, "dense tiles need a padded rank in [16, 256], not %d", h->Kp);
  lp.dense_min = h->dense_min >= 0 ? h->dense_min : (split_auto && dense_supported(h->Kp) ? kDenseAuto : 0);
  lp.dense_target = PS_MF_DENSE_CELLS;
  lp.workers = h->P;
  if (seq) {
    lp.seq_groups = h->seq_groups;
    lp.dense_min = 0;
    lp.cell_rows = lp.cell_groups = 0;
  }
  if (h->cells) {
    // automatic hot-item sub-tiles: none next to dense tiles, else one (on the 100M-rating
    // K = 128 workload: 1 measured best among 0..4 without dense tiles; with them the
    // light users' extra partial rows cost the commit more than the cells save)
    lp.hot_steps = h->hot_steps >= 0 ? h->hot_steps : (lp.dense_min > 0 || !split_auto ? 0 : 1);
  }
  std::string err;
  const int rc = psmf::build_layout(lp, user, item, value, n, h->layout, err);
  if (rc == -1) return fail(h, PS_MF_EINVAL, "%s", err.c_str());
  if (rc) return fail(h, PS_MF_ENOMEM, "%s", err.c_str());
  h->worker_ratings.assign(static_cast<size_t>(h->B) * h->P, 0);
  for (int b = 0; b < h->B; ++b)
    for (int64_t i = 0; i < h->N; ++i)
      h->worker_ratings[static_cast<size_t>(b) * h->P + h->owner[i]] += h->layout[b].ucount[i];
  // partial sums of the loss: one per workgroup of lane groups, a lane group per loss
  // segment (a user's ratings of a block, cut every kLossSegment)
  h->loss_parts = 0;
  for (int b = 0; b < h->B; ++b) {
    int64_t nseg = 0;
    for (int64_t i = 0; i < h->N; ++i) nseg += (h->layout[b].ucount[i] + kLossSegment - 1) / kLossSegment;
    const int64_t groups = kBlock / shape_for(h->Kp).G;
    h->loss_parts += (nseg + groups - 1) / groups;
  }
  if (h->host_only) {
    for (int b = 0; b < h->B; ++b)
      if (psmf::check_layout(lp, h->layout[b], err))
        return fail(h, PS_MF_EINTERNAL, "layout self-check of block %d: %s", b, err.c_str());
    h->loaded = true;
    return PS_MF_OK;
  }
  h->loaded = true;

  int r = ensure_device(h);
  if (r) { h->loaded = false; return r; }
  const size_t slot = static_cast<size_t>((h->N + h->M) * h->Kp);
  auto undo = [h](int code) { h->loaded = false; return code; };
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->ring), slot * (h->s + 1) * sizeof(float)))) return undo(r);
  h->dblocks.assign(static_cast<size_t>(h->B), DeviceBlock());
  int64_t max_units_u = 1, max_units_i = 1, loss_len = 0;
  for (int b = 0; b < h->B; ++b) {
    const psmf::BlockLayout &L = h->layout[b];
    DeviceBlock &d = h->dblocks[b];
    d.nnz = L.nnz;
    if ((r = upload(h, &d.ucount, L.ucount)) || (r = upload(h, &d.icount, L.icount)) ||
        (r = upload(h, &d.icount_cls, L.icount_cls)) || (r = upload(h, &d.col, L.col)) ||
        (r = upload(h, &d.val, L.val)))
      return undo(r);
    if (seq) {
      const psmf::SeqSet &S = L.seq;
      DeviceSeq &q = d.seq;
      q.epoch_chain = S.epoch_chain;
      std::vector<int32_t> rec(S.user.size() * 4);
      for (size_t x = 0; x < S.user.size(); ++x) {
        rec[4 * x] = S.user[x];
        rec[4 * x + 1] = S.item[x];
        std::memcpy(&rec[4 * x + 2], &S.val[x], sizeof(float));
        rec[4 * x + 3] = S.flag[x];
      }
      if ((r = upload(h, &q.chain_beg, S.chain_beg)) || (r = upload(h, &q.chain_worker, S.chain_worker)) ||
          (r = upload(h, &q.rec, rec)) || (r = upload(h, &q.item_wptr, S.item_wptr)) ||
          (r = upload(h, &q.item_workers, S.item_workers)))
        return undo(r);
    } else if ((r = upload_units(h, d.by_user, L.by_user)) || (r = upload_units(h, d.by_item, L.by_item)) ||
               (r = upload(h, &d.by_user.sole, L.by_user.sole)) ||
               (r = upload_cells(h, d.cells_user, L.cells_user)) || (r = upload_cells(h, d.cells_item, L.cells_item)) ||
               (r = upload_dense(h, d.dense_user, L.dense_user, true)) ||
               (r = upload_dense(h, d.dense_item, L.dense_item, false))) {
      return undo(r);
    }
    // partial rows of units and cells, + the row the padding units write
    max_units_u = std::max<int64_t>(max_units_u, L.partial_rows_user + 1);
    max_units_i = std::max<int64_t>(max_units_i, L.partial_rows_item + 1);
    {
      std::vector<int32_t> su;
      std::vector<int64_t> sb;
      for (int64_t i = 0; i < h->N; ++i)
        for (int64_t t = L.row_ptr[i]; t < L.row_ptr[i + 1]; t += kLossSegment) {
          su.push_back(static_cast<int32_t>(i));
          sb.push_back(t);
        }
      sb.push_back(L.nnz);
      d.nseg = static_cast<int64_t>(su.size());
      if ((r = upload(h, &d.seg_user, su)) || (r = upload(h, &d.seg_beg, sb))) return undo(r);
    }
    d.loss_grid = (d.nseg + kBlock / shape_for(h->Kp).G - 1) / (kBlock / shape_for(h->Kp).G);
    loss_len += d.loss_grid;
  }
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->partial_u), static_cast<size_t>(max_units_u * h->Kp) * sizeof(float))) ||
      (r = dev_alloc(h, reinterpret_cast<void **>(&h->partial_i), static_cast<size_t>(max_units_i * h->Kp) * sizeof(float))))
    return undo(r);
  // user class (for the finalize of L), loss partials (one per workgroup of each block)
  std::vector<int32_t> ucls(static_cast<size_t>(h->N));
  for (int64_t i = 0; i < h->N; ++i) ucls[i] = h->cls_of_worker[h->owner[i]];
  if ((r = upload(h, &h->ucls, ucls))) return undo(r);
  if (loss_len != h->loss_parts) return undo(fail(h, PS_MF_EINTERNAL, "loss partials %lld, expected %lld",
                                                  (long long)loss_len, (long long)h->loss_parts));
  h->loss_partial_len = std::max<int64_t>(1, loss_len);
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->loss_partial), static_cast<size_t>(h->loss_partial_len) * sizeof(double))))
    return undo(r);
  if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->loss_out), sizeof(double)))) return undo(r);
  if ((r = upload(h, &h->zero_row, std::vector<float>(static_cast<size_t>(h->Kp), 0.f)))) return undo(r);
  if (per_row_policy(h)) {
    const size_t ni = static_cast<size_t>(h->nclass) * static_cast<size_t>(h->M);
    if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->ver_u), h->N * sizeof(int32_t))) ||
        (r = dev_alloc(h, reinterpret_cast<void **>(&h->slot_u), h->N * sizeof(int32_t))) ||
        (r = dev_alloc(h, reinterpret_cast<void **>(&h->ver_i), ni * sizeof(int32_t))) ||
        (r = dev_alloc(h, reinterpret_cast<void **>(&h->slot_i), ni * sizeof(int32_t))) ||
        (r = dev_alloc(h, reinterpret_cast<void **>(&h->stale), (h->s + 1) * sizeof(unsigned long long))))
      return undo(r);
  }
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
  if ((r = upload(h, &h->wcls, h->cls_of_worker))) return undo(r);
  if (h->policy == PS_MF_VAP &&
      ((r = upload(h, &h->vap_slot, std::vector<int32_t>(1, 0))) || (r = vap_reserve(h, 0))))
    return undo(r);
  if (seq) {
    // the users' rows between their runs and every worker's copy of the item rows
    const size_t rw = static_cast<size_t>(h->P) * static_cast<size_t>(h->M) * static_cast<size_t>(h->Kp);
    if ((r = dev_alloc(h, reinterpret_cast<void **>(&h->lwork), static_cast<size_t>(h->N * h->Kp) * sizeof(float))) ||
        (r = dev_alloc(h, reinterpret_cast<void **>(&h->rwork), rw * sizeof(float))))
      return undo(r);
  }
  return PS_MF_OK;
}

// Squared loss of the latest version: one k_loss launch per block writes its workgroups'
// fp64 partials into partial[], k_sum_partials adds them in a fixed order into *result
// (device memory), and the host waits for the value.  Allocates nothing.
int loss_into(ps_mf_t *h, double *partial, double *result, double *out) {
  const int64_t slot_stride = (h->N + h->M) * h->Kp;
  const int32_t sl = static_cast<int32_t>(h->clock % (h->s + 1));
  const float *L = h->ring + sl * slot_stride;
  const float *R = L + h->N * h->Kp;
  int64_t off = 0;
  for (int b = 0; b < h->B; ++b) {
    const DeviceBlock &d = h->dblocks[b];
    if (d.nnz == 0) continue;
    HIP_TRY(h, dispatch<LaunchLoss>(h->Kp, d.seg_user, d.seg_beg, d.nseg, d.col, d.val, L, R, d.loss_grid,
                                     partial + off, h->stream));
    off += d.loss_grid;
  }
  if (off == 0) {
    *out = 0.0;
    return PS_MF_OK;
  }
  hipLaunchKernelGGL(k_sum_partials, dim3(1), dim3(kBlock), 0, h->stream, partial, off, result);
  HIP_TRY(h, hipGetLastError());
  double v = 0;
  HIP_TRY(h, hipMemcpyAsync(&v, result, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  *out = v;
  return PS_MF_OK;
}

// The device address of `scratch` on the handle's device (current: ensure_device ran),
// looked up once per device and kept for the process.
constexpr int kMaxDevices = 256;
std::mutex scratch_mu;
double *scratch_dev[kMaxDevices] = {};

int scratch_address(ps_mf_t *h, double **out) {
  if (h->device < 0 || h->device >= kMaxDevices) return fail(h, PS_MF_EDEVICE, "device %d out of range", h->device);
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_dev[h->device]) {
    void *p = nullptr;
    HIP_TRY(h, hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(h, PS_MF_EDEVICE, "no device address for the static scratch");
    scratch_dev[h->device] = static_cast<double *>(p);
  }
  *out = scratch_dev[h->device];
  return PS_MF_OK;
}

}  // namespace

extern "C" {

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
  HIP_TRY(h, hipMemcpy2D(h->ring, h->Kp * sizeof(float), L, h->K * sizeof(float), h->K * sizeof(float),
                         static_cast<size_t>(h->N), hipMemcpyHostToDevice));
  HIP_TRY(h, hipMemcpy2D(h->ring + h->N * h->Kp, h->Kp * sizeof(float), R, h->K * sizeof(float),
                         h->K * sizeof(float), static_cast<size_t>(h->M), hipMemcpyHostToDevice));
  if (per_row_policy(h)) {
    // no row cached yet (version -1); slots 0 keep every address inside the ring
    const size_t ni = static_cast<size_t>(h->nclass) * static_cast<size_t>(h->M);
    HIP_TRY(h, hipMemset(h->ver_u, 0xff, h->N * sizeof(int32_t)));
    HIP_TRY(h, hipMemset(h->ver_i, 0xff, ni * sizeof(int32_t)));
    HIP_TRY(h, hipMemset(h->slot_u, 0, h->N * sizeof(int32_t)));
    HIP_TRY(h, hipMemset(h->slot_i, 0, ni * sizeof(int32_t)));
    HIP_TRY(h, hipMemset(h->stale, 0, (h->s + 1) * sizeof(unsigned long long)));
  }
  if (h->vap_norms)
    HIP_TRY(h, hipMemset(h->vap_norms, 0, static_cast<size_t>(h->vap_cap) * (h->s + 1) * sizeof(unsigned)));
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
  return loss_into(h, h->loss_partial, h->loss_out, out);
}

int ps_mf_loss_noalloc(ps_mf_t *h, double *out) {
  if (!h || !out) return PS_MF_EINVAL;
  if (!h->loaded) return fail(h, PS_MF_ESTATE, "load ratings and set factors before the loss");
  if (h->loss_parts > kNoAllocPartials)
    return fail(h, PS_MF_EINVAL, "the loss needs %lld partial sums; the static scratch holds %lld",
                (long long)h->loss_parts, (long long)kNoAllocPartials);
  if (!h->has_factors) return fail(h, PS_MF_ESTATE, "load ratings and set factors before the loss");
  int r = ensure_device(h);
  if (r) return r;
  double *sc = nullptr;
  if ((r = scratch_address(h, &sc))) return r;
  return loss_into(h, sc, sc + kNoAllocPartials, out);
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
  if ((kind == PS_MF_IDX_STALENESS || kind == PS_MF_IDX_ROW_VERSIONS) && !h->loaded)
    return fail(h, PS_MF_ESTATE, "no ratings loaded");
  if (kind != PS_MF_IDX_OWNER && kind != PS_MF_IDX_VERSION_LOG && kind != PS_MF_IDX_STALENESS &&
      kind != PS_MF_IDX_ROW_VERSIONS && kind != PS_MF_IDX_VAP_NORMS) {
    if (!h->loaded) return fail(h, PS_MF_ESTATE, "no ratings loaded");
    if (block < 0 || block >= h->B) return fail(h, PS_MF_EINVAL, "block %d out of range", block);
  }
  if (kind == PS_MF_IDX_SEQ_ORDER && h->step != PS_MF_STEP_SEQ)
    return fail(h, PS_MF_EINVAL, "the order of the sequential step exists under PS_MF_STEP_SEQ only");
  if (kind == PS_MF_IDX_VAP_NORMS && h->policy != PS_MF_VAP)
    return fail(h, PS_MF_EINVAL, "in-transit norms exist under PS_MF_VAP only");
  if (kind == PS_MF_IDX_VERSION_LOG || kind == PS_MF_IDX_STALENESS) {
    const int r = vap_sync_log(h);
    if (r) return r;
  }
  std::vector<double> vap_norms;
  if (kind == PS_MF_IDX_VAP_NORMS && h->clock > 0) {
    const int64_t S1 = h->s + 1;
    std::vector<unsigned> bits(static_cast<size_t>(h->clock * S1));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    HIP_TRY(h, hipMemcpy(bits.data(), h->vap_norms, bits.size() * sizeof(unsigned), hipMemcpyDeviceToHost));
    vap_norms.resize(bits.size());
    for (int64_t c = 0; c < h->clock; ++c)
      for (int64_t d = 0; d < S1; ++d) {
        float f;
        std::memcpy(&f, &bits[c * S1 + d], sizeof f);
        vap_norms[c * S1 + d] = d <= c ? static_cast<double>(f) : -1.0;
      }
  }
  if (kind == PS_MF_IDX_OWNER && h->owner.empty()) {
    h->owner.resize(static_cast<size_t>(h->N));
    for (int64_t i = 0; i < h->N; ++i) h->owner[i] = static_cast<int32_t>(i % h->P);
  }
  const void *src = nullptr;
  size_t esz = 0;
  int64_t n = 0;
  int64_t split[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (kind == PS_MF_IDX_SPLIT) {
    const psmf::BlockLayout &L = h->layout[block];
    auto unit_ratings = [](const psmf::UnitSet &u) {
      int64_t t = 0;
      for (int32_t len : u.unit_len) t += len;
      return t;
    };
    if (h->step == PS_MF_STEP_SEQ) {
      split[0] = static_cast<int64_t>(L.seq.chain_worker.size());
      for (uint8_t f : L.seq.flag) split[1] += (f & psmf::kSeqRunStart) != 0;
      split[2] = L.nnz;
    } else {
      split[0] = L.dense_user.nnz;
      split[1] = L.cells_user.nnz;
      split[2] = unit_ratings(L.by_user);
      split[3] = L.dense_item.nnz;
      split[4] = L.cells_item.nnz;
      split[5] = unit_ratings(L.by_item);
      split[6] = L.partial_rows_user;
      split[7] = L.partial_rows_item;
    }
  }
  std::vector<int64_t> stale, rowver, seq_order;
  if (kind == PS_MF_IDX_SEQ_ORDER) {
    const psmf::BlockLayout &L = h->layout[block];
    seq_order.resize(L.seq.canon.size());
    for (size_t x = 0; x < seq_order.size(); ++x) seq_order[x] = L.perm[L.seq.canon[x]];
  }
  if (kind == PS_MF_IDX_STALENESS) {
    stale.assign(static_cast<size_t>(h->s) + 1, 0);
    if (per_row_policy(h)) {
      // counted on the device by the per-row view kernel
      if (h->stale) {
        HIP_TRY(h, hipStreamSynchronize(h->stream));
        HIP_TRY(h, hipMemcpy(stale.data(), h->stale, stale.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
      }
    } else {
      // the version log holds v(p, c) for every clock run; worker p reads two rows per rating
      const int64_t clocks = static_cast<int64_t>(h->vlog.size()) / h->P;
      for (int64_t c = 0; c < clocks; ++c)
        for (int64_t p = 0; p < h->P; ++p)
          stale[static_cast<size_t>(c - h->vlog[c * h->P + p])] +=
              2 * h->worker_ratings[static_cast<size_t>(c % h->B) * h->P + p];
    }
  }
  if (kind == PS_MF_IDX_ROW_VERSIONS && per_row_policy(h)) {
    const size_t nu = static_cast<size_t>(h->N), ni = static_cast<size_t>(h->nclass) * static_cast<size_t>(h->M);
    rowver.assign(nu + ni, -1);
    if (h->ver_u && h->has_factors) {
      std::vector<int32_t> t(nu + ni);
      HIP_TRY(h, hipStreamSynchronize(h->stream));
      HIP_TRY(h, hipMemcpy(t.data(), h->ver_u, nu * sizeof(int32_t), hipMemcpyDeviceToHost));
      HIP_TRY(h, hipMemcpy(t.data() + nu, h->ver_i, ni * sizeof(int32_t), hipMemcpyDeviceToHost));
      for (size_t x = 0; x < nu + ni; ++x) rowver[x] = t[x];
    }
  }
  switch (kind) {
    case PS_MF_IDX_ROW_VERSIONS: src = rowver.data(); esz = 8; n = static_cast<int64_t>(rowver.size()); break;
    case PS_MF_IDX_STALENESS: src = stale.data(); esz = 8; n = h->s + 1; break;
    case PS_MF_IDX_OWNER: src = h->owner.data(); esz = 4; n = h->N; break;
    case PS_MF_IDX_ROW_PTR: src = h->layout[block].row_ptr.data(); esz = 8; n = h->N + 1; break;
    case PS_MF_IDX_COL: src = h->layout[block].col.data(); esz = 4; n = h->layout[block].nnz; break;
    case PS_MF_IDX_PERM: src = h->layout[block].perm.data(); esz = 8; n = h->layout[block].nnz; break;
    case PS_MF_IDX_USER_COUNT: src = h->layout[block].ucount.data(); esz = 4; n = h->N; break;
    case PS_MF_IDX_ITEM_COUNT: src = h->layout[block].icount.data(); esz = 4; n = h->M; break;
    case PS_MF_IDX_VERSION_LOG: src = h->vlog.data(); esz = 8; n = static_cast<int64_t>(h->vlog.size()); break;
    case PS_MF_IDX_SPLIT: src = split; esz = 8; n = 8; break;
    case PS_MF_IDX_SEQ_ORDER: src = seq_order.data(); esz = 8; n = static_cast<int64_t>(seq_order.size()); break;
    case PS_MF_IDX_VAP_NORMS: src = vap_norms.data(); esz = 8; n = static_cast<int64_t>(vap_norms.size()); break;
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
  if (h->side_stream) (void)hipStreamSynchronize(h->side_stream);
  if (h->cell_stream) (void)hipStreamSynchronize(h->cell_stream);
  for (hipGraphExec_t ex : h->seq_exec)
    if (ex) (void)hipGraphExecDestroy(ex);
  for (hipGraphExec_t ex : h->sweep_exec)
    if (ex) (void)hipGraphExecDestroy(ex);
  for (void *p : h->allocations) (void)hipFree(p);
  if (h->side_stream) (void)hipStreamDestroy(h->side_stream);
  if (h->cell_stream) (void)hipStreamDestroy(h->cell_stream);
  if (h->fork) (void)hipEventDestroy(h->fork);
  if (h->join) (void)hipEventDestroy(h->join);
  if (h->join_cells) (void)hipEventDestroy(h->join_cells);
  if (h->own_stream && h->stream) (void)hipStreamDestroy(h->stream);
  delete h;
}

}  // extern "C"
