// Map (Sec. III-A step 4), Fill-Values (step 5) and the sparse update of the
// embedding rows (step 7). The id lists come out of Unique strictly
// ascending, so every destination row is owned by exactly one wave: plain
// row stores, no atomics and no locks.
//
// Layout: lanes across the columns in 16-byte vectors (64 x VEC floats per
// vector step), NV vector steps per pass so a lane keeps NV loads of every
// operand in flight. Loop bounds and row indices are wave-uniform and loads
// are unconditional (a column past D loads a valid clamped column and is not
// stored): a load under a lane condition makes the compiler wait for every
// earlier load.
#include "common.hpp"

namespace lmz {

constexpr int kFillThreads = 256;
constexpr int kFillWaves = kFillThreads / kWave;
#ifndef LMZ_FILL_ROWS_PER_WAVE
#define LMZ_FILL_ROWS_PER_WAVE 1     // rows of a scatter / an update per wave
#endif
constexpr int kRowsPerWave = LMZ_FILL_ROWS_PER_WAVE;
#ifndef LMZ_ZERO_ROWS
#define LMZ_ZERO_ROWS 8              // rows a wave of the EXPAND zero fill stores
#endif
constexpr int kZeroRows = LMZ_ZERO_ROWS;
#ifndef LMZ_ZERO_NT
#define LMZ_ZERO_NT 1                // non-temporal stores for the zero fill
#endif

template <typename KeyT>
__device__ __forceinline__ int64_t find_row(const KeyT* __restrict__ ids, int64_t n, KeyT x) {
  const int64_t r = lower_bound_dev(ids, n, x);
  return (r < n && ids[r] == x) ? r : -1;
}

__device__ __forceinline__ int64_t clamp_count(const int64_t* n, int64_t cap, int32_t* dev_err,
                                               bool report) {
  int64_t v = *n;
  if (v > cap) {
    if (report) raise_err(dev_err, LM_DEVERR_CAPACITY);
    v = cap;
  }
  return v < 0 ? 0 : v;
}

// ---------------------------------------------------------------------------
// Map: map[u] = position of sub[u] in sup, or -1.
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ __launch_bounds__(kFillThreads) void k_map_ids(
    const KeyT* __restrict__ sub, const int64_t* __restrict__ n_sub, int64_t sub_cap,
    const KeyT* __restrict__ sup, const int64_t* __restrict__ n_sup, int64_t sup_cap,
    int32_t* __restrict__ map, int32_t* __restrict__ dev_err) {
  const int64_t i = blockIdx.x * int64_t(kFillThreads) + threadIdx.x;
  const int64_t n = clamp_count(n_sub, sub_cap, dev_err, i == 0);
  const int64_t ns = clamp_count(n_sup, sup_cap, dev_err, i == 0);
  bool missing = false;
  if (i < n) {
    const int64_t r = find_row(sup, ns, sub[i]);
    map[i] = static_cast<int32_t>(r);
    missing = r < 0;
  }
  if (ballot(missing) && lane_id() == 0) raise_err(dev_err, LM_DEVERR_NOT_FOUND);
}

// ---------------------------------------------------------------------------
// Columns of one pass: lane vectors at cb + j*64*VEC + lane*VEC, j < NV.
// ---------------------------------------------------------------------------
template <int VEC, int NV>
struct PassCols {
  int col[NV], ld[NV];
  bool ok[NV];
  __device__ __forceinline__ PassCols(int cb, int lane, int D) {
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      col[j] = cb + j * kWave * VEC + lane * VEC;
      ok[j] = col[j] < D;
      ld[j] = ok[j] ? col[j] : D - VEC;  // a valid column, loaded and not stored
    }
  }
};

template <int VEC, int NV>
__device__ __forceinline__ void copy_row(float* __restrict__ dst, const float* __restrict__ src,
                                         int D, int lane) {
  for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
    const PassCols<VEC, NV> pc(cb, lane, D);
    float v[NV][VEC];
#pragma unroll
    for (int j = 0; j < NV; ++j) load_vec<VEC>(src + pc.ld[j], v[j]);
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (pc.ok[j]) store_vec<VEC>(dst + pc.col[j], v[j]);
  }
}

template <int VEC, int NV>
__device__ __forceinline__ void zero_row(float* __restrict__ dst, int D, int lane) {
  float z[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) z[e] = 0.f;
  for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
    const PassCols<VEC, NV> pc(cb, lane, D);
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (pc.ok[j]) {
#if LMZ_ZERO_NT
        store_vec_nt<VEC>(dst + pc.col[j], z);
#else
        store_vec<VEC>(dst + pc.col[j], z);
#endif
      }
  }
}

template <int VEC, int NV>
__device__ __forceinline__ void add_row(float* __restrict__ dst, const float* __restrict__ src,
                                        int D, int lane) {
  for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
    const PassCols<VEC, NV> pc(cb, lane, D);
    float v[NV][VEC], t[NV][VEC];
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      load_vec<VEC>(src + pc.ld[j], v[j]);
      load_vec<VEC>(dst + pc.ld[j], t[j]);
    }
#pragma unroll
    for (int j = 0; j < NV; ++j) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) t[j][e] += v[j][e];
      if (pc.ok[j]) store_vec<VEC>(dst + pc.col[j], t[j]);
    }
  }
}

// ---------------------------------------------------------------------------
// EXPAND (step 5): the zero fill of rows [0, n_dst) of dst, then the SCATTER
// of the source rows into the rows of dst_ids (k_scatter, which also flags a
// source id missing from dst_ids). The fill is a pure store stream: a wave
// zeroes kZeroRows consecutive rows (most of the merged rows have no source
// on a given shard). Writing the few present rows twice is cheaper than
// interleaving their loads with the fill, whose stores a later load would
// have to wait for.
// ---------------------------------------------------------------------------
template <int VEC, int NV>
__global__ __launch_bounds__(kFillThreads) void k_zero_rows(
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, float* __restrict__ dst,
    int64_t ld_dst, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = first_lane(static_cast<int64_t>(blockIdx.x) * kFillWaves + (threadIdx.x >> 6));
  const int64_t nd = first_lane(clamp_count(n_dst, dst_rows, dev_err, w == 0 && lane == 0));
  for (int64_t r0 = w * kZeroRows; r0 < nd; r0 += nwaves * kZeroRows) {
    const int nr = nd - r0 < kZeroRows ? static_cast<int>(nd - r0) : kZeroRows;
    for (int j = 0; j < nr; ++j) zero_row<VEC, NV>(dst + (r0 + j) * ld_dst, D, lane);
  }
}

// ---------------------------------------------------------------------------
// SCATTER / SCATTER_ADD: kRowsPerWave source rows per wave (grid-stride).
// ---------------------------------------------------------------------------
template <typename KeyT, int VEC, int NV, bool ADD>
__global__ __launch_bounds__(kFillThreads) void k_scatter(
    const float* __restrict__ src, int64_t ld_src, const KeyT* __restrict__ src_ids,
    const int64_t* __restrict__ n_src, int64_t src_cap, const KeyT* __restrict__ dst_ids,
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, float* __restrict__ dst,
    int64_t ld_dst, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = first_lane(static_cast<int64_t>(blockIdx.x) * kFillWaves + (threadIdx.x >> 6));
  const bool first = w == 0 && lane == 0;
  const int64_t ns = first_lane(clamp_count(n_src, src_cap, dev_err, first));
  const int64_t nd = dst_ids ? first_lane(clamp_count(n_dst, dst_rows, dev_err, first)) : dst_rows;
  for (int64_t u = w; u < ns; u += nwaves) {
    const KeyT id = first_lane(src_ids[u]);
    int64_t row;
    if (dst_ids) {
      const int64_t lb = lower_bound_wave(dst_ids, nd, id);
      row = (lb < nd && first_lane(dst_ids[lb]) == id) ? lb : -1;
      if (row < 0 && lane == 0) raise_err(dev_err, LM_DEVERR_NOT_FOUND);
    } else {
      row = (id >= 0 && static_cast<int64_t>(id) < dst_rows) ? static_cast<int64_t>(id) : -1;
      if (row < 0 && lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
    }
    if (row < 0) continue;
    if (ADD) add_row<VEC, NV>(dst + row * ld_dst, src + u * ld_src, D, lane);
    else copy_row<VEC, NV>(dst + row * ld_dst, src + u * ld_src, D, lane);
  }
}

// ---------------------------------------------------------------------------
// binary16 payload (Sec. III-C): EXPAND / SCATTER of fp32 rows into a
// binary16 matrix, each value multiplied by the compression scale in fp32
// and rounded once. A stored inf or NaN raises LM_DEVERR_NONFINITE.
// ---------------------------------------------------------------------------
template <int VEC, int NV>
__global__ __launch_bounds__(kFillThreads) void k_zero_rows_h(
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, uint16_t* __restrict__ dst,
    int64_t ld_dst, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = first_lane(static_cast<int64_t>(blockIdx.x) * kFillWaves + (threadIdx.x >> 6));
  const int64_t nd = first_lane(clamp_count(n_dst, dst_rows, dev_err, w == 0 && lane == 0));
  for (int64_t r0 = w * kZeroRows; r0 < nd; r0 += nwaves * kZeroRows) {
    const int nr = nd - r0 < kZeroRows ? static_cast<int>(nd - r0) : kZeroRows;
    for (int j = 0; j < nr; ++j) {
      uint16_t* row = dst + (r0 + j) * ld_dst;
      for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
        const PassCols<VEC, NV> pc(cb, lane, D);
#pragma unroll
        for (int k = 0; k < NV; ++k)
          if (pc.ok[k]) store_half_zero<VEC>(row + pc.col[k]);
      }
    }
  }
}

template <typename KeyT, int VEC, int NV>
__global__ __launch_bounds__(kFillThreads) void k_scatter_h(
    const float* __restrict__ src, int64_t ld_src, const KeyT* __restrict__ src_ids,
    const int64_t* __restrict__ n_src, int64_t src_cap, const KeyT* __restrict__ dst_ids,
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, uint16_t* __restrict__ dst,
    int64_t ld_dst, float scale, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = first_lane(static_cast<int64_t>(blockIdx.x) * kFillWaves + (threadIdx.x >> 6));
  const bool first = w == 0 && lane == 0;
  const int64_t ns = first_lane(clamp_count(n_src, src_cap, dev_err, first));
  const int64_t nd = dst_ids ? first_lane(clamp_count(n_dst, dst_rows, dev_err, first)) : dst_rows;
  bool bad = false;
  for (int64_t u = w; u < ns; u += nwaves) {
    const KeyT id = first_lane(src_ids[u]);
    int64_t row;
    if (dst_ids) {
      const int64_t lb = lower_bound_wave(dst_ids, nd, id);
      row = (lb < nd && first_lane(dst_ids[lb]) == id) ? lb : -1;
      if (row < 0 && lane == 0) raise_err(dev_err, LM_DEVERR_NOT_FOUND);
    } else {
      row = (id >= 0 && static_cast<int64_t>(id) < dst_rows) ? static_cast<int64_t>(id) : -1;
      if (row < 0 && lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
    }
    if (row < 0) continue;
    const float* srow = src + u * ld_src;
    uint16_t* drow = dst + row * ld_dst;
    for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
      const PassCols<VEC, NV> pc(cb, lane, D);
      float v[NV][VEC];
#pragma unroll
      for (int k = 0; k < NV; ++k) load_vec<VEC>(srow + pc.ld[k], v[k]);
#pragma unroll
      for (int k = 0; k < NV; ++k)
        if (pc.ok[k]) bad |= store_half_scaled<VEC>(drow + pc.col[k], v[k], scale);
    }
  }
  if (ballot(bad) && lane == 0) raise_err(dev_err, LM_DEVERR_NONFINITE);
}

// ---------------------------------------------------------------------------
// Sparse apply (step 7): one wave per touched row (the update of each value:
// sgd_value, adam_value).
// ---------------------------------------------------------------------------

// ValT float: fp32 gradients; ValT uint16_t: the binary16 payload of
// Sec. III-C, each value multiplied by o.g_scale (1/F) after the up-cast.
template <typename KeyT, typename ValT, int VEC, int NV, bool ADAM>
__global__ __launch_bounds__(kFillThreads) void k_apply(
    float* __restrict__ table, int64_t V, int D, int64_t ld_table, const KeyT* __restrict__ rows,
    const int64_t* __restrict__ n_rows, int64_t rows_cap, const ValT* __restrict__ vals,
    int64_t ld_vals, OptParams o, float* __restrict__ m, float* __restrict__ v, int64_t nwaves,
    int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = first_lane(static_cast<int64_t>(blockIdx.x) * kFillWaves + (threadIdx.x >> 6));
  const int64_t n = first_lane(clamp_count(n_rows, rows_cap, dev_err, w == 0 && lane == 0));
  for (int64_t u = w; u < n; u += nwaves) {
    const KeyT id = first_lane(rows[u]);
    if (!(id >= 0 && static_cast<int64_t>(id) < V)) {
      if (lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
      continue;
    }
    float* p = table + static_cast<int64_t>(id) * ld_table;
    const ValT* g = vals + u * ld_vals;
    float* mm = ADAM ? m + static_cast<int64_t>(id) * ld_table : nullptr;
    float* vv = ADAM ? v + static_cast<int64_t>(id) * ld_table : nullptr;
    for (int cb = 0; cb < D; cb += NV * kWave * VEC) {
      const PassCols<VEC, NV> pc(cb, lane, D);
      float gr[NV][VEC], pr[NV][VEC], mr[NV][VEC], vr[NV][VEC];
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        if constexpr (sizeof(ValT) == 2) load_half_scaled<VEC>(g + pc.ld[j], gr[j], o.g_scale);
        else load_vec<VEC>(g + pc.ld[j], gr[j]);
        load_vec<VEC>(p + pc.ld[j], pr[j]);
        if constexpr (ADAM) {
          load_vec<VEC>(mm + pc.ld[j], mr[j]);
          load_vec<VEC>(vv + pc.ld[j], vr[j]);
        }
      }
#pragma unroll
      for (int j = 0; j < NV; ++j) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          if constexpr (ADAM) adam_value(pr[j][e], mr[j][e], vr[j][e], gr[j][e], o);
          else sgd_value(pr[j][e], gr[j][e], o);
        }
        if (pc.ok[j]) {
          store_vec<VEC>(p + pc.col[j], pr[j]);
          if constexpr (ADAM) {
            store_vec<VEC>(mm + pc.col[j], mr[j]);
            store_vec<VEC>(vv + pc.col[j], vr[j]);
          }
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
static bool a16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Waves for `rows` rows at `per` rows per wave (grid-stride beyond a million).
static int64_t grid_waves(int64_t rows, int per) {
  int64_t w = (rows + per - 1) / per;
  if (w < 1) w = 1;
  const int64_t cap = int64_t(1) << 20;
  return w < cap ? w : cap;
}

template <typename KeyT>
static int map_run_t(const void* sub, const int64_t* n_sub, int64_t sub_cap, const void* sup,
                     const int64_t* n_sup, int64_t sup_cap, int32_t* map, int32_t* dev_err,
                     hipStream_t st) {
  if (sub_cap == 0) return LM_OK;
  const int64_t blocks = (sub_cap + kFillThreads - 1) / kFillThreads;
  k_map_ids<KeyT><<<dim3(static_cast<uint32_t>(blocks)), kFillThreads, 0, st>>>(
      static_cast<const KeyT*>(sub), n_sub, sub_cap, static_cast<const KeyT*>(sup), n_sup, sup_cap,
      map, dev_err);
  return launch_status(hipGetLastError());
}

int map_run(const void* sub, const int64_t* n_sub, int64_t sub_cap, const void* sup,
            const int64_t* n_sup, int64_t sup_cap, int idtype, int32_t* map, int32_t* dev_err,
            hipStream_t st) {
  return idtype == LM_I64
             ? map_run_t<int64_t>(sub, n_sub, sub_cap, sup, n_sup, sup_cap, map, dev_err, st)
             : map_run_t<int32_t>(sub, n_sub, sub_cap, sup, n_sup, sup_cap, map, dev_err, st);
}

template <typename KeyT, int VEC>
static hipError_t fill_launch(const float* src, int64_t ld_src, const void* src_ids,
                              const int64_t* n_src, int64_t src_cap, const void* dst_ids,
                              const int64_t* n_dst, int64_t D, float* dst, int64_t dst_rows,
                              int64_t ld_dst, int mode, int32_t* dev_err, hipStream_t st) {
  const KeyT* si = static_cast<const KeyT*>(src_ids);
  const KeyT* di = static_cast<const KeyT*>(dst_ids);
  if (mode == LM_FILL_EXPAND) {
    const int64_t waves = grid_waves(dst_rows, kZeroRows);
    const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
    k_zero_rows<VEC, 4><<<blocks, kFillThreads, 0, st>>>(
        n_dst, dst_rows, static_cast<int>(D), dst, ld_dst, int64_t(blocks) * kFillWaves, dev_err);
    if (src_cap == 0) return hipGetLastError();
    const int64_t swaves = grid_waves(src_cap, kRowsPerWave);
    const uint32_t sblocks = static_cast<uint32_t>((swaves + kFillWaves - 1) / kFillWaves);
    k_scatter<KeyT, VEC, 4, false><<<sblocks, kFillThreads, 0, st>>>(
        src, ld_src, si, n_src, src_cap, di, n_dst, dst_rows, static_cast<int>(D), dst, ld_dst,
        int64_t(sblocks) * kFillWaves, dev_err);
  } else {
    const int64_t waves = grid_waves(src_cap, kRowsPerWave);
    const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
    if (mode == LM_FILL_SCATTER)
      k_scatter<KeyT, VEC, 4, false><<<blocks, kFillThreads, 0, st>>>(
          src, ld_src, si, n_src, src_cap, di, n_dst, dst_rows, static_cast<int>(D), dst, ld_dst,
          int64_t(blocks) * kFillWaves, dev_err);
    else
      k_scatter<KeyT, VEC, 4, true><<<blocks, kFillThreads, 0, st>>>(
          src, ld_src, si, n_src, src_cap, di, n_dst, dst_rows, static_cast<int>(D), dst, ld_dst,
          int64_t(blocks) * kFillWaves, dev_err);
  }
  return hipGetLastError();
}

int fill_run(const float* src, int64_t ld_src, const void* src_ids, const int64_t* n_src,
             int64_t src_cap, const void* dst_ids, const int64_t* n_dst, int idtype, int64_t D,
             float* dst, int64_t dst_rows, int64_t ld_dst, int mode, int32_t* dev_err,
             hipStream_t st) {
  if (D == 0) return LM_OK;
  if (mode == LM_FILL_EXPAND ? dst_rows == 0 : src_cap == 0) return LM_OK;
  const bool vec = a16(src) && a16(dst) && ld_src % 4 == 0 && ld_dst % 4 == 0 && D % 4 == 0;
  hipError_t e;
  if (idtype == LM_I64)
    e = vec ? fill_launch<int64_t, 4>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D, dst,
                                      dst_rows, ld_dst, mode, dev_err, st)
            : fill_launch<int64_t, 1>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D, dst,
                                      dst_rows, ld_dst, mode, dev_err, st);
  else
    e = vec ? fill_launch<int32_t, 4>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D, dst,
                                      dst_rows, ld_dst, mode, dev_err, st)
            : fill_launch<int32_t, 1>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D, dst,
                                      dst_rows, ld_dst, mode, dev_err, st);
  return launch_status(e);
}

template <typename KeyT, typename ValT, int VEC, int NV>
static hipError_t apply_launch(float* table, int64_t V, int64_t D, int64_t ld_table,
                               const void* rows, const int64_t* n_rows, int64_t rows_cap,
                               const ValT* vals, int64_t ld_vals, bool adam, const OptParams& o,
                               float* m, float* v, int32_t* dev_err, hipStream_t st) {
  const int64_t waves = grid_waves(rows_cap, kRowsPerWave);
  const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
  const KeyT* r = static_cast<const KeyT*>(rows);
  if (adam)
    k_apply<KeyT, ValT, VEC, NV, true><<<blocks, kFillThreads, 0, st>>>(
        table, V, static_cast<int>(D), ld_table, r, n_rows, rows_cap, vals, ld_vals, o, m, v,
        int64_t(blocks) * kFillWaves, dev_err);
  else
    k_apply<KeyT, ValT, VEC, NV, false><<<blocks, kFillThreads, 0, st>>>(
        table, V, static_cast<int>(D), ld_table, r, n_rows, rows_cap, vals, ld_vals, o, m, v,
        int64_t(blocks) * kFillWaves, dev_err);
  return hipGetLastError();
}

static OptParams opt_params(int opt, float lr, float beta1, float beta2, float eps,
                            float weight_decay, int64_t step, float g_scale) {
  return make_opt_params(opt == LM_OPT_ADAM, lr, beta1, beta2, eps, weight_decay, step, g_scale);
}

int apply_run(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows, int idtype,
              const int64_t* n_rows, int64_t rows_cap, const float* vals, int64_t ld_vals,
              int opt, float lr, float beta1, float beta2, float eps, float weight_decay,
              int64_t step, float* m, float* v, int32_t* dev_err, hipStream_t st) {
  if (D == 0 || rows_cap == 0) return LM_OK;
  const bool adam = opt == LM_OPT_ADAM;
  const OptParams o = opt_params(opt, lr, beta1, beta2, eps, weight_decay, step, 1.f);
  bool vec = a16(table) && a16(vals) && ld_table % 4 == 0 && ld_vals % 4 == 0 && D % 4 == 0;
  if (adam) vec = vec && a16(m) && a16(v);
  hipError_t e;
  if (idtype == LM_I64)
    e = vec ? apply_launch<int64_t, float, 4, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                 vals, ld_vals, adam, o, m, v, dev_err, st)
            : apply_launch<int64_t, float, 1, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                 vals, ld_vals, adam, o, m, v, dev_err, st);
  else
    e = vec ? apply_launch<int32_t, float, 4, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                 vals, ld_vals, adam, o, m, v, dev_err, st)
            : apply_launch<int32_t, float, 1, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                 vals, ld_vals, adam, o, m, v, dev_err, st);
  return launch_status(e);
}

int apply_run_f16(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows,
                  int idtype, const int64_t* n_rows, int64_t rows_cap, const uint16_t* vals,
                  int64_t ld_vals, float inv_scale, int opt, float lr, float beta1, float beta2,
                  float eps, float weight_decay, int64_t step, float* m, float* v,
                  int32_t* dev_err, hipStream_t st) {
  if (D == 0 || rows_cap == 0) return LM_OK;
  const bool adam = opt == LM_OPT_ADAM;
  const OptParams o = opt_params(opt, lr, beta1, beta2, eps, weight_decay, step, inv_scale);
  // 8 columns per lane: one 16-byte payload vector, two of every fp32 table.
  bool vec = a16(table) && a16(vals) && ld_table % 4 == 0 && ld_vals % 8 == 0 && D % 8 == 0;
  if (adam) vec = vec && a16(m) && a16(v);
  hipError_t e;
  if (idtype == LM_I64)
    e = vec ? apply_launch<int64_t, uint16_t, 8, 2>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                    vals, ld_vals, adam, o, m, v, dev_err, st)
            : apply_launch<int64_t, uint16_t, 1, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                    vals, ld_vals, adam, o, m, v, dev_err, st);
  else
    e = vec ? apply_launch<int32_t, uint16_t, 8, 2>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                    vals, ld_vals, adam, o, m, v, dev_err, st)
            : apply_launch<int32_t, uint16_t, 1, 4>(table, V, D, ld_table, rows, n_rows, rows_cap,
                                                    vals, ld_vals, adam, o, m, v, dev_err, st);
  return launch_status(e);
}

template <typename KeyT, int VEC>
static hipError_t fill_launch_f16(const float* src, int64_t ld_src, const void* src_ids,
                                  const int64_t* n_src, int64_t src_cap, const void* dst_ids,
                                  const int64_t* n_dst, int64_t D, uint16_t* dst,
                                  int64_t dst_rows, int64_t ld_dst, int mode, float scale,
                                  int32_t* dev_err, hipStream_t st) {
  constexpr int NV = VEC == 8 ? 2 : 4;
  const KeyT* si = static_cast<const KeyT*>(src_ids);
  const KeyT* di = static_cast<const KeyT*>(dst_ids);
  if (mode == LM_FILL_EXPAND) {
    const int64_t waves = grid_waves(dst_rows, kZeroRows);
    const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
    k_zero_rows_h<VEC, NV><<<blocks, kFillThreads, 0, st>>>(
        n_dst, dst_rows, static_cast<int>(D), dst, ld_dst, int64_t(blocks) * kFillWaves, dev_err);
    if (src_cap == 0) return hipGetLastError();
  }
  const int64_t swaves = grid_waves(src_cap, kRowsPerWave);
  const uint32_t sblocks = static_cast<uint32_t>((swaves + kFillWaves - 1) / kFillWaves);
  k_scatter_h<KeyT, VEC, NV><<<sblocks, kFillThreads, 0, st>>>(
      src, ld_src, si, n_src, src_cap, di, n_dst, dst_rows, static_cast<int>(D), dst, ld_dst,
      scale, int64_t(sblocks) * kFillWaves, dev_err);
  return hipGetLastError();
}

int fill_run_f16(const float* src, int64_t ld_src, const void* src_ids, const int64_t* n_src,
                 int64_t src_cap, const void* dst_ids, const int64_t* n_dst, int idtype,
                 int64_t D, uint16_t* dst, int64_t dst_rows, int64_t ld_dst, int mode,
                 float scale, int32_t* dev_err, hipStream_t st) {
  if (D == 0) return LM_OK;
  if (mode == LM_FILL_EXPAND ? dst_rows == 0 : src_cap == 0) return LM_OK;
  const bool vec = a16(src) && a16(dst) && ld_src % 4 == 0 && ld_dst % 8 == 0 && D % 8 == 0;
  hipError_t e;
  if (idtype == LM_I64)
    e = vec ? fill_launch_f16<int64_t, 8>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D,
                                          dst, dst_rows, ld_dst, mode, scale, dev_err, st)
            : fill_launch_f16<int64_t, 1>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D,
                                          dst, dst_rows, ld_dst, mode, scale, dev_err, st);
  else
    e = vec ? fill_launch_f16<int32_t, 8>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D,
                                          dst, dst_rows, ld_dst, mode, scale, dev_err, st)
            : fill_launch_f16<int32_t, 1>(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, D,
                                          dst, dst_rows, ld_dst, mode, scale, dev_err, st);
  return launch_status(e);
}

}  // namespace lmz

// ---------------------------------------------------------------------------
// Candidate sampler of the sampled softmax (Sec. II-A, Sec. III-B): the id of
// a 64-bit random word r is floor(r * V / 2^64), the high word of the
// product, so every id in [0, V) is equally likely. The random words come
// from the caller (one stream per seed group of GPUs).
// ---------------------------------------------------------------------------
namespace lmz {

template <typename KeyT>
__global__ __launch_bounds__(kFillThreads) void k_sample_ids(const uint64_t* __restrict__ r,
                                                             int64_t n, uint64_t V,
                                                             KeyT* __restrict__ ids) {
  for (int64_t i = blockIdx.x * int64_t(kFillThreads) + threadIdx.x; i < n;
       i += int64_t(gridDim.x) * kFillThreads)
    ids[i] = static_cast<KeyT>(__umul64hi(r[i], V));
}

int sample_run(const uint64_t* r, int64_t n, int64_t V, void* ids, int idtype, hipStream_t st) {
  if (n == 0) return LM_OK;
  int64_t blocks = (n + kFillThreads - 1) / kFillThreads;
  if (blocks > 65536) blocks = 65536;
  if (idtype == LM_I64)
    k_sample_ids<int64_t><<<static_cast<uint32_t>(blocks), kFillThreads, 0, st>>>(
        r, n, static_cast<uint64_t>(V), static_cast<int64_t*>(ids));
  else
    k_sample_ids<int32_t><<<static_cast<uint32_t>(blocks), kFillThreads, 0, st>>>(
        r, n, static_cast<uint64_t>(V), static_cast<int32_t*>(ids));
  return launch_status(hipGetLastError());
}

}  // namespace lmz
