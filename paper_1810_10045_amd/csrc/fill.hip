// Map (Sec. III-A step 4), Fill-Values (step 5) and the sparse update of the
// embedding rows (step 7). The id lists come out of Unique strictly
// ascending, so every destination row is owned by exactly one wave: plain
// row stores, no atomics and no locks.
//
// Layout: one wave per row, lanes across the columns in 16-byte vectors
// (64 x 4 floats = 256 columns per vector step), NV vector steps unrolled so
// a lane keeps NV loads of every operand in flight.
#include "common.hpp"

namespace lmz {

constexpr int kFillThreads = 256;
constexpr int kFillWaves = kFillThreads / kWave;

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
// Row helpers: lanes cover columns [lane*VEC + j*64*VEC] for j < steps.
// ---------------------------------------------------------------------------
template <int VEC, int NV>
__device__ __forceinline__ void copy_row(float* __restrict__ dst, const float* __restrict__ src,
                                         int D, int lane) {
  for (int c0 = lane * VEC; c0 < D; c0 += NV * kWave * VEC) {
    float v[NV][VEC];
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (c0 + j * kWave * VEC < D) load_vec<VEC>(src + c0 + j * kWave * VEC, v[j]);
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (c0 + j * kWave * VEC < D) store_vec<VEC>(dst + c0 + j * kWave * VEC, v[j]);
  }
}

template <int VEC, int NV>
__device__ __forceinline__ void zero_row(float* __restrict__ dst, int D, int lane) {
  float z[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) z[e] = 0.f;
  for (int c0 = lane * VEC; c0 < D; c0 += kWave * VEC) store_vec<VEC>(dst + c0, z);
}

template <int VEC, int NV>
__device__ __forceinline__ void add_row(float* __restrict__ dst, const float* __restrict__ src,
                                        int D, int lane) {
  for (int c0 = lane * VEC; c0 < D; c0 += NV * kWave * VEC) {
    float v[NV][VEC], t[NV][VEC];
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (c0 + j * kWave * VEC < D) {
        load_vec<VEC>(src + c0 + j * kWave * VEC, v[j]);
        load_vec<VEC>(dst + c0 + j * kWave * VEC, t[j]);
      }
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (c0 + j * kWave * VEC < D) {
#pragma unroll
        for (int e = 0; e < VEC; ++e) t[j][e] += v[j][e];
        store_vec<VEC>(dst + c0 + j * kWave * VEC, t[j]);
      }
  }
}

// ---------------------------------------------------------------------------
// EXPAND: one wave per destination row r < n_dst: dst[r] = src[u] where
// src_ids[u] == dst_ids[r], else zeros. The same waves also check that every
// source id occurs in dst_ids (LM_DEVERR_NOT_FOUND otherwise).
// ---------------------------------------------------------------------------
template <typename KeyT, int VEC, int NV>
__global__ __launch_bounds__(kFillThreads) void k_expand(
    const float* __restrict__ src, int64_t ld_src, const KeyT* __restrict__ src_ids,
    const int64_t* __restrict__ n_src, int64_t src_cap, const KeyT* __restrict__ dst_ids,
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, float* __restrict__ dst,
    int64_t ld_dst, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = blockIdx.x * int64_t(kFillWaves) + (threadIdx.x >> 6);
  const bool first = w == 0 && lane == 0;
  const int64_t ns = clamp_count(n_src, src_cap, dev_err, first);
  const int64_t nd = clamp_count(n_dst, dst_rows, dev_err, first);
  // Source-side check: lanes of the waves cover the source ids.
  bool missing = false;
  for (int64_t u = w * kWave + lane; u < ns; u += nwaves * kWave)
    missing |= find_row(dst_ids, nd, src_ids[u]) < 0;
  if (ballot(missing) && lane == 0) raise_err(dev_err, LM_DEVERR_NOT_FOUND);

  for (int64_t r = w; r < nd; r += nwaves) {
    const int64_t u = find_row(src_ids, ns, dst_ids[r]);  // uniform: same r in every lane
    float* d = dst + r * ld_dst;
    if (u >= 0) copy_row<VEC, NV>(d, src + u * ld_src, D, lane);
    else zero_row<VEC, NV>(d, D, lane);
  }
}

// ---------------------------------------------------------------------------
// SCATTER / SCATTER_ADD: one wave per source row.
// ---------------------------------------------------------------------------
template <typename KeyT, int VEC, int NV, bool ADD>
__global__ __launch_bounds__(kFillThreads) void k_scatter(
    const float* __restrict__ src, int64_t ld_src, const KeyT* __restrict__ src_ids,
    const int64_t* __restrict__ n_src, int64_t src_cap, const KeyT* __restrict__ dst_ids,
    const int64_t* __restrict__ n_dst, int64_t dst_rows, int D, float* __restrict__ dst,
    int64_t ld_dst, int64_t nwaves, int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = blockIdx.x * int64_t(kFillWaves) + (threadIdx.x >> 6);
  const bool first = w == 0 && lane == 0;
  const int64_t ns = clamp_count(n_src, src_cap, dev_err, first);
  const int64_t nd = dst_ids ? clamp_count(n_dst, dst_rows, dev_err, first) : dst_rows;
  for (int64_t u = w; u < ns; u += nwaves) {
    const KeyT id = src_ids[u];
    int64_t row;
    if (dst_ids) {
      row = find_row(dst_ids, nd, id);
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
// Sparse apply (step 7): one wave per touched row.
// ---------------------------------------------------------------------------
struct OptParams {
  float lr, b1, b2, eps, wd, inv_c1, inv_c2;
};

template <typename KeyT, int VEC, int NV, bool ADAM>
__global__ __launch_bounds__(kFillThreads) void k_apply(
    float* __restrict__ table, int64_t V, int D, int64_t ld_table, const KeyT* __restrict__ rows,
    const int64_t* __restrict__ n_rows, int64_t rows_cap, const float* __restrict__ vals,
    int64_t ld_vals, OptParams o, float* __restrict__ m, float* __restrict__ v, int64_t nwaves,
    int32_t* __restrict__ dev_err) {
  const int lane = lane_id();
  const int64_t w = blockIdx.x * int64_t(kFillWaves) + (threadIdx.x >> 6);
  const int64_t n = clamp_count(n_rows, rows_cap, dev_err, w == 0 && lane == 0);
  for (int64_t u = w; u < n; u += nwaves) {
    const KeyT id = rows[u];
    if (!(id >= 0 && static_cast<int64_t>(id) < V)) {
      if (lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
      continue;
    }
    float* p = table + static_cast<int64_t>(id) * ld_table;
    const float* g = vals + u * ld_vals;
    float* mm = ADAM ? m + static_cast<int64_t>(id) * ld_table : nullptr;
    float* vv = ADAM ? v + static_cast<int64_t>(id) * ld_table : nullptr;
    for (int c0 = lane * VEC; c0 < D; c0 += NV * kWave * VEC) {
      float gr[NV][VEC], pr[NV][VEC], mr[NV][VEC], vr[NV][VEC];
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int c = c0 + j * kWave * VEC;
        if (c < D) {
          load_vec<VEC>(g + c, gr[j]);
          load_vec<VEC>(p + c, pr[j]);
          if constexpr (ADAM) {
            load_vec<VEC>(mm + c, mr[j]);
            load_vec<VEC>(vv + c, vr[j]);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        const int c = c0 + j * kWave * VEC;
        if (c < D) {
#pragma unroll
          for (int e = 0; e < VEC; ++e) {
            if constexpr (ADAM) {
              const float gg = gr[j][e];
              mr[j][e] = o.b1 * mr[j][e] + (1.f - o.b1) * gg;
              vr[j][e] = o.b2 * vr[j][e] + (1.f - o.b2) * gg * gg;
              const float mhat = mr[j][e] * o.inv_c1;
              const float vhat = vr[j][e] * o.inv_c2;
              pr[j][e] -= o.lr * (mhat / (sqrtf(vhat) + o.eps) + o.wd * pr[j][e]);
            } else {
              pr[j][e] -= o.lr * gr[j][e];
            }
          }
          store_vec<VEC>(p + c, pr[j]);
          if constexpr (ADAM) {
            store_vec<VEC>(mm + c, mr[j]);
            store_vec<VEC>(vv + c, vr[j]);
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

static int64_t grid_waves(int64_t rows) {
  int64_t w = rows < 1 ? 1 : rows;
  const int64_t cap = int64_t(1) << 20;  // grid-stride beyond a million waves
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
    const int64_t waves = grid_waves(dst_rows);
    const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
    k_expand<KeyT, VEC, 4><<<blocks, kFillThreads, 0, st>>>(
        src, ld_src, si, n_src, src_cap, di, n_dst, dst_rows, static_cast<int>(D), dst, ld_dst,
        int64_t(blocks) * kFillWaves, dev_err);
  } else {
    const int64_t waves = grid_waves(src_cap);
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

template <typename KeyT, int VEC>
static hipError_t apply_launch(float* table, int64_t V, int64_t D, int64_t ld_table,
                               const void* rows, const int64_t* n_rows, int64_t rows_cap,
                               const float* vals, int64_t ld_vals, bool adam, const OptParams& o,
                               float* m, float* v, int32_t* dev_err, hipStream_t st) {
  const int64_t waves = grid_waves(rows_cap);
  const uint32_t blocks = static_cast<uint32_t>((waves + kFillWaves - 1) / kFillWaves);
  const KeyT* r = static_cast<const KeyT*>(rows);
  if (adam)
    k_apply<KeyT, VEC, 4, true><<<blocks, kFillThreads, 0, st>>>(
        table, V, static_cast<int>(D), ld_table, r, n_rows, rows_cap, vals, ld_vals, o, m, v,
        int64_t(blocks) * kFillWaves, dev_err);
  else
    k_apply<KeyT, VEC, 4, false><<<blocks, kFillThreads, 0, st>>>(
        table, V, static_cast<int>(D), ld_table, r, n_rows, rows_cap, vals, ld_vals, o, m, v,
        int64_t(blocks) * kFillWaves, dev_err);
  return hipGetLastError();
}

int apply_run(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows, int idtype,
              const int64_t* n_rows, int64_t rows_cap, const float* vals, int64_t ld_vals,
              int opt, float lr, float beta1, float beta2, float eps, float weight_decay,
              int64_t step, float* m, float* v, int32_t* dev_err, hipStream_t st) {
  if (D == 0 || rows_cap == 0) return LM_OK;
  const bool adam = opt == LM_OPT_ADAM;
  OptParams o{};
  o.lr = lr;
  o.b1 = beta1;
  o.b2 = beta2;
  o.eps = eps;
  o.wd = weight_decay;
  if (adam) {
    // Bias corrections 1 - beta^t, computed once on the host in double.
    o.inv_c1 = static_cast<float>(1.0 / (1.0 - __builtin_pow(static_cast<double>(beta1), static_cast<double>(step))));
    o.inv_c2 = static_cast<float>(1.0 / (1.0 - __builtin_pow(static_cast<double>(beta2), static_cast<double>(step))));
  }
  bool vec = a16(table) && a16(vals) && ld_table % 4 == 0 && ld_vals % 4 == 0 && D % 4 == 0;
  if (adam) vec = vec && a16(m) && a16(v);
  hipError_t e;
  if (idtype == LM_I64)
    e = vec ? apply_launch<int64_t, 4>(table, V, D, ld_table, rows, n_rows, rows_cap, vals, ld_vals,
                                       adam, o, m, v, dev_err, st)
            : apply_launch<int64_t, 1>(table, V, D, ld_table, rows, n_rows, rows_cap, vals, ld_vals,
                                       adam, o, m, v, dev_err, st);
  else
    e = vec ? apply_launch<int32_t, 4>(table, V, D, ld_table, rows, n_rows, rows_cap, vals, ld_vals,
                                       adam, o, m, v, dev_err, st)
            : apply_launch<int32_t, 1>(table, V, D, ld_table, rows, n_rows, rows_cap, vals, ld_vals,
                                       adam, o, m, v, dev_err, st);
  return launch_status(e);
}

}  // namespace lmz
