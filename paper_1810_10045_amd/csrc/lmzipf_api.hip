// The C ABI declared in include/lmzipf.h: argument validation (before any
// launch), dtype dispatch and stream plumbing. The kernels live in
// unique.hip, segsum.hip and fill.hip.
#include "common.hpp"

namespace lmz {

size_t unique_workspace_bytes(int64_t K, int idtype, int64_t V);
int unique_run(const void* ids, int idtype, int64_t K, int64_t V, void* uniq, int32_t* counts,
               int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
               int32_t* dev_err, void* ws, size_t ws_bytes, hipStream_t st);
size_t segsum_workspace_bytes(int64_t K, int64_t D);
int segsum_run(const void* grad, int gtype, int64_t K, int64_t D, int64_t ld_grad,
               const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
               const int64_t* num_unique, int64_t u_cap, float* out, int64_t ld_out,
               int32_t* dev_err, void* ws, size_t ws_bytes, hipStream_t st,
               const void* row_ids = nullptr, int row_ids64 = 0, int64_t out_rows = 0,
               int op = 0, const OptParams& opt = OptParams{}, float* m = nullptr,
               float* v = nullptr);
int map_run(const void* sub, const int64_t* n_sub, int64_t sub_cap, const void* sup,
            const int64_t* n_sup, int64_t sup_cap, int idtype, int32_t* map, int32_t* dev_err,
            hipStream_t st);
int fill_run(const float* src, int64_t ld_src, const void* src_ids, const int64_t* n_src,
             int64_t src_cap, const void* dst_ids, const int64_t* n_dst, int idtype, int64_t D,
             float* dst, int64_t dst_rows, int64_t ld_dst, int mode, int32_t* dev_err,
             hipStream_t st);
int apply_run(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows, int idtype,
              const int64_t* n_rows, int64_t rows_cap, const float* vals, int64_t ld_vals,
              int opt, float lr, float beta1, float beta2, float eps, float weight_decay,
              int64_t step, float* m, float* v, int32_t* dev_err, hipStream_t st);

int fill_run_f16(const float* src, int64_t ld_src, const void* src_ids, const int64_t* n_src,
                 int64_t src_cap, const void* dst_ids, const int64_t* n_dst, int idtype,
                 int64_t D, uint16_t* dst, int64_t dst_rows, int64_t ld_dst, int mode,
                 float scale, int32_t* dev_err, hipStream_t st);
int apply_run_f16(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows,
                  int idtype, const int64_t* n_rows, int64_t rows_cap, const uint16_t* vals,
                  int64_t ld_vals, float inv_scale, int opt, float lr, float beta1, float beta2,
                  float eps, float weight_decay, int64_t step, float* m, float* v,
                  int32_t* dev_err, hipStream_t st);

int sample_run(const uint64_t* r, int64_t n, int64_t V, void* ids, int idtype, hipStream_t st);
void segsum_force_wait_failure(bool enable, uint32_t limit);
int segsum_set_two_launches(bool enable);
void unique_force_wait_failure(bool enable, uint32_t limit);

int launch_status(hipError_t e) { return e == hipSuccess ? LM_OK : LM_E_HIP; }

static bool finite_nonzero(float x) { return x == x && x != 0.f && x - x == 0.f; }

__global__ __launch_bounds__(256) void k_clear(uint32_t* p, int64_t words, uint8_t* tail,
                                               int tail_bytes) {
  for (int64_t i = blockIdx.x * int64_t(256) + threadIdx.x; i < words;
       i += int64_t(gridDim.x) * 256)
    p[i] = 0u;
  if (blockIdx.x == 0 && static_cast<int>(threadIdx.x) < tail_bytes) tail[threadIdx.x] = 0;
}

static bool valid_idtype(int32_t t) { return t == LM_I32 || t == LM_I64; }

}  // namespace lmz

using namespace lmz;

extern "C" {

const char* lm_status_string(int status) {
  switch (status) {
    case LM_OK: return "LM_OK";
    case LM_E_INVAL: return "LM_E_INVAL: invalid argument";
    case LM_E_WORKSPACE: return "LM_E_WORKSPACE: workspace too small";
    case LM_E_HIP: return "LM_E_HIP: HIP launch or runtime error";
    case LM_E_UNSUPPORTED: return "LM_E_UNSUPPORTED: unsupported dtype, mode or size";
    default: return "unknown lmzipf status";
  }
}

int lm_abi_version(void) { return 106; }

int lm_workspace_clear(void* ws, size_t bytes, void* stream) {
  if (bytes == 0) return LM_OK;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 3)) return LM_E_INVAL;
  const int64_t words = static_cast<int64_t>(bytes / 4);
  const int tail = static_cast<int>(bytes % 4);
  int64_t blocks = (words + 256 * 16 - 1) / (256 * 16);
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  k_clear<<<static_cast<uint32_t>(blocks), 256, 0, static_cast<hipStream_t>(stream)>>>(
      static_cast<uint32_t*>(ws), words, static_cast<uint8_t*>(ws) + words * 4, tail);
  return launch_status(hipGetLastError());
}

size_t lm_unique_workspace_bytes(int64_t K, int32_t idtype, int64_t V) {
  if (K < 0 || K >= LM_MAX_K || V < 1 || !valid_idtype(idtype)) return 0;
  return unique_workspace_bytes(K, idtype, V);
}

int lm_unique(const void* ids, int32_t idtype, int64_t K, int64_t V, void* uniq, int32_t* counts,
              int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
              int32_t* dev_err, void* ws, size_t ws_bytes, void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (K < 0 || V < 1) return LM_E_INVAL;
  if (K >= LM_MAX_K) return LM_E_UNSUPPORTED;
  if (!offsets || !num_unique || !ws) return LM_E_INVAL;
  if (K > 0 && (!ids || !uniq || !counts || !inverse || !perm || !dev_err)) return LM_E_INVAL;
  if (reinterpret_cast<uintptr_t>(ws) & 255) return LM_E_INVAL;
  if (ws_bytes < unique_workspace_bytes(K, idtype, V)) return LM_E_WORKSPACE;
  return unique_run(ids, idtype, K, V, uniq, counts, offsets, inverse, perm, num_unique, dev_err,
                    ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int lm_segsum_set_two_launches(int32_t enable) { return segsum_set_two_launches(enable != 0); }

int lm_test_force_wait_failure(int32_t enable, uint32_t spin_limit) {
  segsum_force_wait_failure(enable != 0, spin_limit);
  unique_force_wait_failure(enable != 0, spin_limit);
  return LM_OK;
}

size_t lm_segsum_workspace_bytes(int64_t K, int64_t D) {
  if (K < 0 || K >= LM_MAX_K || D < 0) return 0;
  return segsum_workspace_bytes(K, D);
}

int lm_segsum(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
              const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
              const int64_t* num_unique, int64_t u_cap, float* out, int64_t ld_out,
              int32_t* dev_err, void* ws, size_t ws_bytes, void* stream) {
  if (gtype != LM_F32 && gtype != LM_BF16) return LM_E_UNSUPPORTED;
  if (K < 0 || D < 0 || u_cap < 0 || ld_grad < D || ld_out < D) return LM_E_INVAL;
  if (K >= LM_MAX_K || D > (int64_t(1) << 24)) return LM_E_UNSUPPORTED;
  if (K > 0 && D > 0 && u_cap > 0 &&
      (!grad || !perm || !inverse || !offsets || !num_unique || !out || !dev_err || !ws))
    return LM_E_INVAL;
  if (ws && (reinterpret_cast<uintptr_t>(ws) & 255)) return LM_E_INVAL;
  if (ws_bytes < segsum_workspace_bytes(K, D)) return LM_E_WORKSPACE;
  return segsum_run(grad, gtype, K, D, ld_grad, perm, inverse, offsets, num_unique, u_cap, out,
                    ld_out, dev_err, ws, ws_bytes, static_cast<hipStream_t>(stream));
}

int lm_segsum_rows(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                   const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                   const int64_t* num_unique, const void* row_ids, int32_t idtype,
                   int64_t rows_cap, float* out, int64_t out_rows, int64_t ld_out,
                   int32_t* dev_err, void* ws, size_t ws_bytes, void* stream) {
  if (gtype != LM_F32 && gtype != LM_BF16) return LM_E_UNSUPPORTED;
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (K < 0 || D < 0 || rows_cap < 0 || out_rows < 0 || ld_grad < D || ld_out < D)
    return LM_E_INVAL;
  if (K >= LM_MAX_K || D > (int64_t(1) << 24) || out_rows > INT32_MAX) return LM_E_UNSUPPORTED;
  if (K > 0 && D > 0 && rows_cap > 0 &&
      (!grad || !perm || !inverse || !offsets || !num_unique || !row_ids || !out || !dev_err ||
       !ws))
    return LM_E_INVAL;
  if (ws && (reinterpret_cast<uintptr_t>(ws) & 255)) return LM_E_INVAL;
  if (ws_bytes < segsum_workspace_bytes(K, D)) return LM_E_WORKSPACE;
  return segsum_run(grad, gtype, K, D, ld_grad, perm, inverse, offsets, num_unique, rows_cap,
                    out, ld_out, dev_err, ws, ws_bytes, static_cast<hipStream_t>(stream),
                    row_ids, idtype == LM_I64 ? 1 : 0, out_rows);
}

int lm_segsum_sgd(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                  const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                  const int64_t* num_unique, const void* row_ids, int32_t idtype,
                  int64_t rows_cap, float* table, int64_t V, int64_t ld_table, float lr,
                  int32_t* dev_err, void* ws, size_t ws_bytes, void* stream) {
  if (gtype != LM_F32 && gtype != LM_BF16) return LM_E_UNSUPPORTED;
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (K < 0 || D < 0 || rows_cap < 0 || V < 0 || ld_grad < D || ld_table < D) return LM_E_INVAL;
  if (K >= LM_MAX_K || D > (int64_t(1) << 24) || V > INT32_MAX) return LM_E_UNSUPPORTED;
  if (K > 0 && D > 0 && rows_cap > 0 &&
      (!grad || !perm || !inverse || !offsets || !num_unique || !row_ids || !table || !dev_err ||
       !ws))
    return LM_E_INVAL;
  if (ws && (reinterpret_cast<uintptr_t>(ws) & 255)) return LM_E_INVAL;
  if (ws_bytes < segsum_workspace_bytes(K, D)) return LM_E_WORKSPACE;
  return segsum_run(grad, gtype, K, D, ld_grad, perm, inverse, offsets, num_unique, rows_cap,
                    table, ld_table, dev_err, ws, ws_bytes, static_cast<hipStream_t>(stream),
                    row_ids, idtype == LM_I64 ? 1 : 0, V, 1,
                    make_opt_params(false, lr, 0.f, 0.f, 0.f, 0.f, 1, 1.f));
}

int lm_segsum_adam(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                   const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                   const int64_t* num_unique, const void* row_ids, int32_t idtype,
                   int64_t rows_cap, float* table, int64_t V, int64_t ld_table, float lr,
                   float beta1, float beta2, float eps, float weight_decay, int64_t step,
                   float* m, float* v, int32_t* dev_err, void* ws, size_t ws_bytes,
                   void* stream) {
  if (gtype != LM_F32 && gtype != LM_BF16) return LM_E_UNSUPPORTED;
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (K < 0 || D < 0 || rows_cap < 0 || V < 0 || ld_grad < D || ld_table < D) return LM_E_INVAL;
  if (K >= LM_MAX_K || D > (int64_t(1) << 24) || V > INT32_MAX) return LM_E_UNSUPPORTED;
  if (step < 1 || !(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f)) return LM_E_INVAL;
  if (K > 0 && D > 0 && rows_cap > 0 &&
      (!grad || !perm || !inverse || !offsets || !num_unique || !row_ids || !table || !m || !v ||
       !dev_err || !ws))
    return LM_E_INVAL;
  if (ws && (reinterpret_cast<uintptr_t>(ws) & 255)) return LM_E_INVAL;
  if (ws_bytes < segsum_workspace_bytes(K, D)) return LM_E_WORKSPACE;
  return segsum_run(grad, gtype, K, D, ld_grad, perm, inverse, offsets, num_unique, rows_cap,
                    table, ld_table, dev_err, ws, ws_bytes, static_cast<hipStream_t>(stream),
                    row_ids, idtype == LM_I64 ? 1 : 0, V, 2,
                    make_opt_params(true, lr, beta1, beta2, eps, weight_decay, step, 1.f), m, v);
}

int lm_map_ids(const void* sub_ids, const int64_t* n_sub, int64_t sub_cap, const void* sup_ids,
               const int64_t* n_sup, int64_t sup_cap, int32_t idtype, int32_t* map,
               int32_t* dev_err, void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (sub_cap < 0 || sup_cap < 0) return LM_E_INVAL;
  if (sub_cap > 0 && (!sub_ids || !n_sub || !sup_ids || !n_sup || !map || !dev_err))
    return LM_E_INVAL;
  if (sub_cap >= (int64_t(1) << 31) * kWave) return LM_E_UNSUPPORTED;
  return map_run(sub_ids, n_sub, sub_cap, sup_ids, n_sup, sup_cap, idtype, map, dev_err,
                 static_cast<hipStream_t>(stream));
}

int lm_fill_values(const float* src, int64_t ld_src, const void* src_ids, const int64_t* n_src,
                   int64_t src_cap, const void* dst_ids, const int64_t* n_dst, int32_t idtype,
                   int64_t D, float* dst, int64_t dst_rows, int64_t ld_dst, int32_t mode,
                   int32_t* dev_err, void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (mode != LM_FILL_EXPAND && mode != LM_FILL_SCATTER && mode != LM_FILL_SCATTER_ADD)
    return LM_E_UNSUPPORTED;
  if (D < 0 || src_cap < 0 || dst_rows < 0 || ld_src < D || ld_dst < D) return LM_E_INVAL;
  if (D > (int64_t(1) << 24)) return LM_E_UNSUPPORTED;
  if (mode == LM_FILL_EXPAND && (!dst_ids || !n_dst)) return LM_E_INVAL;
  if (dst_ids && !n_dst) return LM_E_INVAL;
  if ((src_cap > 0 || dst_rows > 0) && D > 0 && (!src_ids || !n_src || !dev_err)) return LM_E_INVAL;
  if (src_cap > 0 && D > 0 && !src) return LM_E_INVAL;
  if (dst_rows > 0 && D > 0 && !dst) return LM_E_INVAL;
  return fill_run(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, idtype, D, dst, dst_rows,
                  ld_dst, mode, dev_err, static_cast<hipStream_t>(stream));
}

int lm_sparse_apply(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows,
                    int32_t idtype, const int64_t* n_rows, int64_t rows_cap, const float* vals,
                    int64_t ld_vals, int32_t opt, float lr, float beta1, float beta2, float eps,
                    float weight_decay, int64_t step, float* m, float* v, int32_t* dev_err,
                    void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (opt != LM_OPT_SGD && opt != LM_OPT_ADAM) return LM_E_UNSUPPORTED;
  if (V < 0 || D < 0 || rows_cap < 0 || ld_table < D || ld_vals < D) return LM_E_INVAL;
  if (D > (int64_t(1) << 24)) return LM_E_UNSUPPORTED;
  if (rows_cap > 0 && D > 0 && (!table || !rows || !n_rows || !vals || !dev_err))
    return LM_E_INVAL;
  if (opt == LM_OPT_ADAM) {
    if (step < 1) return LM_E_INVAL;
    if (rows_cap > 0 && D > 0 && (!m || !v)) return LM_E_INVAL;
    if (!(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f)) return LM_E_INVAL;
  }
  return apply_run(table, V, D, ld_table, rows, idtype, n_rows, rows_cap, vals, ld_vals, opt, lr,
                   beta1, beta2, eps, weight_decay, step, m, v, dev_err,
                   static_cast<hipStream_t>(stream));
}

int lm_fill_values_f16(const float* src, int64_t ld_src, const void* src_ids,
                       const int64_t* n_src, int64_t src_cap, const void* dst_ids,
                       const int64_t* n_dst, int32_t idtype, int64_t D, uint16_t* dst,
                       int64_t dst_rows, int64_t ld_dst, int32_t mode, float scale,
                       int32_t* dev_err, void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (mode != LM_FILL_EXPAND && mode != LM_FILL_SCATTER) return LM_E_UNSUPPORTED;
  if (!finite_nonzero(scale)) return LM_E_INVAL;
  if (D < 0 || src_cap < 0 || dst_rows < 0 || ld_src < D || ld_dst < D) return LM_E_INVAL;
  if (D > (int64_t(1) << 24)) return LM_E_UNSUPPORTED;
  if (mode == LM_FILL_EXPAND && (!dst_ids || !n_dst)) return LM_E_INVAL;
  if (dst_ids && !n_dst) return LM_E_INVAL;
  if ((src_cap > 0 || dst_rows > 0) && D > 0 && (!src_ids || !n_src || !dev_err)) return LM_E_INVAL;
  if (src_cap > 0 && D > 0 && !src) return LM_E_INVAL;
  if (dst_rows > 0 && D > 0 && !dst) return LM_E_INVAL;
  return fill_run_f16(src, ld_src, src_ids, n_src, src_cap, dst_ids, n_dst, idtype, D, dst,
                      dst_rows, ld_dst, mode, scale, dev_err, static_cast<hipStream_t>(stream));
}

int lm_sparse_apply_f16(float* table, int64_t V, int64_t D, int64_t ld_table, const void* rows,
                        int32_t idtype, const int64_t* n_rows, int64_t rows_cap,
                        const uint16_t* vals, int64_t ld_vals, float inv_scale, int32_t opt,
                        float lr, float beta1, float beta2, float eps, float weight_decay,
                        int64_t step, float* m, float* v, int32_t* dev_err, void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (opt != LM_OPT_SGD && opt != LM_OPT_ADAM) return LM_E_UNSUPPORTED;
  if (!finite_nonzero(inv_scale)) return LM_E_INVAL;
  if (V < 0 || D < 0 || rows_cap < 0 || ld_table < D || ld_vals < D) return LM_E_INVAL;
  if (D > (int64_t(1) << 24)) return LM_E_UNSUPPORTED;
  if (rows_cap > 0 && D > 0 && (!table || !rows || !n_rows || !vals || !dev_err))
    return LM_E_INVAL;
  if (opt == LM_OPT_ADAM) {
    if (step < 1) return LM_E_INVAL;
    if (rows_cap > 0 && D > 0 && (!m || !v)) return LM_E_INVAL;
    if (!(beta1 >= 0.f && beta1 < 1.f && beta2 >= 0.f && beta2 < 1.f)) return LM_E_INVAL;
  }
  return apply_run_f16(table, V, D, ld_table, rows, idtype, n_rows, rows_cap, vals, ld_vals,
                       inv_scale, opt, lr, beta1, beta2, eps, weight_decay, step, m, v, dev_err,
                       static_cast<hipStream_t>(stream));
}

int lm_sample_ids(const uint64_t* r, int64_t n, int64_t V, void* ids, int32_t idtype,
                  void* stream) {
  if (!valid_idtype(idtype)) return LM_E_UNSUPPORTED;
  if (n < 0 || V < 1) return LM_E_INVAL;
  if (idtype == LM_I32 && V > (int64_t(1) << 31)) return LM_E_INVAL;
  if (n > 0 && (!r || !ids)) return LM_E_INVAL;
  return sample_run(r, n, V, ids, idtype, static_cast<hipStream_t>(stream));
}

}  // extern "C"
