/*
 * lmzipf.h — C ABI of the Zipf gradient-compression hot path of
 * "Language Modeling at Scale" (Patwary et al., arXiv:1810.10045), built
 * for AMD Instinct MI355X (gfx950).
 *
 * The paper's uniqueness method (Sec. III-A, the seven-step list and Fig. 4)
 * replaces an AllGather of K x D embedding gradients with:
 *   step 1   Unique      — the distinct word indices of a batch (J -> J^),
 *   step 2   Seg-Sum     — the local reduction of gradient rows that share a
 *                          word (Delta, K x D -> Delta^, U x D),
 *   step 4   Unique      — the same operation over the G*K gathered indices
 *                          (I -> I^), plus the map J^ -> I^ (lm_map_ids),
 *   step 5   Fill-Values — expansion of Delta^ into a zero-filled U_g x D
 *                          matrix M (lm_fill_values, LM_FILL_EXPAND),
 *   step 7   update      — the conflict-free in-place update of the rows of
 *                          the embedding matrix E named by I^
 *                          (lm_sparse_apply).
 * Steps 3 and 6 are collectives and are not part of this library.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every pointer named as a device buffer is device memory (hipMalloc or a
 *   torch CUDA tensor); host pointers are never accepted for those.
 * - The caller owns every buffer. The library allocates nothing and keeps
 *   no pointer past the call. Its only global state is a per-process call
 *   counter (lm_segsum's flag tags) and the lm_segsum_set_two_launches
 *   setting. All work is enqueued on `stream` (a hipStream_t; NULL is the
 *   default stream) and the call returns without synchronising.
 * - Counts that the GPU computes (num_unique, n_src, ...) stay on the device.
 *   Grids are sized from the host-side capacities (K, u_cap, ...), and the
 *   kernels stop at the device-side count, so no call syncs the host.
 * - Rows are contiguous in memory; `ld_*` is the distance between row starts
 *   in elements and must be >= D.
 * - Host-detectable argument errors (NULL or negative arguments, ld < D, a
 *   workspace that is too small, an unknown enum value) are reported by the
 *   return code before anything is enqueued and nothing is written.
 * - Data-dependent errors are reported by OR-ing LM_DEVERR_* bits into
 *   `*dev_err` (a device int32 that the caller zeroes); the outputs of that
 *   call are then unspecified, but every kernel still only touches memory
 *   inside the buffers it was given.
 * - Concurrent calls that share a workspace or an output buffer race.
 */
#ifndef LMZIPF_H
#define LMZIPF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
enum {
  LM_OK = 0,
  LM_E_INVAL = 1,       /* a NULL, negative or inconsistent argument */
  LM_E_WORKSPACE = 3,   /* ws_bytes below the size the *_workspace_bytes query returns */
  LM_E_HIP = 4,         /* a HIP launch or runtime call failed */
  LM_E_UNSUPPORTED = 5  /* an enum value or a size the library does not handle */
};

/* Bits OR-ed into *dev_err by the kernels. */
enum {
  LM_DEVERR_ID_RANGE = 1,   /* an id outside [0, V) (or outside the dense table) */
  LM_DEVERR_NOT_FOUND = 2,  /* a source id that the destination id list lacks */
  LM_DEVERR_CAPACITY = 4,   /* a device-side count above its buffer's capacity */
  LM_DEVERR_SPIN = 8,       /* a bounded inter-workgroup wait gave up */
  LM_DEVERR_NONFINITE = 16  /* a compressed (binary16) value is infinite or NaN */
};

/* Index dtypes: word indices are int32 or int64; every position, count and
 * row index the library produces is int32 (K < 2^30). */
enum { LM_I32 = 0, LM_I64 = 1 };

/* Gradient dtypes: fp32, or bf16 (accumulated in fp32). */
enum { LM_F32 = 0, LM_BF16 = 1 };

/* Fill-Values modes. */
enum {
  LM_FILL_EXPAND = 0,      /* dst = 0 except dst[map(src_ids[u])] = src[u]        */
  LM_FILL_SCATTER = 1,     /* dst[row(src_ids[u])]  = src[u], other rows untouched */
  LM_FILL_SCATTER_ADD = 2  /* dst[row(src_ids[u])] += src[u], other rows untouched */
};

/* Optimizers for the step-7 update. */
enum { LM_OPT_SGD = 0, LM_OPT_ADAM = 1 };

/* Largest K (tokens per call) the library accepts. */
#define LM_MAX_K ((int64_t)1 << 30)

/* Human-readable name of a return code. Never NULL. */
const char* lm_status_string(int status);

/* ABI version of this header (major * 100 + minor). */
int lm_abi_version(void);

/* Zero `bytes` bytes of a device workspace on `stream` with a fill kernel
 * (safe inside a captured HIP graph). */
int lm_workspace_clear(void* ws, size_t bytes, void* stream);

/* ------------------------------------------------------------------------
 * Unique — Sec. III-A steps 1 and 4: the distinct word indices of a batch,
 * kept in a total order (here: ascending), with the maps from tokens to
 * types.
 *
 * ids        device, K word indices of dtype `idtype` (LM_I32 / LM_I64),
 *            each expected in [0, V). An id outside that range sets
 *            LM_DEVERR_ID_RANGE.
 * K          number of tokens, 0 <= K < LM_MAX_K. K == 0 is valid: it
 *            writes num_unique = 0 and offsets[0] = 0.
 * V          vocabulary size, >= 1. Only ceil(log2 V) key bits are sorted.
 * Outputs (all device; capacities in elements, with C = min(K, V)):
 * uniq       [C] of `idtype`: the U distinct ids in ascending order (J^).
 * counts     [C] int32: counts[u] = number of tokens whose id is uniq[u].
 * offsets    [C+1] int32: exclusive prefix sum of counts; offsets[U] = K.
 * inverse    [K] int32: uniq[inverse[k]] == ids[k] (the map J -> J^).
 * perm       [K] int32: the stable sort permutation: ids[perm[i]] is
 *            non-decreasing and equal ids keep ascending k, so
 *            perm[offsets[u] .. offsets[u+1]) lists the tokens of uniq[u].
 * num_unique [1] int64: U.
 * dev_err    [1] int32, zeroed by the caller.
 * ws         device workspace of at least lm_unique_workspace_bytes(K,
 *            idtype, V) bytes, 256-byte aligned; no initial contents are
 *            required (the first kernel clears what the call needs).
 * ------------------------------------------------------------------------ */
size_t lm_unique_workspace_bytes(int64_t K, int32_t idtype, int64_t V);
int lm_unique(const void* ids, int32_t idtype, int64_t K, int64_t V,
              void* uniq, int32_t* counts, int32_t* offsets, int32_t* inverse,
              int32_t* perm, int64_t* num_unique, int32_t* dev_err,
              void* ws, size_t ws_bytes, void* stream);

/* lm_unique_noalloc — for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): lm_unique with the same arguments, outputs and errors, but
 * with its workspace in a 12 MiB device array of the library instead of a
 * caller's buffer. The call allocates nothing (no hipMalloc, no allocating
 * library routine). Each GPU the library runs on holds its own array from
 * module load until the process ends; its address is looked up on the first
 * call on a device (the current device, which must be the stream's).
 * K > LM_UNIQUE_NOALLOC_MAX_K returns LM_E_UNSUPPORTED before anything is
 * enqueued. The array needs no initial contents (the call's first kernel
 * clears what it uses), but every call on one GPU shares it: calls that
 * overlap on one GPU (other streams, other host threads) race, so order
 * them on one stream or use lm_unique with a workspace each. */
#define LM_UNIQUE_NOALLOC_MAX_K ((int64_t)262144)
int lm_unique_noalloc(const void* ids, int32_t idtype, int64_t K, int64_t V,
                      void* uniq, int32_t* counts, int32_t* offsets, int32_t* inverse,
                      int32_t* perm, int64_t* num_unique, int32_t* dev_err, void* stream);

/* ------------------------------------------------------------------------
 * Seg-Sum — Sec. III-A step 2 (and Sec. II-A: several rows of Delta map to
 * one row of E, so the reverse map is an accumulation):
 *     out[u, :] = sum over i in [offsets[u], offsets[u+1]) of grad[perm[i], :]
 * for u < U = *num_unique, accumulated in fp32 in a fixed order, so repeated
 * calls give bit-identical results. The order depends on K, D, u_cap (the
 * walk's chunks are sized from min(K, u_cap)), the launch form and the
 * number of compute units `stream` may use (the chunks are also sized to
 * fill whole rounds of the waves that fit there: all of the device's, or
 * those of a stream created with hipExtStreamCreateWithCUMask), not on the
 * values.
 *
 * grad       device, K rows of D values of dtype `gtype` (LM_F32 / LM_BF16),
 *            row stride ld_grad elements.
 * perm, inverse, offsets, num_unique
 *            device, as produced by lm_unique for the same ids: perm [K],
 *            inverse [K] (inverse[perm[i]] is the type of sorted position
 *            i), offsets [U+1]. Inconsistent arrays set LM_DEVERR_CAPACITY;
 *            the kernels still stay inside the buffers.
 * u_cap      rows allocated in `out`; U > u_cap sets LM_DEVERR_CAPACITY
 *            and only the first u_cap rows are written.
 * out        device, u_cap x D fp32, row stride ld_out; rows >= U untouched.
 * dev_err    device int32, zeroed by the caller.
 * ws         device workspace of lm_segsum_workspace_bytes(K, D) bytes,
 *            256-byte aligned; no initial contents are required.
 *
 * With D <= 4096 on the 16-byte vector path, the segments that span the
 * walk's chunks are summed by workgroups of the same launch, which wait for
 * per-chunk flags tagged with a per-call value from a process-wide counter
 * (bounded waits; LM_DEVERR_SPIN if one gave up, which a correct call never
 * does). Otherwise, always while `stream` is being captured into a graph (a
 * replay would repeat the tag), and while lm_segsum_set_two_launches is on,
 * they are summed by a second launch.
 * ------------------------------------------------------------------------ */
size_t lm_segsum_workspace_bytes(int64_t K, int64_t D);

int lm_segsum(const void* grad, int32_t gtype, int64_t K, int64_t D,
              int64_t ld_grad, const int32_t* perm, const int32_t* inverse,
              const int32_t* offsets, const int64_t* num_unique, int64_t u_cap,
              float* out, int64_t ld_out, int32_t* dev_err, void* ws,
              size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Seg-Sum into chosen rows — Sec. III-A steps 2 and 5 in one pass on one
 * GPU: the same sums as lm_segsum, but type u's row goes to row row_ids[u]
 * of `out` instead of row u:
 *     out[row_ids[u], :] = sum over i in [offsets[u], offsets[u+1]) of
 *                          grad[perm[i], :]          for u < *num_unique,
 * with the same fixed summation order (so bit-identical to lm_segsum with
 * u_cap = rows_cap, in the same launch form on a stream with the same
 * compute units, followed by a row copy). With
 * row_ids = uniq from lm_unique and `out` a
 * dense V x D table, this is Seg-Sum followed by Fill-Values SCATTER
 * (lm_fill_values, LM_FILL_SCATTER, dst_ids NULL) without writing and
 * re-reading the U x D intermediate; rows of `out` that no type names are
 * left untouched.
 *
 * row_ids    device, rows_cap ids of dtype `idtype`, the first *num_unique
 *            used; they must be distinct (lm_unique's uniq are). An id
 *            outside [0, out_rows) sets LM_DEVERR_ID_RANGE and that type is
 *            not written. *num_unique > rows_cap sets LM_DEVERR_CAPACITY and
 *            only the first rows_cap types are written.
 * out        device, out_rows x D fp32 (out_rows < 2^31), row stride ld_out.
 * The other arguments, the workspace (lm_segsum_workspace_bytes(K, D)) and
 * the launch forms are those of lm_segsum.
 * ------------------------------------------------------------------------ */
int lm_segsum_rows(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                   const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                   const int64_t* num_unique, const void* row_ids, int32_t idtype,
                   int64_t rows_cap, float* out, int64_t out_rows, int64_t ld_out,
                   int32_t* dev_err, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Seg-Sum with the SGD update — Sec. III-A steps 2 and 7 in one pass on one
 * GPU (where the exchange of steps 3 to 6 leaves the reduced rows as they
 * are): the same sums as lm_segsum, applied to the rows of the table that
 * row_ids names instead of written out:
 *     table[row_ids[u], :] -= lr * (sum over i in [offsets[u], offsets[u+1])
 *                                   of grad[perm[i], :])   for u < *num_unique,
 * bit-identical to lm_segsum (u_cap = rows_cap, the same launch form, on a
 * stream with the same compute units) followed by lm_sparse_apply with
 * LM_OPT_SGD and the same lr, without writing and re-reading the U x D
 * intermediate. Rows that no type names are left untouched.
 *
 * row_ids    device, rows_cap distinct ids of dtype `idtype` (lm_unique's
 *            uniq), the first *num_unique used. An id outside [0, V) sets
 *            LM_DEVERR_ID_RANGE and that row is not updated;
 *            *num_unique > rows_cap sets LM_DEVERR_CAPACITY and only the
 *            first rows_cap types are applied.
 * table      device, V x D fp32 (V < 2^31), row stride ld_table, updated in
 *            place.
 * The other arguments, the workspace (lm_segsum_workspace_bytes(K, D)) and
 * the launch forms are those of lm_segsum.
 * ------------------------------------------------------------------------ */
int lm_segsum_sgd(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                  const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                  const int64_t* num_unique, const void* row_ids, int32_t idtype,
                  int64_t rows_cap, float* table, int64_t V, int64_t ld_table, float lr,
                  int32_t* dev_err, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Seg-Sum with the lazy-Adam update — Sec. III-A steps 2 and 7 in one pass
 * on one GPU: the step of lm_sparse_apply with LM_OPT_ADAM on the rows
 * row_ids names, with type u's sum as the gradient of row row_ids[u]:
 *     g = sum over i in [offsets[u], offsets[u+1]) of grad[perm[i], :]
 *     m = beta1 m + (1 - beta1) g,  v = beta2 v + (1 - beta2) g^2,
 *     E -= lr (m / (1 - beta1^step) / (sqrt(v / (1 - beta2^step)) + eps)
 *              + weight_decay E),
 * on E = table[row_ids[u], :] and the m and v rows of the same index,
 * bit-identical to lm_segsum (u_cap = rows_cap, the same launch form, on a
 * stream with the same compute units) followed by lm_sparse_apply with
 * LM_OPT_ADAM and the same arguments, without the U x D intermediate. Rows
 * that no type names are left untouched in all three arrays.
 *
 * m, v       device, V x D fp32 with the table's row stride, updated in
 *            place.
 * step       >= 1 (the bias corrections); beta1, beta2 in [0, 1).
 * The other arguments and their errors are those of lm_segsum_sgd.
 * ------------------------------------------------------------------------ */
int lm_segsum_adam(const void* grad, int32_t gtype, int64_t K, int64_t D, int64_t ld_grad,
                   const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
                   const int64_t* num_unique, const void* row_ids, int32_t idtype,
                   int64_t rows_cap, float* table, int64_t V, int64_t ld_table, float lr,
                   float beta1, float beta2, float eps, float weight_decay, int64_t step,
                   float* m, float* v, int32_t* dev_err, void* ws, size_t ws_bytes,
                   void* stream);

/* The one-launch form of lm_segsum (and lm_segsum_rows, lm_segsum_sgd,
 * lm_segsum_adam) relies on the hardware starting the walk's workgroups
 * before the fix-up workgroups that wait on them (they come first in the
 * grid). lm_segsum_set_two_launches(1)
 * makes every later call in the process use the two-launch form instead
 * (the walk, then a separate fix-up kernel: no workgroup ever waits on
 * another), the fallback should a
 * device break that order; 0 restores the default. The environment variable
 * LMZIPF_SEGSUM_TWO_LAUNCHES=1, read at the first lm_segsum call, sets it
 * too. Results agree with the one-launch form within the Seg-Sum tolerance
 * (the heads' partial rows are added in a different grouping) and are
 * bit-identical from run to run. Process-wide; returns the previous
 * setting (0 or 1). */
int lm_segsum_set_two_launches(int32_t enable);

/* ------------------------------------------------------------------------
 * Map — Sec. III-A step 4: the local-to-global map J^ -> I^. Both id lists
 * are strictly ascending (outputs of lm_unique):
 *     map[u] = the position of sub_ids[u] in sup_ids,  u < *n_sub.
 * An id of sub_ids absent from sup_ids sets LM_DEVERR_NOT_FOUND (map[u] is
 * then -1).
 *
 * sub_ids    device, *n_sub ids (capacity sub_cap) of dtype `idtype`.
 * sup_ids    device, *n_sup ids (capacity sup_cap) of the same dtype.
 * n_sub, n_sup  device int64 counts; a count above its capacity sets
 *            LM_DEVERR_CAPACITY and is clamped to it.
 * map        device, sub_cap int32.
 * ------------------------------------------------------------------------ */
int lm_map_ids(const void* sub_ids, const int64_t* n_sub, int64_t sub_cap,
               const void* sup_ids, const int64_t* n_sup, int64_t sup_cap,
               int32_t idtype, int32_t* map, int32_t* dev_err, void* stream);

/* ------------------------------------------------------------------------
 * Fill-Values — Sec. III-A step 5: move reduced rows into the row space of
 * another id list.
 *   LM_FILL_EXPAND       dst has *n_dst rows, one per dst_ids entry; row r
 *                        becomes src[u] where src_ids[u] == dst_ids[r], and
 *                        zero where no src id equals dst_ids[r] (rows of
 *                        words this batch lacks are zero). Every row
 *                        < *n_dst is written exactly once.
 *   LM_FILL_SCATTER      dst[row] = src[u],  row = position of src_ids[u] in
 *   LM_FILL_SCATTER_ADD  dst[row] += src[u]  dst_ids, or row = src_ids[u]
 *                        itself when dst_ids is NULL (a dense V x D table);
 *                        rows that no src id names are left untouched.
 * src_ids must be strictly ascending and dst_ids (when given) strictly
 * ascending, as lm_unique produces them; then no two source rows reach the
 * same destination row and no atomics are needed (Sec. III-A, last
 * paragraph: unique indices leave no write conflicts).
 *
 * src        device, src_cap x D fp32, row stride ld_src.
 * src_ids    device, at least src_cap ids of dtype `idtype`; the first
 *            *n_src are used.
 * n_src      device int64 (<= src_cap).
 * dst_ids    device, at least dst_rows ids of dtype `idtype`, the first
 *            *n_dst used, or NULL (SCATTER modes only: row = id, which must
 *            be < dst_rows).
 * n_dst      device int64 (<= dst_rows); ignored when dst_ids is NULL.
 * dst        device, dst_rows x D fp32, row stride ld_dst.
 * A source id missing from dst_ids sets LM_DEVERR_NOT_FOUND; an id
 * outside [0, dst_rows) with dst_ids NULL sets LM_DEVERR_ID_RANGE.
 * ------------------------------------------------------------------------ */
int lm_fill_values(const float* src, int64_t ld_src, const void* src_ids,
                   const int64_t* n_src, int64_t src_cap, const void* dst_ids,
                   const int64_t* n_dst, int32_t idtype, int64_t D, float* dst,
                   int64_t dst_rows, int64_t ld_dst, int32_t mode,
                   int32_t* dev_err, void* stream);

/* ------------------------------------------------------------------------
 * Sparse apply — Sec. III-A step 7: update the rows of the embedding
 * matrix E named by the (unique) ids with the reduced gradients, in place.
 * The ids are distinct, so every row is owned by one workgroup: no locks and
 * no atomics (the serialisation on frequent words that the paper removes).
 *   LM_OPT_SGD   E[id] -= lr * g
 *   LM_OPT_ADAM  lazy Adam on the touched rows only, with bias correction
 *                at step `step` (>= 1) and decoupled weight decay:
 *                  m = beta1*m + (1-beta1)*g
 *                  v = beta2*v + (1-beta2)*g*g
 *                  E[id] -= lr * ( (m/(1-beta1^step)) /
 *                                  (sqrt(v/(1-beta2^step)) + eps)
 *                                  + weight_decay * E[id] )
 * table      device, V x D fp32, row stride ld_table; updated in place.
 * rows       device, *n_rows strictly ascending ids of dtype `idtype`.
 * n_rows     device int64 (<= rows_cap).
 * vals       device, rows_cap x D fp32 gradients, row stride ld_vals.
 * m, v       device, V x D fp32 Adam moments (row stride ld_table), or NULL
 *            for SGD.
 * An id outside [0, V) sets LM_DEVERR_ID_RANGE and that row is skipped.
 * ------------------------------------------------------------------------ */
int lm_sparse_apply(float* table, int64_t V, int64_t D, int64_t ld_table,
                    const void* rows, int32_t idtype, const int64_t* n_rows,
                    int64_t rows_cap, const float* vals, int64_t ld_vals,
                    int32_t opt, float lr, float beta1, float beta2, float eps,
                    float weight_decay, int64_t step, float* m, float* v,
                    int32_t* dev_err, void* stream);

/* ------------------------------------------------------------------------
 * Compressed payload — Sec. III-C (lower precision): the U_g x D matrix the
 * GPUs all-reduce in step 6 travels as IEEE binary16 after a multiplication
 * by a compression scale F, and is multiplied by 1/F after the up-cast at the
 * receiving end. These two entry points are the two ends, fused into the
 * steps that write and read the payload (the collective itself is not part
 * of this library). A power-of-two F makes both scalings exact.
 *
 * lm_fill_values_f16: as lm_fill_values, but dst is binary16 and each value
 * written is binary16(fp32(src * scale)) (round to nearest even; EXPAND's
 * zero rows are +0). Modes LM_FILL_EXPAND and LM_FILL_SCATTER;
 * LM_FILL_SCATTER_ADD returns LM_E_UNSUPPORTED.
 * dst        device, dst_rows x D binary16 (uint16 bit patterns), row
 *            stride ld_dst (in elements).
 * scale      the compression scale F (finite, nonzero).
 * A written value that is infinite or NaN (|src * scale| rounds above
 * 65504, the binary16 maximum) sets LM_DEVERR_NONFINITE, the signal a
 * caller uses to lower F; the value is still written.
 * ------------------------------------------------------------------------ */
int lm_fill_values_f16(const float* src, int64_t ld_src, const void* src_ids,
                       const int64_t* n_src, int64_t src_cap, const void* dst_ids,
                       const int64_t* n_dst, int32_t idtype, int64_t D, uint16_t* dst,
                       int64_t dst_rows, int64_t ld_dst, int32_t mode, float scale,
                       int32_t* dev_err, void* stream);

/* lm_sparse_apply_f16: as lm_sparse_apply, but vals is the binary16 payload
 * (rows_cap x D uint16 bit patterns, row stride ld_vals) and each gradient
 * value is fp32(vals) * inv_scale (inv_scale = 1/F; finite, nonzero). */
int lm_sparse_apply_f16(float* table, int64_t V, int64_t D, int64_t ld_table,
                        const void* rows, int32_t idtype, const int64_t* n_rows,
                        int64_t rows_cap, const uint16_t* vals, int64_t ld_vals,
                        float inv_scale, int32_t opt, float lr, float beta1, float beta2,
                        float eps, float weight_decay, int64_t step, float* m, float* v,
                        int32_t* dev_err, void* stream);

/* ------------------------------------------------------------------------
 * Candidate sampler — Sec. II-A (sampled softmax) and Sec. III-B
 * (controlled randomness): the output embedding is updated at a random,
 * uniformly drawn subset of the vocabulary plus the batch's own words.
 * Groups of GPUs share a seed so that their subsets coincide; the random
 * words are drawn by the caller from its group's seed and passed in.
 *   ids[i] = floor(r[i] * V / 2^64)   (the high word of the product)
 * r          device, n uint64 random words.
 * V          vocabulary size (>= 1; <= 2^31 for int32 ids).
 * ids        device, n ids of dtype `idtype`, written.
 * ------------------------------------------------------------------------ */
int lm_sample_ids(const uint64_t* r, int64_t n, int64_t V, void* ids, int32_t idtype,
                  void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LMZIPF_H */
