/*
 * lmoracle.c — CPU oracle for the Zipf gradient-compression path of
 * "Language Modeling at Scale" (arXiv:1810.10045).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the slow, plainly written reference
 * that the GPU library is checked against. Only the tests, the smoke check
 * and the CPU-baseline leg of the benchmark may load it; the product path
 * never does. It shares no code, header, table or helper with the GPU
 * library.
 *
 * Every routine writes out the definition of one step of the paper's
 * uniqueness method (Sec. III-A) with no blocking, fusion or reordering:
 *   orc_unique          steps 1 and 4   (types of a token list, total order)
 *   orc_segsum          step 2          (local reduction of gradient rows)
 *   orc_segsum_cols     step 2, over a range of columns (one thread's share
 *                                        in the all-core CPU baseline)
 *   orc_segsum_select   step 2, evaluated for a chosen set of word ids only
 *   orc_dense_scatter   Sec. II-A       (the baseline reverse map: every
 *                                        gradient row accumulated into its
 *                                        embedding row, duplicates included)
 *   orc_map             step 4          (the map J^ -> I^)
 *   orc_expand          step 5          (zero-filled expansion to U_g rows)
 *   orc_scatter         step 5/7        (row write / accumulate at an id)
 *   orc_sgd, orc_adam   step 7          (update of the touched rows; the
 *                                        Adam variant follows the char-LM
 *                                        setup of Sec. IV-B)
 * Floating point is fp64 throughout; bf16 inputs are widened exactly.
 * Status: 0 = ok, 2 = an id out of range, 3 = an id not found, 1 = bad args.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORC_OK = 0, ORC_BADARG = 1, ORC_RANGE = 2, ORC_NOTFOUND = 3 };
enum { ORC_F32 = 0, ORC_BF16 = 1 };

/* Value d of row k of a gradient matrix stored as fp32 or as bf16 bits. */
static double grad_at(const void* grad, int gtype, int64_t ld, int64_t k,
                      int64_t d) {
  if (gtype == ORC_F32) return (double)((const float*)grad)[k * ld + d];
  /* bf16 is the upper half of an IEEE binary32: widening is exact. */
  uint32_t bits = (uint32_t)((const uint16_t*)grad)[k * ld + d] << 16;
  float f;
  memcpy(&f, &bits, sizeof f);
  return (double)f;
}

/* A token: its word index and its position in the batch. */
typedef struct {
  int64_t id;
  int64_t k;
} token;

/* Total order on (word index, position): ascending ids, ties by position. */
static int token_cmp(const void* a, const void* b) {
  const token* x = (const token*)a;
  const token* y = (const token*)b;
  if (x->id != y->id) return x->id < y->id ? -1 : 1;
  if (x->k != y->k) return x->k < y->k ? -1 : 1;
  return 0;
}

/*
 * Steps 1 and 4 (Sec. III-A): the "types" of a list of K tokens J, in total
 * (ascending) order, and the map from every token to its type.
 *   uniq[u]     the u-th distinct word index, ascending       (J^ or I^)
 *   counts[u]   how many tokens are uniq[u]
 *   offsets[u]  tokens before type u in sorted order; offsets[U] = K
 *   inverse[k]  u such that uniq[u] == J[k]                  (J -> J^)
 *   perm[i]     the position of the i-th token in (id, position) order
 * Caller capacities: uniq/counts min(K,V) (or K), offsets that plus one,
 * inverse/perm K.
 */
int orc_unique(const int64_t* J, int64_t K, int64_t V, int64_t* uniq,
               int32_t* counts, int32_t* offsets, int32_t* inverse,
               int32_t* perm, int64_t* U_out) {
  if (K < 0 || V < 1 || (K > 0 && !J) || !U_out) return ORC_BADARG;
  for (int64_t k = 0; k < K; ++k)
    if (J[k] < 0 || J[k] >= V) return ORC_RANGE;

  token* t = (token*)malloc((size_t)(K > 0 ? K : 1) * sizeof(token));
  if (!t) return ORC_BADARG;
  for (int64_t k = 0; k < K; ++k) {
    t[k].id = J[k];
    t[k].k = k;
  }
  qsort(t, (size_t)K, sizeof(token), token_cmp);

  int64_t U = 0;
  for (int64_t i = 0; i < K; ++i) {
    if (i == 0 || t[i].id != t[i - 1].id) {
      uniq[U] = t[i].id;
      offsets[U] = (int32_t)i;
      counts[U] = 0;
      ++U;
    }
    counts[U - 1] += 1;
    inverse[t[i].k] = (int32_t)(U - 1);
    perm[i] = (int32_t)t[i].k;
  }
  offsets[U] = (int32_t)K;
  *U_out = U;
  free(t);
  return ORC_OK;
}

/*
 * Step 2 (Sec. III-A), with the accumulation of Sec. II-A: row u of the
 * reduced gradient is the sum of the gradient rows of every token of type u.
 *   out[u][d] = sum over k with inverse[k] == u of grad[k][d]
 * out is U x D fp64 (row stride D), overwritten. Tokens are visited in
 * ascending position.
 */
int orc_segsum(const void* grad, int gtype, int64_t K, int64_t D, int64_t ld,
               const int32_t* inverse, int64_t U, double* out) {
  if (K < 0 || D < 0 || U < 0 || ld < D || (gtype != ORC_F32 && gtype != ORC_BF16))
    return ORC_BADARG;
  memset(out, 0, (size_t)(U * D) * sizeof(double));
  for (int64_t k = 0; k < K; ++k) {
    int64_t u = inverse[k];
    if (u < 0 || u >= U) return ORC_RANGE;
    for (int64_t d = 0; d < D; ++d) out[u * D + d] += grad_at(grad, gtype, ld, k, d);
  }
  return ORC_OK;
}

/*
 * Step 2 over the columns [d0, d1) only: the same sums as orc_segsum, in
 * the same token order, for those columns of out (U x D fp64, row stride D);
 * the other columns are left as they are. Columns of the reduction are
 * independent, so calls on disjoint column ranges share no writes: the
 * all-core CPU baseline runs one such call per thread.
 */
int orc_segsum_cols(const void* grad, int gtype, int64_t K, int64_t D, int64_t ld,
                    const int32_t* inverse, int64_t U, int64_t d0, int64_t d1,
                    double* out) {
  if (K < 0 || D < 0 || U < 0 || ld < D || d0 < 0 || d1 < d0 || d1 > D ||
      (gtype != ORC_F32 && gtype != ORC_BF16))
    return ORC_BADARG;
  for (int64_t u = 0; u < U; ++u)
    for (int64_t d = d0; d < d1; ++d) out[u * D + d] = 0.0;
  for (int64_t k = 0; k < K; ++k) {
    int64_t u = inverse[k];
    if (u < 0 || u >= U) return ORC_RANGE;
    for (int64_t d = d0; d < d1; ++d) out[u * D + d] += grad_at(grad, gtype, ld, k, d);
  }
  return ORC_OK;
}

/*
 * Step 2 for a chosen set of word ids only: out[j][d] is the sum of the
 * gradient rows of the tokens whose word index is sel[j]. sel must be
 * strictly ascending; an id that no token carries gives a zero row. Used to
 * check full-size runs one output row at a time.
 */
int orc_segsum_select(const void* grad, int gtype, int64_t K, int64_t D,
                      int64_t ld, const int64_t* J, const int64_t* sel,
                      int64_t nsel, double* out) {
  if (K < 0 || D < 0 || nsel < 0 || ld < D) return ORC_BADARG;
  for (int64_t j = 1; j < nsel; ++j)
    if (sel[j] <= sel[j - 1]) return ORC_BADARG;
  memset(out, 0, (size_t)(nsel * D) * sizeof(double));
  for (int64_t k = 0; k < K; ++k) {
    int64_t lo = 0, hi = nsel; /* first sel[j] >= J[k] */
    while (lo < hi) {
      int64_t mid = lo + (hi - lo) / 2;
      if (sel[mid] < J[k]) lo = mid + 1; else hi = mid;
    }
    if (lo == nsel || sel[lo] != J[k]) continue;
    for (int64_t d = 0; d < D; ++d) out[lo * D + d] += grad_at(grad, gtype, ld, k, d);
  }
  return ORC_OK;
}

/*
 * The baseline reverse map of Sec. II-A, with no uniqueness at all: every
 * gradient row k is accumulated into row J[k] of a dense V x D matrix
 * (the rows are added one token at a time, as a locked scatter-add would).
 * dense is V x D fp64, overwritten.
 */
int orc_dense_scatter(const void* grad, int gtype, int64_t K, int64_t D,
                      int64_t ld, const int64_t* J, int64_t V, double* dense) {
  if (K < 0 || D < 0 || V < 1 || ld < D) return ORC_BADARG;
  memset(dense, 0, (size_t)(V * D) * sizeof(double));
  for (int64_t k = 0; k < K; ++k) {
    if (J[k] < 0 || J[k] >= V) return ORC_RANGE;
    for (int64_t d = 0; d < D; ++d)
      dense[J[k] * D + d] += grad_at(grad, gtype, ld, k, d);
  }
  return ORC_OK;
}

/* Position of x in the strictly ascending list a[0..n), or -1. */
static int64_t find_sorted(const int64_t* a, int64_t n, int64_t x) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    int64_t mid = lo + (hi - lo) / 2;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return (lo < n && a[lo] == x) ? lo : -1;
}

/*
 * Step 4 (Sec. III-A): the map from the local types J^ to the global types
 * I^: map[u] is the position of sub[u] in sup (both ascending), or -1.
 * Returns ORC_NOTFOUND when some sub id is missing from sup.
 */
int orc_map(const int64_t* sub, int64_t n_sub, const int64_t* sup,
            int64_t n_sup, int32_t* map) {
  int missing = 0;
  for (int64_t u = 0; u < n_sub; ++u) {
    int64_t r = find_sorted(sup, n_sup, sub[u]);
    map[u] = (int32_t)r;
    if (r < 0) missing = 1;
  }
  return missing ? ORC_NOTFOUND : ORC_OK;
}

/*
 * Step 5 (Sec. III-A): expand the U_i x D local reduction into a U_g x D
 * matrix M laid out by the global types: the row of dst_ids that equals
 * src_ids[u] receives src[u]; rows with no local type are zero.
 */
int orc_expand(const double* src, int64_t n_src, int64_t D,
               const int64_t* src_ids, const int64_t* dst_ids, int64_t n_dst,
               double* dst) {
  memset(dst, 0, (size_t)(n_dst * D) * sizeof(double));
  for (int64_t u = 0; u < n_src; ++u) {
    int64_t r = find_sorted(dst_ids, n_dst, src_ids[u]);
    if (r < 0) return ORC_NOTFOUND;
    for (int64_t d = 0; d < D; ++d) dst[r * D + d] = src[u * D + d];
  }
  return ORC_OK;
}

/*
 * Row write (add == 0) or row accumulation (add != 0) of src[u] at the row
 * of src_ids[u]: its position in dst_ids, or the id itself when dst_ids is
 * NULL (a dense table of dst_rows rows). Untouched rows keep their values.
 */
int orc_scatter(const double* src, int64_t n_src, int64_t D,
                const int64_t* src_ids, const int64_t* dst_ids, int64_t n_dst,
                double* dst, int64_t dst_rows, int add) {
  for (int64_t u = 0; u < n_src; ++u) {
    int64_t r;
    if (dst_ids) {
      r = find_sorted(dst_ids, n_dst, src_ids[u]);
      if (r < 0) return ORC_NOTFOUND;
    } else {
      r = src_ids[u];
      if (r < 0 || r >= dst_rows) return ORC_RANGE;
    }
    for (int64_t d = 0; d < D; ++d) {
      if (add) dst[r * D + d] += src[u * D + d];
      else dst[r * D + d] = src[u * D + d];
    }
  }
  return ORC_OK;
}

/*
 * Step 7 with plain SGD (the word-LM optimizer, Sec. IV-B): for each touched
 * row, p -= lr * g. p and g are n x D fp64 (the touched rows only).
 */
int orc_sgd(double* p, const double* g, int64_t n, int64_t D, double lr) {
  for (int64_t i = 0; i < n * D; ++i) p[i] -= lr * g[i];
  return ORC_OK;
}

/*
 * Step 7 with Adam (the char-LM optimizer, Sec. IV-B), applied lazily to the
 * touched rows only, with bias correction at step t and decoupled weight
 * decay wd:
 *   m = b1 m + (1-b1) g,  v = b2 v + (1-b2) g^2,
 *   p -= lr * ( (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps) + wd * p ).
 * p, m, v, g are n x D fp64.
 */
int orc_adam(double* p, double* m, double* v, const double* g, int64_t n,
             int64_t D, double lr, double b1, double b2, double eps,
             double wd, int64_t t) {
  if (t < 1) return ORC_BADARG;
  double c1 = 1.0 - pow(b1, (double)t);
  double c2 = 1.0 - pow(b2, (double)t);
  for (int64_t i = 0; i < n * D; ++i) {
    m[i] = b1 * m[i] + (1.0 - b1) * g[i];
    v[i] = b2 * v[i] + (1.0 - b2) * g[i] * g[i];
    double mhat = m[i] / c1;
    double vhat = v[i] / c2;
    p[i] -= lr * (mhat / (sqrt(vhat) + eps) + wd * p[i]);
  }
  return ORC_OK;
}

/*
 * Sec. III-C (lower precision): the payload that the GPUs exchange is cast
 * to IEEE binary16 after multiplying it by a compression scale F, and cast
 * back and divided by F at the receiving end. The kernels multiply in fp32
 * and round once to binary16, so the oracle does the same here.
 *
 * f16_bits: the binary16 encoding of an fp32 value, rounded to nearest with
 * ties to even, written out from the two formats (1 sign, 5 exponent bits
 * biased by 15, 10 fraction bits; subnormals below 2^-14 in units of 2^-24;
 * magnitudes that round past 65504 become infinity).
 */
static uint16_t f16_bits(float f) {
  uint32_t x;
  memcpy(&x, &f, sizeof x);
  const uint32_t sign = (x >> 16) & 0x8000u;
  const int exp32 = (int)((x >> 23) & 0xffu);
  const uint32_t frac = x & 0x7fffffu;
  if (exp32 == 0xff) return (uint16_t)(sign | (frac ? 0x7e00u : 0x7c00u));
  const int e = exp32 - 127 + 15; /* exponent field of binary16 */
  if (e >= 31) return (uint16_t)(sign | 0x7c00u);
  if (e >= 1) {
    /* normal: keep 10 of the 23 fraction bits, round on the other 13 */
    uint32_t h = ((uint32_t)e << 10) | (frac >> 13);
    const uint32_t rest = frac & 0x1fffu;
    if (rest > 0x1000u || (rest == 0x1000u && (h & 1u))) h += 1; /* a carry may reach infinity */
    return (uint16_t)(sign | h);
  }
  /* subnormal or zero: the value is M * 2^(e - 14) units of 2^-24, M the
     24-bit significand with its leading one */
  if (e < -10) return (uint16_t)sign; /* below half the smallest subnormal */
  const uint32_t M = frac | 0x800000u;
  const int s = 14 - e; /* bits dropped, 14..24 */
  uint32_t m = M >> s;
  const uint32_t rest = M & ((1u << s) - 1u), half = 1u << (s - 1);
  if (rest > half || (rest == half && (m & 1u))) m += 1; /* 1024 is the smallest normal */
  return (uint16_t)(sign | m);
}

/* The fp32 value of a binary16 encoding (exact). */
static float f16_value(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  const uint32_t e = (h >> 10) & 0x1fu, m = h & 0x3ffu;
  uint32_t x;
  if (e == 31) {
    x = sign | 0x7f800000u | (m << 13);
  } else if (e == 0) {
    if (m == 0) {
      x = sign;
    } else { /* subnormal: m * 2^-24 */
      float f = (float)m * 0x1p-24f;
      memcpy(&x, &f, sizeof x);
      x |= sign;
    }
  } else {
    x = sign | ((e - 15 + 127) << 23) | (m << 13);
  }
  float f;
  memcpy(&f, &x, sizeof f);
  return f;
}

/* Element-wise conversions, for the pins. */
int orc_f16_from_f32(const float* x, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = f16_bits(x[i]);
  return ORC_OK;
}

int orc_f32_from_f16(const uint16_t* h, int64_t n, float* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = f16_value(h[i]);
  return ORC_OK;
}

/*
 * Compression: out = binary16(fp32(fp32(x) * scale)), n x D. x arrives in
 * fp64 and is first rounded to fp32, the precision the kernels hold it in.
 */
int orc_compress(const double* x, int64_t n, int64_t D, float scale, uint16_t* out) {
  if (n < 0 || D < 0) return ORC_BADARG;
  for (int64_t i = 0; i < n * D; ++i) {
    const float x32 = (float)x[i];
    const float t = x32 * scale;
    out[i] = f16_bits(t);
  }
  return ORC_OK;
}

/* Decompression: out = fp32(fp32(h) * inv_scale), returned as fp64. */
int orc_decompress(const uint16_t* h, int64_t n, int64_t D, float inv_scale, double* out) {
  if (n < 0 || D < 0) return ORC_BADARG;
  for (int64_t i = 0; i < n * D; ++i) {
    const float g = f16_value(h[i]) * inv_scale;
    out[i] = (double)g;
  }
  return ORC_OK;
}

/*
 * Sec. II-A / III-B (sampled softmax): the output embedding is updated only
 * at a random subset of the vocabulary, drawn uniformly. Given 64-bit random
 * words r (drawn by the caller from its seed), the id of each is
 * floor(r * V / 2^64): the high word of the 128-bit product, which splits
 * [0, 2^64) into V runs of equal length (to within one).
 */
int orc_sample_ids(const uint64_t* r, int64_t n, int64_t V, int64_t* ids) {
  if (n < 0 || V < 1) return ORC_BADARG;
  for (int64_t i = 0; i < n; ++i) {
    const unsigned __int128 p = (unsigned __int128)r[i] * (unsigned __int128)(uint64_t)V;
    ids[i] = (int64_t)(uint64_t)(p >> 64);
  }
  return ORC_OK;
}
