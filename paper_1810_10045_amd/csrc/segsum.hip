// Seg-Sum (Sec. III-A step 2): out[u, :] = sum of grad[perm[i], :] over the
// sorted positions i of type u, accumulated in fp32 in a fixed order.
//
// Work partition (no float atomics, run-to-run bit-identical):
//   The K sorted positions are cut into N chunks of equal cost, one chunk per
//   wave and per column tile of up to 1024 columns. A position costs one row
//   read (rw) and a segment end one row write (ww, weighted per gradient
//   dtype by measurement), so the cost before position p
//   of segment u is rw * p + ww * u; chunk c starts where that reaches c * Q,
//   Q = ceil((rw * K + ww * U) / N). Reads and writes thus balance across
//   waves wherever the heads and the tail of the Zipf law fall in the sorted
//   order (equal-length chunks left the waves of the tail, one write per row,
//   twice as long as those of the heads). A wave finds its bounds with a
//   32-ary search of offsets, two targets at once. The search ends at the
//   segments holding the two bounds, which tells the wave where the first
//   and last segment of its chunk begin and end. The segment (type) of a
//   position is inverse[perm[i]], so a wave learns every other segment
//   boundary of its chunk from two gathers and a ballot, without searching.
//   A segment shorter than T rows belongs entirely to the chunk holding its
//   first position, even where it runs past the chunk end; a longer one is
//   cut at chunk boundaries and every chunk sums its piece into a partial
//   row:
//     part_start[c]  the piece of a long segment that starts in chunk c and
//                    continues past it (desc[c] names that segment),
//     part_cont[c]   the piece of a long segment that started before chunk c.
//   The chunk that starts such a segment also records in npieces[c] how many
//   chunks after c it reaches (the chunk of its last position, from the same
//   cost formula), so that k_segsum_fix finds every piece from one load. It
//   sums part_start[c] and part_cont[c + 1 .. c + npieces[c]] in order: one
//   wave per column tile for a segment of fewer than 16 further pieces, all
//   waves of a workgroup (fixed stride split of the pieces, fixed-order
//   combine in LDS) for a head. On the 16-byte vector path (rows of up to
//   LMZ_SEG_FUSED_MAX_D columns) the same fix-up runs as workgroups of the
//   walk's own launch, each waiting for the flags of the chunks and column
//   tiles it reads (the fused launch below).
// A chunk holds at most R positions (N is sized for U = min(K, u_cap)) and
// reads at most R + T - 1 rows.
//
// Each wave gathers whole 16-byte column vectors of RF rows at a time
// (RF x NV x 1 KiB in flight), adds them in fp32 registers and writes a row
// as soon as its segment ends; grad is streamed with non-temporal loads.
//
// lm_segsum_rows runs the same kernels with a row map: type u's sum goes to
// row row_ids[u] of the output (the dense table of a SCATTER). The walk
// gathers the row of each window position's type with the types; the
// fix-up looks it up per segment. Without a row map, row u.
//
// lm_segsum_sgd and lm_segsum_adam (the update instantiations, OP) update
// those rows instead of writing them, the sum in the same order and the
// update the same arithmetic as lm_sparse_apply's (sgd_value, adam_value).
// The walk then closes a gather batch after its kEnds-th segment end and
// loads the table rows of those ends (Adam: the parameters, m and v) with
// its gradient rows, through buffer resources whose range is empty where no
// row is needed (such a load reads nothing and returns zeros), so an update
// costs no round trip of its own.
#include <atomic>
#include <cstdlib>

#include "common.hpp"

namespace lmz {

// Tuning knobs (overridable at build time).
#ifndef LMZ_SEG_TARGET_CHUNKS
#define LMZ_SEG_TARGET_CHUNKS 1024   // R = the power of two near K / this (16..512)
#endif
#ifndef LMZ_SEG_WRITE_X2_F32
#define LMZ_SEG_WRITE_X2_F32 2       // fp32 rows: cost of a row written / a row read, times 2
#endif
#ifndef LMZ_SEG_WRITE_X2_BF16
#define LMZ_SEG_WRITE_X2_BF16 4      // bf16 rows: the same ratio, times 2
#endif
#ifndef LMZ_SEG_TDIV
#define LMZ_SEG_TDIV 4               // long-segment threshold T = R / this (1..64)
#endif
#ifndef LMZ_SEG_RF4
#define LMZ_SEG_RF4 4                // rows per gather batch with 4 vectors per lane
#endif
#ifndef LMZ_SEG_RF2
#define LMZ_SEG_RF2 8                // rows per gather batch with <= 2 vectors per lane
#endif
#ifndef LMZ_SEG_LONG_R
#define LMZ_SEG_LONG_R 512           // from this chunk length on, the *_LONG batches
#endif
#ifndef LMZ_SEG_RF4_LONG
#define LMZ_SEG_RF4_LONG 8           // long chunks walk long enough to keep more rows in flight
#endif
#ifndef LMZ_SEG_RF2_LONG
#define LMZ_SEG_RF2_LONG 16
#endif
#ifndef LMZ_SEG_SGD_ENDS
#define LMZ_SEG_SGD_ENDS 2           // lm_segsum_sgd: segment ends (table rows) per gather batch
#endif
#ifndef LMZ_SEG_SGD_RF4
#define LMZ_SEG_SGD_RF4 3            // lm_segsum_sgd: rows per batch with 4 vectors per lane,
#endif                               // chunks below LMZ_SEG_LONG_R (others as lm_segsum)
#ifndef LMZ_SEG_ADAM_RF4
#define LMZ_SEG_ADAM_RF4 2           // lm_segsum_adam: the same, every chunk length (one end,
                                     // three table rows per batch; 4 at most with fewer vectors)
#endif
#ifndef LMZ_SEG_NV_MAX
#define LMZ_SEG_NV_MAX 4             // 16-byte vectors per lane per row (fp32)
#endif
#ifndef LMZ_SEG_FIX_RF
#define LMZ_SEG_FIX_RF 16            // partial rows per wave in flight in the fix-up
#endif

#ifndef LMZ_SEG_WG_THREADS
#define LMZ_SEG_WG_THREADS 64        // threads of a main-walk workgroup (one chunk per wave)
#endif
#ifndef LMZ_SEG_FUSED
#define LMZ_SEG_FUSED 1              // fix-up workgroups in the walk's launch (one column tile)
#endif
#ifndef LMZ_SEG_FUSED_MAX_D
#define LMZ_SEG_FUSED_MAX_D 4096     // widest rows walked and fixed up in one launch
#endif
#ifndef LMZ_SEG_LDS_PAD
#define LMZ_SEG_LDS_PAD 0            // LDS bytes reserved per workgroup (caps waves per CU)
#endif
constexpr int kSegThreads = LMZ_SEG_WG_THREADS;
constexpr int kSegWaves = kSegThreads / kWave;
constexpr int kMinR = 16, kMaxR = 512;

struct SegArgs {
  const void* grad;
  int64_t ld_grad;
  int K, D;
  const int32_t* perm;
  const int32_t* inverse;
  const int32_t* offsets;
  const int64_t* num_unique;
  int64_t u_cap;
  float* out;
  int64_t ld_out;
  float* part_cont;
  float* part_start;
  int32_t* desc;
  int32_t* npieces;
  uint64_t* flags;   // fused launch: flags[c * tiles + t] == epoch once column tile t of
  uint64_t epoch;    // chunk c (and, for t = 0, its descriptor) is visible everywhere
  uint64_t wait_epoch;  // the value the fix-up waits for: epoch (or, with the
                        // failure-path test hook, one no walk writes)
  uint32_t spin_limit;  // polls of a flag before the wait gives up
  int main_blocks, fix_tiles, fused;
  int tiles, tile_cols;    // column tiles of the walk and the columns of one
  int R, nchunks, rw, ww;  // cost of a position / of a segment end
  int max_chunks;          // chunks the workspace holds
  const void* row_ids;     // lm_segsum_rows: type u goes to out row row_ids[u]
  int row_ids64;           //   (int64 ids when nonzero), < out_rows; nullptr: row u
  int64_t out_rows;
  int32_t* dev_err;
  OptParams opt;           // lm_segsum_sgd / _adam: the step (out is the table)
  float* m;                // lm_segsum_adam: the moments, rows of out's stride
  float* v;
};

// What a finished type row becomes: written (lm_segsum, lm_segsum_rows), or
// applied to the table row by SGD or Adam.
constexpr int kOpStore = 0, kOpSgd = 1, kOpAdam = 2;

struct SegLayout {
  int R, max_chunks;
  size_t cont, start, desc, npieces, flags, total;
};

static inline size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

// Costs: a sorted position (a row read) costs rw = 2 * sizeof(grad) per
// column, a segment end (a row written, always fp32) ww = 4 * X2, where X2 / 2
// is the cost of a written row relative to a read row. Measured on MI355X:
// with fp32 rows a written row is best weighted by its bytes (X2 = 2: 1-5%
// faster Seg-Sum than X2 = 4 on the fp32 workloads), with bf16 rows at twice
// the bytes of a read row (X2 = 4: 3% faster than X2 = 2 on the bf16 merge).
// A call has at most rw * K + ww * min(K, u_cap) of it, at most rw * R per
// chunk.
static inline int read_cost(int gtype) { return gtype == LM_BF16 ? 4 : 8; }
static inline int write_cost(int gtype) {
  return 4 * (gtype == LM_BF16 ? LMZ_SEG_WRITE_X2_BF16 : LMZ_SEG_WRITE_X2_F32);
}
constexpr int kMaxWriteCost =
    4 * (LMZ_SEG_WRITE_X2_BF16 > LMZ_SEG_WRITE_X2_F32 ? LMZ_SEG_WRITE_X2_BF16 : LMZ_SEG_WRITE_X2_F32);
static inline int64_t chunks_for(int64_t K, int R, int rw, int ww, int64_t u_cap) {
  const int64_t ub = u_cap < K ? u_cap : K;
  return (int64_t(rw) * K + int64_t(ww) * ub + int64_t(rw) * R - 1) / (int64_t(rw) * R);
}

static SegLayout seg_layout(int64_t K, int64_t D) {
  SegLayout L{};
  const int64_t want = (K + LMZ_SEG_TARGET_CHUNKS - 1) / LMZ_SEG_TARGET_CHUNKS;
  int R = kMinR;
  while (R < want && R < kMaxR) R *= 2;
  L.R = R;
  L.max_chunks = static_cast<int>(chunks_for(K, R, 4, kMaxWriteCost, K));  // any dtype and capacity
  const size_t n = size_t(L.max_chunks);
  size_t off = 0;
  L.cont = off;     off += a256(n * D * 4);
  L.start = off;    off += a256(n * D * 4);
  L.desc = off;     off += a256(n * 4);
  L.npieces = off;  off += a256(n * 4);
  L.flags = off;    off += a256(n * size_t((D + 1023) / 1024) * 8);  // per chunk and column tile
  L.total = off;
  return L;
}

size_t segsum_workspace_bytes(int64_t K, int64_t D) { return seg_layout(K, D).total; }

// Windows of positions a wave loads up front: [p0 - 1, p0 - 1 + 64 * NW)
// must cover p0 - 1 (to see whether the first segment started earlier), the
// whole walk (at most R + T - 1 rows from p0) and one position past it (to
// see whether the last row ends its segment).
template <int R, int T>
constexpr int windows_for() { return (R + T) / 64 + 1; }

// Chunk bounds: the number of sorted positions whose running cost is below
// t (the cost before position p of segment u is rw * p + ww * u), for
// t = tA in lanes 0..31 and t = tB in lanes 32..63. A 32-ary search per
// half-wave for the largest u < U with f(u) = rw * offsets[u] + ww * u <= t
// (f(0) = 0), then b = offsets[u] + min(ceil((t - f(u)) / rw), len(u));
// b = K once t >= rw * K + ww * U. Every value the search keeps is
// wave-uniform. Besides b it returns that u and offsets[u], offsets[u + 1]:
// b lies strictly inside segment u exactly when offsets[u] < b < offsets[u + 1].
struct Bound {
  int b, u, o0, o1;
};
__device__ __forceinline__ void chunk_bounds(const int32_t* __restrict__ offsets, int U, int rw,
                                             int ww, int K, int64_t tA, int64_t tB, Bound& A,
                                             Bound& B) {
  const int lane = lane_id();
  const bool hi = lane >= 32;
  const int hl = lane & 31;
  int loA = 0, nA = U, loB = 0, nB = U;
  while (nA > 1 || nB > 1) {
    const int sA = (nA + 31) / 32, sB = (nB + 31) / 32;
    const int lo = hi ? loB : loA, n = hi ? nB : nA, st = hi ? sB : sA;
    const int64_t t = hi ? tB : tA;
    const int u = lo + (hl + 1) * st;
    bool le = false;
    if (n > 1 && u < lo + n) le = int64_t(rw) * offsets[u] + int64_t(ww) * u <= t;
    const uint64_t m = ballot(le);
    const int cA = __popcll(m & 0xffffffffull), cB = __popcll(m >> 32);
    if (nA > 1) {
      loA += cA * sA;
      nA = nA - cA * sA < sA ? nA - cA * sA : sA;
    }
    if (nB > 1) {
      loB += cB * sB;
      nB = nB - cB * sB < sB ? nB - cB * sB : sB;
    }
  }
  const int u = hi ? loB : loA;
  const int64_t t = hi ? tB : tA;
  const int o0 = offsets[u], o1 = offsets[u + 1];
  const int64_t into = (t - (int64_t(rw) * o0 + int64_t(ww) * u) + rw - 1) / rw;
  int b = int64_t(o0) + into < int64_t(o1) ? static_cast<int>(int64_t(o0) + into) : o1;
  if (t >= int64_t(rw) * K + int64_t(ww) * U) b = K;
  A = Bound{first_lane(b), first_lane(u), first_lane(o0), first_lane(o1)};
  B = Bound{read_lane(b, 32), read_lane(u, 32), read_lane(o0, 32), read_lane(o1, 32)};
}

// ---------------------------------------------------------------------------
// Fused launch: fix-up workgroups after the walk's in the same grid.
// Workgroups are dispatched in the order of their index (per XCD), so every
// walk workgroup holds a slot or has finished before a fix-up workgroup
// starts; walk workgroups never wait, so a fix-up's wait for their flags
// always ends (bounded all the same: LM_DEVERR_SPIN). Partial rows and
// descriptors go out as agent-scope stores (coherent across the XCDs'
// L2s), the walk waits for them before it sets its flag to the call's
// epoch, and the fix-up reads them with agent-scope loads once the flag
// holds that epoch: no workspace contents need clearing between calls.
// Rows wider than one walk tile (1024 columns) take one flag per chunk and
// tile: workgroup b of the walk is column tile b % tiles of chunks
// (b / tiles) * 4 ..., and a fix-up tile of 256 columns, which lies inside
// one walk tile, waits for that tile's flags (tile 0's also covers the
// chunk's descriptor).
// ---------------------------------------------------------------------------
constexpr int kFusedThreads = 256;
constexpr int kFusedWaves = kFusedThreads / kWave;
#ifndef LMZ_SEG_FUSED_SPAN
#define LMZ_SEG_FUSED_SPAN 4         // chunks a fused fix-up workgroup looks after (<= 64)
#endif
#ifndef LMZ_SEG_FUSED_RF
#define LMZ_SEG_FUSED_RF 8           // pieces per wave per round in the fused fix-up
#endif
#ifndef LMZ_SEG_FUSED_SLEEP
#define LMZ_SEG_FUSED_SLEEP 8        // s_sleep argument (x 64 cycles) between flag polls
#endif
constexpr int kFusedSpan = LMZ_SEG_FUSED_SPAN;
constexpr int kFusedCols = kWave * 4;  // columns of a fused fix-up tile
static_assert(kFusedSpan <= kWave, "one descriptor per lane");

// The output row of type s: s itself, or row_ids[s] for lm_segsum_rows
// (-1 when that id lies outside [0, out_rows); LM_DEVERR_ID_RANGE is raised
// and the row is not written).
__device__ __forceinline__ int64_t out_row_of(const SegArgs& a, int s) {
  if (!a.row_ids) return s;
  const int64_t r = a.row_ids64 ? static_cast<const int64_t*>(a.row_ids)[s]
                                : static_cast<const int32_t*>(a.row_ids)[s];
  if (r < 0 || r >= a.out_rows) {
    raise_err(a.dev_err, LM_DEVERR_ID_RANGE);
    return -1;
  }
  return r;
}

// The update instantiations: a buffer resource over row r (D fp32 values)
// of base (the table, m or v, all of out's row stride), or over nothing for
// r < 0: loads through an empty range read no memory and return zeros, so
// a batch loads its table rows unconditionally.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t table_row(const SegArgs& a, float* base,
                                                            int64_t r) {
  constexpr int kRawBufferWord3 = 0x00020000;  // 32-bit data format, no swizzle
  return __builtin_amdgcn_make_buffer_rsrc(base + (r >= 0 ? r : 0) * a.ld_out, 0,
                                           r >= 0 ? a.D * 4 : 0, kRawBufferWord3);
}

// VEC fp32 values at column col of the row behind resource rs.
template <int VEC>
__device__ __forceinline__ void table_vec(__amdgpu_buffer_rsrc_t rs, int col, float* v) {
  if constexpr (VEC % 4 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 4) {
      const f32x4 x = __builtin_bit_cast(
          f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, (col + i) * 4, 0, 0));
      v[i] = x.x;
      v[i + 1] = x.y;
      v[i + 2] = x.z;
      v[i + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      v[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, (col + i) * 4, 0, 0));
  }
}

// Finish VEC columns from col of type row orow: out = sum, or the table
// row (and Adam's moments) updated with it.
template <int VEC, int OP>
__device__ __forceinline__ void finish_row(const SegArgs& a, int64_t orow, int col, float* sum) {
  const int64_t off = orow * a.ld_out + col;
  if constexpr (OP == kOpSgd) {
    float p[VEC];
    load_vec<VEC>(a.out + off, p);
#pragma unroll
    for (int e = 0; e < VEC; ++e) sgd_value(p[e], sum[e], a.opt);
    store_vec<VEC>(a.out + off, p);
  } else if constexpr (OP == kOpAdam) {
    float p[VEC], m[VEC], v[VEC];
    load_vec<VEC>(a.out + off, p);
    load_vec<VEC>(a.m + off, m);
    load_vec<VEC>(a.v + off, v);
#pragma unroll
    for (int e = 0; e < VEC; ++e) adam_value(p[e], m[e], v[e], sum[e], a.opt);
    store_vec<VEC>(a.out + off, p);
    store_vec<VEC>(a.m + off, m);
    store_vec<VEC>(a.v + off, v);
  } else {
    store_vec<VEC>(a.out + off, sum);
  }
}

template <int VEC>
__device__ __forceinline__ void store_vec_agent(float* p, const float* v) {
  static_assert(VEC % 2 == 0, "pairs of fp32 values");
#pragma unroll
  for (int i = 0; i < VEC; i += 2)
    st_agent(reinterpret_cast<uint64_t*>(p + i),
             uint64_t(__float_as_uint(v[i])) | (uint64_t(__float_as_uint(v[i + 1])) << 32));
}

__device__ __forceinline__ void load4_agent(const float* p, float* v) {
  const uint64_t x = ld_agent(reinterpret_cast<const uint64_t*>(p));
  const uint64_t y = ld_agent(reinterpret_cast<const uint64_t*>(p) + 1);
  v[0] = __uint_as_float(static_cast<uint32_t>(x));
  v[1] = __uint_as_float(static_cast<uint32_t>(x >> 32));
  v[2] = __uint_as_float(static_cast<uint32_t>(y));
  v[3] = __uint_as_float(static_cast<uint32_t>(y >> 32));
}

// Every lane of the wave calls this; the lanes with need wait until
// flags[idx] holds the epoch. False if the wait gave up.
__device__ __forceinline__ bool wait_flags(const SegArgs& a, int idx, bool need) {
  for (uint32_t spin = 0;; ++spin) {
    const bool ok = !need || ld_agent(a.flags + idx) == a.wait_epoch;
    if (!ballot(!ok)) return true;
    if (spin >= a.spin_limit) {
      if (lane_id() == 0) raise_err(a.dev_err, LM_DEVERR_SPIN);
      return false;
    }
    __builtin_amdgcn_s_sleep(LMZ_SEG_FUSED_SLEEP);
  }
}

// Fix-up workgroup f: chunks [c0, c0 + kFusedSpan) of span f / fix_tiles,
// columns of tile f % fix_tiles. It waits for the span's descriptors, then
// sums each long segment that starts there as k_segsum_fix does (one wave
// for fewer than 16 further pieces, all waves and an LDS combine for a
// head), waiting for each piece's flag before loading it.
template <int OP>
__device__ __forceinline__ void fused_fix(const SegArgs& a) {
  constexpr int RF = LMZ_SEG_FUSED_RF;
  constexpr int kShortMax = 16;  // further pieces below this: one wave
  __shared__ float s_part[kFusedWaves][kFusedCols];
  const int lane = lane_id();
  const int wave = first_lane(static_cast<int>(threadIdx.x >> 6));
  const int f = static_cast<int>(blockIdx.x) - a.main_blocks;
  const int c0 = (f / a.fix_tiles) * kFusedSpan;
  const int nc = a.nchunks - c0 < kFusedSpan ? a.nchunks - c0 : kFusedSpan;
  const int D = a.D;
  const int col = (f % a.fix_tiles) * kFusedCols + lane * 4;
  const int col_ld = col < D ? col : D - 4;  // past the end: a valid, unstored vector
  // The walk's column tile these columns belong to (a fix-up tile of
  // kFusedCols columns never straddles two), and the flag of chunk x's part
  // of it; tile 0's flag also covers x's descriptor.
  const int wt = (f % a.fix_tiles) * kFusedCols / a.tile_cols;
  auto flag_of = [&](int x, int t) { return x * a.tiles + t; };
  const int U = first_lane(static_cast<int>(*a.num_unique));

  // Wave 0 waits for the span and reads its descriptors once; every wave
  // takes them from LDS, so all agree on the heads (and on the barriers).
  __shared__ int s_desc[kWave], s_np[kWave];
  const bool mine = lane < nc;
  const int ci = c0 + (mine ? lane : 0);
  if (wave == 0) {
    wait_flags(a, flag_of(ci, 0), mine);
    s_desc[lane] = mine ? ld_agent(a.desc + ci) : -1;
    s_np[lane] = mine ? ld_agent(a.npieces + ci) : 0;
  }
  __syncthreads();
  const int sd = s_desc[lane], np = s_np[lane];
  const bool has = sd >= 0 && sd < U && sd < a.u_cap && np >= 1 && np <= a.nchunks - 1 - ci;
  const uint64_t todo = ballot(has);
  const uint64_t heads = ballot(has && np >= kShortMax);
  auto piece = [&](int cs, int t) {
    return (t == 0 ? a.part_start + static_cast<int64_t>(cs) * D
                   : a.part_cont + static_cast<int64_t>(cs + t) * D) + col_ld;
  };

  // Shorter long segments: the j-th to wave j % kFusedWaves.
  int j = 0;
  for (uint64_t m = todo & ~heads; m; m &= m - 1, ++j) {
    if (j % kFusedWaves != wave) continue;
    const int i = __builtin_ctzll(m);
    const int cs = c0 + i, s = read_lane(sd, i), P = read_lane(np, i);
    wait_flags(a, flag_of(cs + (lane <= P ? lane : 0), wt), lane <= P);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int t0 = 0; t0 <= P; t0 += RF) {
      float buf[RF][4];
#pragma unroll
      for (int r = 0; r < RF; ++r) load4_agent(piece(cs, t0 + r <= P ? t0 + r : 0), buf[r]);
#pragma unroll
      for (int r = 0; r < RF; ++r)
        if (t0 + r <= P)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += buf[r][e];
    }
    const int64_t orow = out_row_of(a, s);
    if (col < D && orow >= 0) finish_row<4, OP>(a, orow, col, acc);
  }

  // Heads, one after the other, all waves: wave w adds pieces w, w + W, ...
  for (uint64_t m = heads; m; m &= m - 1) {
    const int i = __builtin_ctzll(m);
    const int cs = c0 + i, s = read_lane(sd, i), P = read_lane(np, i);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int t0 = wave; t0 <= P; t0 += kFusedWaves * RF) {
      const int tl = t0 + (lane < RF ? lane : 0) * kFusedWaves;  // lane r: piece t0 + r * W
      wait_flags(a, flag_of(cs + (tl <= P ? tl : 0), wt), lane < RF && tl <= P);
      float buf[RF][4];
#pragma unroll
      for (int r = 0; r < RF; ++r) {
        const int t = t0 + r * kFusedWaves;
        load4_agent(piece(cs, t <= P ? t : t0), buf[r]);
      }
#pragma unroll
      for (int r = 0; r < RF; ++r)
        if (t0 + r * kFusedWaves <= P)
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[e] += buf[r][e];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) s_part[wave][lane * 4 + e] = acc[e];
    __syncthreads();
    const int64_t orow = out_row_of(a, s);
    for (int x = threadIdx.x; x < kFusedCols; x += kFusedThreads) {
      const int cx = (f % a.fix_tiles) * kFusedCols + x;
      if (cx < D && orow >= 0) {
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < kFusedWaves; ++w) sum += s_part[w][x];
        finish_row<1, OP>(a, orow, cx, &sum);
      }
    }
    __syncthreads();
  }
}

template <typename GT, int VEC, int NV, int RF, int R, int T, int NTHR, bool FUSED, int OP>
__global__ __launch_bounds__(NTHR) void k_segsum(SegArgs a) {
  if constexpr (FUSED) {
    if (static_cast<int>(blockIdx.x) >= a.main_blocks) {
      fused_fix<OP>(a);
      return;
    }
  }
  using RV = RowVec<GT, VEC>;
  using raw_t = typename RV::raw_t;
  constexpr int kColsPerVec = kWave * VEC;
  constexpr int CT = NV * kColsPerVec;
  constexpr int NW = windows_for<R, T>();

  const int lane = lane_id();
  // One chunk and column tile per wave: the fused grid is one-dimensional,
  // column tile = block % tiles; otherwise the tile is blockIdx.y.
  const int blk = FUSED ? static_cast<int>(blockIdx.x) / a.tiles : static_cast<int>(blockIdx.x);
  const int ct = FUSED ? static_cast<int>(blockIdx.x) % a.tiles : static_cast<int>(blockIdx.y);
  const int c = first_lane(blk * (NTHR / kWave) + static_cast<int>(threadIdx.x >> 6));
  if (c >= a.nchunks) return;
  // Fused launch: once this chunk's descriptor and partial rows are visible
  // at agent scope (written with agent-scope stores, then waited for),
  // flags[c] says so to the fix-up workgroups.
  auto publish = [&]() {
    if constexpr (FUSED) {
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (lane_id() == 0) st_agent(a.flags + size_t(c) * a.tiles + ct, a.epoch);
    }
  };
  const int K = a.K, D = a.D;

  // 0. This chunk's positions [p0, p1): equal shares of the cost rw * K + ww * U.
  const int64_t U64 = *a.num_unique;
  if (U64 > a.u_cap && c == 0 && ct == 0 && lane == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
  const int U = first_lane(static_cast<int>(U64 < K ? U64 : K));
  if (U < 1) {  // K > 0 always has a type: only a bad count gets here
    if (ct == 0 && lane == 0) {
      st_agent(a.desc + c, -1);
      st_agent(a.npieces + c, 0);
      if (c == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
    }
    publish();
    return;
  }
  const int Ub = U < a.u_cap ? U : static_cast<int>(a.u_cap);
  const int64_t cost = int64_t(a.rw) * K + int64_t(a.ww) * Ub;
  const int64_t Q = (cost + a.nchunks - 1) / a.nchunks;
  Bound A, B;
  chunk_bounds(a.offsets, U, a.rw, a.ww, K, int64_t(c) * Q, int64_t(c + 1) * Q, A, B);
  const int p0 = A.b;
  int p1 = B.b;
  bool cut_after = c < a.nchunks - 1;  // p1 is a cut of the cost, not the end of the positions
  if (!cut_after) p1 = K;
  if (p1 - p0 > R) {  // only inconsistent offsets: never walk past the windows
    if (lane == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
    p1 = p0 + R;
    cut_after = false;
  }
  if (p1 <= p0) {  // an empty chunk (a segment end cost more than Q)
    if (ct == 0 && lane == 0) {
      st_agent(a.desc + c, -1);
      st_agent(a.npieces + c, 0);
    }
    publish();
    return;
  }

  // 1. The first and the last segment of the chunk, from the search: the
  //    first started before the chunk when p0 lies strictly inside it, the
  //    last runs on after the chunk when p1 does.
  const bool started_before = p0 > A.o0 && p0 < A.o1;
  const int s_f = A.u, len_f = A.o1 - A.o0;
  const bool cont_after = cut_after && p1 > B.o0 && p1 < B.o1;
  const int s_l = B.u, len_l = B.o1 - B.o0;
  const bool long_f = started_before && len_f >= T;
  const bool long_l = cont_after && len_l >= T;
  if (ct == 0 && lane == 0) {
    // A long segment that starts in this chunk ends in the chunk of its last
    // position, whose cost is rw * (offsets[s_l + 1] - 1) + ww * s_l.
    const bool starts_long = long_l && !(started_before && s_l == s_f);
    int np = 0;
    if (starts_long) {
      int64_t ce = (int64_t(a.rw) * (B.o1 - 1) + int64_t(a.ww) * s_l) / Q;
      if (ce > a.nchunks - 1) ce = a.nchunks - 1;
      np = static_cast<int>(ce - c);
    }
    st_agent(a.desc + c, starts_long && np >= 1 ? s_l : -1);
    st_agent(a.npieces + c, np);
  }
  // Rows this chunk sums: skip a short segment owned by the previous chunk,
  // run a short last segment to its end, stop a long one at p1.
  const int q = started_before && !long_f ? A.o1 : p0;
  int q_end = cont_after && !long_l ? B.o1 : p1;
  const int walk_max = p0 - 1 + NW * kWave - 1;  // last position whose end bit is known
  bool bad = false;
  if (q_end > walk_max) {
    bad = true;  // only inconsistent offsets get here: never walk past the windows
    q_end = walk_max;
  }

  // 2. Gather the permutation and the segment of every position in the
  //    windows (sentinels: -2 before position 0, -1 from position K on).
  //    The loads are unconditional, at clamped positions: a load under a
  //    lane condition makes the compiler wait for every load before it.
  //    The windows cover the longest chunk; the walk reads rows q ..
  //    q_end - 1, and the end bit of row q_end - 1 needs the segment of
  //    position q_end, so past q_end every lane repeats it (one line, a
  //    cache hit) instead of fetching positions no row uses.
  int pw[NW], sw[NW];
  auto win_pos = [&](int w) {
    const int p = p0 - 1 + w * kWave + lane;
    return p < q_end ? p : q_end;
  };
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int pos = win_pos(w);
    pw[w] = a.perm[pos < 0 ? 0 : (pos < K ? pos : K - 1)];
  }
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int pos = win_pos(w);
    const bool ok = pos >= 0 && pos < K;
    const bool kin = static_cast<uint32_t>(pw[w]) < static_cast<uint32_t>(K);
    bad |= ok && !kin;
    if (!kin) pw[w] = 0;
    const int sv = a.inverse[pw[w]];
    sw[w] = ok ? sv : (pos < 0 ? -2 : -1);
  }
  // ends[w] bit j: position p0-1+64w+j is the last of its segment.
  uint64_t ends[NW];
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    int nxt = __shfl_down(sw[w], 1, kWave);
    if (lane == kWave - 1) nxt = w + 1 < NW ? read_lane(sw[w + 1 < NW ? w + 1 : w], 0) : -3;
    ends[w] = ballot(sw[w] != nxt);
  }
  // lm_segsum_rows: the output row of every position's type, gathered with
  // the windows (the first segment end needs it, not the first row loads);
  // -1 marks an id outside [0, out_rows) (and clamped positions).
  int orw[NW];
  const bool rows = a.row_ids != nullptr;
  if (rows) {
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const int sv = sw[w] >= 0 && sw[w] < a.u_cap ? sw[w] : 0;
      const int64_t r = a.row_ids64 ? static_cast<const int64_t*>(a.row_ids)[sv]
                                    : static_cast<const int32_t*>(a.row_ids)[sv];
      orw[w] = r >= 0 && r < a.out_rows ? static_cast<int>(r) : -1;
    }
  }

  // 3. Walk rows q .. q_end - 1, window by window. Lanes past the last column
  //    load a valid vector of the same row (col_ld) and never store it, so
  //    the loads need no per-lane guard.
  const int col0 = ct * CT + lane * VEC;
  bool col_ok[NV];
  int col_ld[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int col = col0 + v * kColsPerVec;
    col_ok[v] = col < D;
    col_ld[v] = col < D ? col : D - VEC;
  }
  const GT* __restrict__ grad = static_cast<const GT*>(a.grad);
  bool bad_row = false;
  // Update instantiations: segment ends per batch, and table rows per end
  // (Adam: the parameters, m and v; one end per batch, as three rows per
  // end fill the registers).
  constexpr int kEnds = OP == kOpSgd ? LMZ_SEG_SGD_ENDS : 1;
  constexpr int kRows = OP == kOpAdam ? 3 : 1;
  static_assert(kEnds >= 1 && kEnds <= RF, "table rows per batch");

  float acc[NV][VEC];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[v][e] = 0.f;

#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int wbase = p0 - 1 + w * kWave;
    const int lo = q > wbase ? q - wbase : 0;
    const int hi = q_end - wbase < kWave ? q_end - wbase : kWave;
    for (int j0 = lo; j0 < hi;) {
      int n = hi - j0 < RF ? hi - j0 : RF;
      // Updates: at most kEnds segment ends per batch (bm: their bits),
      // whose table rows load with the batch's gradient rows.
      uint64_t bm = 0;
      float tb[kEnds][kRows][NV][VEC];
      if constexpr (OP != kOpStore) {
        bm = (ends[w] >> j0) & ((uint64_t(1) << n) - 1);
        uint64_t past = bm;  // the ends after the first kEnds
#pragma unroll
        for (int k = 0; k < kEnds; ++k) past &= past - 1;
        if (past) {
          n = __builtin_ctzll(past);
          bm &= (uint64_t(1) << n) - 1;
        }
        uint64_t mm = bm;
#pragma unroll
        for (int k = 0; k < kEnds; ++k) {
          int64_t orow = -1;  // no row: a partial row, a type past u_cap, a bad id, no end
          if (mm) {
            const int j = j0 + __builtin_ctzll(mm);
            mm &= mm - 1;
            const int s = read_lane(sw[w], j);
            if (!(s == s_f && started_before) && s >= 0 && s < a.u_cap) orow = read_lane(orw[w], j);
          }
#pragma unroll
          for (int x = 0; x < kRows; ++x) {
            const __amdgpu_buffer_rsrc_t rs = table_row(a, x == 0 ? a.out : x == 1 ? a.m : a.v, orow);
#pragma unroll
            for (int v = 0; v < NV; ++v) table_vec<VEC>(rs, col_ld[v], tb[k][x][v]);
          }
        }
      }
      // Always RF row loads (rows past n repeat row n-1, a cache hit): a load
      // under a condition makes the compiler wait for every earlier load.
      raw_t buf[RF][NV];
#pragma unroll
      for (int r = 0; r < RF; ++r) {
        const int k = read_lane(pw[w], j0 + (r < n ? r : n - 1));
        const GT* row = grad + static_cast<int64_t>(k) * a.ld_grad;
#pragma unroll
        for (int v = 0; v < NV; ++v) buf[r][v] = RV::load(row + col_ld[v]);
      }
      // All RF rows in flight before the first add: keep the scheduler from
      // interleaving the adds of early rows with the loads of later ones.
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int r = 0; r < RF; ++r) {
        if (r < n) {
#pragma unroll
          for (int v = 0; v < NV; ++v) RV::add(acc[v], buf[r][v]);
          const int j = j0 + r;
          const bool is_end = (ends[w] >> j) & 1u;
          if (is_end || wbase + j == q_end - 1) {
            // is_end false here means a long last segment stopped at p1.
            const int s = read_lane(sw[w], j);
            float* dst;
            bool part = true;
            if (s == s_f && started_before) dst = a.part_cont + static_cast<int64_t>(c) * D;
            else if (!is_end) dst = a.part_start + static_cast<int64_t>(c) * D;
            else {
              part = false;
              const int64_t orow = rows ? read_lane(orw[w], j) : s;
              bad_row |= rows && orow < 0 && s >= 0 && s < a.u_cap;
              dst = (s >= 0 && s < a.u_cap && orow >= 0) ? a.out + orow * a.ld_out : nullptr;
            }
            if constexpr (OP == kOpSgd) {
              if (!part) {  // the batch's k-th end: table row k
                const int k = __popcll(bm & ((uint64_t(1) << (j - j0)) - 1));
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                  for (int e = 0; e < VEC; ++e) {
                    float t = tb[0][0][v][e];
#pragma unroll
                    for (int x = 1; x < kEnds; ++x) t = k == x ? tb[x][0][v][e] : t;
                    sgd_value(t, acc[v][e], a.opt);
                    acc[v][e] = t;
                  }
              }
            } else if constexpr (OP == kOpAdam) {
              if (!part) {  // the batch's one end: the parameters into acc, the moments in place
#pragma unroll
                for (int v = 0; v < NV; ++v)
#pragma unroll
                  for (int e = 0; e < VEC; ++e) {
                    adam_value(tb[0][0][v][e], tb[0][1][v][e], tb[0][2][v][e], acc[v][e], a.opt);
                    acc[v][e] = tb[0][0][v][e];
                  }
                if (dst) {
                  const int64_t off = dst - a.out;
#pragma unroll
                  for (int v = 0; v < NV; ++v) {
                    if (!col_ok[v]) continue;
                    store_vec<VEC>(a.m + off + col0 + v * kColsPerVec, tb[0][1][v]);
                    store_vec<VEC>(a.v + off + col0 + v * kColsPerVec, tb[0][2][v]);
                  }
                }
              }
            }
            if (dst) {
#pragma unroll
              for (int v = 0; v < NV; ++v) {
                if (!col_ok[v]) continue;
                float* d = dst + col0 + v * kColsPerVec;
                if constexpr (FUSED) {
                  if (part) store_vec_agent<VEC>(d, acc[v]);
                  else store_vec<VEC>(d, acc[v]);
                } else {
                  store_vec<VEC>(d, acc[v]);
                }
              }
            }
#pragma unroll
            for (int v = 0; v < NV; ++v)
#pragma unroll
              for (int e = 0; e < VEC; ++e) acc[v][e] = 0.f;
          }
        }
      }
      j0 += n;
    }
  }
  // Report a segment map that disagrees with offsets at the chunk start.
  const int seg_before = read_lane(sw[0], 0), seg_p0 = read_lane(sw[0], 1);
  if (started_before) bad |= seg_before != s_f || seg_p0 != s_f;
  else bad |= seg_before == seg_p0 || seg_p0 != (p0 == A.o1 ? A.u + 1 : A.u);
  if (ballot(bad) && lane == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
  if (ballot(bad_row) && lane == 0) raise_err(a.dev_err, LM_DEVERR_ID_RANGE);
  publish();
}

// Sum the pieces of every long segment that spans chunks (piece 0 is
// part_start[c], piece t >= 1 is part_cont[c + t], added in order of t).
// Grid: one workgroup of kFixWaves waves per kFixChunks chunks and per
// column tile of 64 * VEC columns. Few chunks start such a segment, so a
// workgroup reads the desc and npieces entries of its chunks with one
// coalesced load and a ballot, and only waves with work touch the partial
// rows (launching a wave per chunk cost more than the sums). The partial
// rows were just written, so the sums are bound by load latency: every wave
// issues all its piece loads before it waits for any. A segment of fewer
// than RF further pieces is summed by one wave; a longer one (a head of the
// Zipf law) by all kFixWaves waves, wave v adding pieces v, v + kFixWaves,
// ... in order, their partial rows then added in wave order through LDS.
// Long segments start at least RF chunks apart, so with kFixChunks <= RF a
// workgroup holds at most one head, and with kFixChunks <= kFixWaves each
// wave at most one shorter segment.
#ifndef LMZ_SEG_FIX_WAVES
#define LMZ_SEG_FIX_WAVES 8          // waves of a fix-up workgroup
#endif
#ifndef LMZ_SEG_FIX_CHUNKS
#define LMZ_SEG_FIX_CHUNKS 8         // chunks a fix-up workgroup looks after
#endif
constexpr int kFixWaves = LMZ_SEG_FIX_WAVES;
constexpr int kFixThreads = kFixWaves * kWave;
constexpr int kFixChunks = LMZ_SEG_FIX_CHUNKS;
static_assert(kFixChunks <= kFixWaves && kFixChunks <= LMZ_SEG_FIX_RF,
              "at most one short segment per wave and one head per workgroup");

template <int VEC, int RF, int OP>
__global__ __launch_bounds__(kFixThreads) void k_segsum_fix(SegArgs a) {
  constexpr int kCols = kWave * VEC;  // columns of a tile
  __shared__ float s_part[kFixWaves][kCols];
  const int lane = lane_id();
  const int wave = first_lane(static_cast<int>(threadIdx.x >> 6));
  const int D = a.D;
  const int U = first_lane(static_cast<int>(*a.num_unique));
  const int c0 = blockIdx.x * kFixChunks;
  const int col = blockIdx.y * kCols + lane * VEC;
  const int col_ld = col < D ? col : D - VEC;  // past the end: a valid, unstored vector

  // Chunks c0 + i that start a long segment (the same masks in every wave).
  const int ci = c0 + lane;
  const bool mine = lane < kFixChunks && ci < a.nchunks;
  const int sd = mine ? a.desc[ci] : -1;
  const int np = mine ? a.npieces[ci] : 0;
  const bool has = sd >= 0 && sd < U && sd < a.u_cap && np >= 1 && np <= a.nchunks - 1 - ci;
  const uint64_t todo = ballot(has);
  if (!todo) return;
  const uint64_t heads = ballot(has && np >= RF);
  const uint64_t shorts = todo & ~heads;
  auto piece = [&](int cs, int t) {
    return (t == 0 ? a.part_start + static_cast<int64_t>(cs) * D
                   : a.part_cont + static_cast<int64_t>(cs + t) * D) + col_ld;
  };

  // This wave's short segment: the wave-th of the mask.
  uint64_t m = shorts;
  for (int j = 0; j < wave && m; ++j) m &= m - 1;
  const int is = m ? __builtin_ctzll(m) : -1;
  const int ss = is >= 0 ? read_lane(sd, is) : -1, sP = is >= 0 ? read_lane(np, is) : 0;
  // The head, if any.
  const int ih = heads ? __builtin_ctzll(heads) : -1;
  const int hs = ih >= 0 ? read_lane(sd, ih) : -1, hP = ih >= 0 ? read_lane(np, ih) : 0;

  float sbuf[RF][VEC], hbuf[RF][VEC];
  if (is >= 0) {
#pragma unroll
    for (int r = 0; r < RF; ++r) load_vec<VEC>(piece(c0 + is, r <= sP ? r : 0), sbuf[r]);
  }
  if (ih >= 0) {
#pragma unroll
    for (int r = 0; r < RF; ++r) {
      const int t = wave + r * kFixWaves;
      load_vec<VEC>(piece(c0 + ih, t <= hP ? t : wave), hbuf[r]);
    }
  }
  if (is >= 0) {
    float acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = sbuf[0][e];
#pragma unroll
    for (int r = 1; r < RF; ++r)
      if (r <= sP)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += sbuf[r][e];
    const int64_t orow = out_row_of(a, ss);
    if (col < D && orow >= 0) finish_row<VEC, OP>(a, orow, col, acc);
  }
  if (ih < 0) return;  // the same in every wave: no barrier below is skipped by only some
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
#pragma unroll
  for (int r = 0; r < RF; ++r)
    if (wave + r * kFixWaves <= hP)
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += hbuf[r][e];
  // Heads longer than kFixWaves * RF pieces: further rounds.
  for (int t0 = wave + kFixWaves * RF; t0 <= hP; t0 += kFixWaves * RF) {
#pragma unroll
    for (int r = 0; r < RF; ++r) {
      const int t = t0 + r * kFixWaves;
      load_vec<VEC>(piece(c0 + ih, t <= hP ? t : t0), hbuf[r]);
    }
#pragma unroll
    for (int r = 0; r < RF; ++r)
      if (t0 + r * kFixWaves <= hP)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += hbuf[r][e];
  }
#pragma unroll
  for (int e = 0; e < VEC; ++e) s_part[wave][lane * VEC + e] = acc[e];
  __syncthreads();
  // Thread x adds column x of the tile over the waves in order.
  const int64_t orow = out_row_of(a, hs);
  for (int x = threadIdx.x; x < kCols; x += kFixThreads) {
    const int cx = blockIdx.y * kCols + x;
    if (cx < D && orow >= 0) {
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < kFixWaves; ++w) sum += s_part[w][x];
      finish_row<1, OP>(a, orow, cx, &sum);
    }
  }
}

template <int R>
constexpr int t_for() {
  constexpr int t = R / LMZ_SEG_TDIV;
  return t < 1 ? 1 : (t > 64 ? 64 : t);
}

// Rows per gather batch: more for long chunks (R >= LMZ_SEG_LONG_R), whose
// walks are long enough to use the extra rows in flight.
template <int NV, int R>
constexpr int rf_for() {
  return NV >= 4 ? (R >= LMZ_SEG_LONG_R ? LMZ_SEG_RF4_LONG : LMZ_SEG_RF4)
                 : (R >= LMZ_SEG_LONG_R ? LMZ_SEG_RF2_LONG : LMZ_SEG_RF2);
}

// lm_segsum_sgd's rows per batch, whose table rows take registers too.
// Measured at 65,536 ids over 800K words, D = 1024 (at most two ends per
// batch): 3 rows 98.4 us per call, 2 rows 99-101, 4 rows (lm_segsum's) 102,
// 5 rows 106; one end per batch 118 us with 4 rows, 111 with 3.
template <int NV, int R>
constexpr int rf_sgd_for() {
  return NV >= 4 && R < LMZ_SEG_LONG_R ? LMZ_SEG_SGD_RF4 : rf_for<NV, R>();
}

// lm_segsum_adam's rows per batch: three table rows per end take registers
// from the gradient batch, at every chunk length.
template <int NV, int R>
constexpr int rf_adam_for() {
  return NV >= 4 ? LMZ_SEG_ADAM_RF4 : (rf_for<NV, R>() < 4 ? rf_for<NV, R>() : 4);
}

// Multiprocessors of the current device (queried once per device).
static int device_cus() {
  static std::atomic<int> cus[64];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
    (void)hipGetLastError();
    return 0;
  }
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n <= 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      (void)hipGetLastError();
      return 0;
    }
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// Multiprocessors a launch on stream st may use: a stream created with a CU
// mask runs its workgroups on the masked ones only. Any other stream, or a
// failed query, gets the whole device.
static int stream_cus(hipStream_t st) {
  const int n = device_cus();
  uint32_t mask[32] = {};
  if (hipExtStreamGetCUMask(st, 32, mask) != hipSuccess) {
    (void)hipGetLastError();
    return n;
  }
  int c = 0;
  for (uint32_t m : mask) c += __builtin_popcount(m);
  return c > 0 && c < n ? c : n;
}

// Workgroups of kernel k that fit on one multiprocessor at once (the
// occupancy the compiled kernel allows), cached by the caller.
template <typename Kern>
static int blocks_per_cu(Kern k, int threads, size_t lds, std::atomic<int>& cache) {
  int b = cache.load(std::memory_order_relaxed);
  if (b < 0) {
    b = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, k, threads, lds) != hipSuccess) {
      (void)hipGetLastError();
      b = 0;
    }
    cache.store(b, std::memory_order_relaxed);
  }
  return b;
}

// Whole rounds of waves. The walk's waves (chunks x column tiles) of equal
// cost run in rounds of as many waves as fit at once on the compute units
// the launch's stream may use. Where a
// last round would be less than half full, its few waves run nearly alone,
// far below the memory system's rate: the chunk count then grows (so the
// chunks shrink) until the last round is full, at most to the workspace's
// capacity (a chunk count above the minimum only shortens chunks).
// Measured at K = 1,048,576, D = 2048 fp32 (two column tiles, room for
// 2,048 waves): 2,088 chunks (4,176 waves) 1,591 us, 3,072 chunks 1,488 us.
// Where the last round was half full or more (the bf16 merge: 10,347 waves
// on room for 4,096) rounding up changed nothing measurable, and inputs of
// less than one round are left as they are (more chunks made the 2M
// vocabulary 2% slower).
static int whole_rounds(int nchunks, int tiles, int64_t waves_per_round, int max_chunks) {
  if (waves_per_round <= 0 || tiles <= 0) return nchunks;
  const int64_t waves = int64_t(nchunks) * tiles;
  const int64_t last = waves % waves_per_round;
  if (waves <= waves_per_round || last == 0 || 2 * last >= waves_per_round) return nchunks;
  const int64_t rounds = (waves + waves_per_round - 1) / waves_per_round;
  int64_t n = (rounds * waves_per_round + tiles - 1) / tiles;
  if (n > max_chunks) n = max_chunks;
  return static_cast<int>(n < nchunks ? nchunks : n);
}

template <typename GT, int VEC, int NV, int R, int OP>
static void launch_one(SegArgs& a, int tiles, hipStream_t st) {
  constexpr int RFp = rf_for<NV, R>(), T = t_for<R>();
  constexpr int RF = OP == kOpSgd ? rf_sgd_for<NV, R>() : OP == kOpAdam ? rf_adam_for<NV, R>() : RFp;
  a.tiles = tiles;
  a.tile_cols = NV * kWave * VEC;
  // The rounds are those of the plain kernel (kOpStore) for the update
  // instantiations too: its occupancy fixes the chunks, and with them the
  // order of every sum, so lm_segsum_sgd and _adam add in lm_segsum's order.
  if constexpr (VEC >= 2) {
    if (a.fused) {
      auto k = k_segsum<GT, VEC, NV, RF, R, T, kFusedThreads, true, OP>;
      static std::atomic<int> bpc{-1};
      const int64_t room =
          int64_t(blocks_per_cu(k_segsum<GT, VEC, NV, RFp, R, T, kFusedThreads, true, kOpStore>,
                                kFusedThreads, 0, bpc)) *
          kFusedWaves * stream_cus(st);
      a.nchunks = whole_rounds(a.nchunks, tiles, room, a.max_chunks);
      a.main_blocks = (a.nchunks + kFusedWaves - 1) / kFusedWaves * tiles;
      const int fix_blocks = (a.nchunks + kFusedSpan - 1) / kFusedSpan * a.fix_tiles;
      k<<<dim3(a.main_blocks + fix_blocks), kFusedThreads, 0, st>>>(a);
      return;
    }
  }
  auto k = k_segsum<GT, VEC, NV, RF, R, T, kSegThreads, false, OP>;
  static std::atomic<int> bpc{-1};
  const int64_t room =
      int64_t(blocks_per_cu(k_segsum<GT, VEC, NV, RFp, R, T, kSegThreads, false, kOpStore>,
                            kSegThreads, LMZ_SEG_LDS_PAD, bpc)) *
      kSegWaves * stream_cus(st);
  a.nchunks = whole_rounds(a.nchunks, tiles, room, a.max_chunks);
  const dim3 grid((a.nchunks + kSegWaves - 1) / kSegWaves, tiles);
  k<<<grid, kSegThreads, LMZ_SEG_LDS_PAD, st>>>(a);
}

template <typename GT, int VEC, int NV, int OP>
static hipError_t launch_r(SegArgs& a, hipStream_t st) {
  constexpr int CT = NV * kWave * VEC;
  const int tiles = (a.D + CT - 1) / CT;
  switch (a.R) {
    case 16: launch_one<GT, VEC, NV, 16, OP>(a, tiles, st); break;
    case 32: launch_one<GT, VEC, NV, 32, OP>(a, tiles, st); break;
    case 64: launch_one<GT, VEC, NV, 64, OP>(a, tiles, st); break;
    case 128: launch_one<GT, VEC, NV, 128, OP>(a, tiles, st); break;
    case 256: launch_one<GT, VEC, NV, 256, OP>(a, tiles, st); break;
    default: launch_one<GT, VEC, NV, 512, OP>(a, tiles, st); break;
  }
  return hipGetLastError();
}

template <typename GT, int VEC, int OP>
static hipError_t dispatch_nv(SegArgs& a, int nv_max, hipStream_t st) {
  const int per = kWave * VEC;
  int nv = (a.D + per - 1) / per;
  if (nv > nv_max) nv = nv_max;
  if (nv <= 1) return launch_r<GT, VEC, 1, OP>(a, st);
  if (nv == 2) return launch_r<GT, VEC, 2, OP>(a, st);
  if constexpr (sizeof(GT) == 4 || VEC == 1) return launch_r<GT, VEC, 4, OP>(a, st);
  return launch_r<GT, VEC, 2, OP>(a, st);
}

template <int OP>
static hipError_t dispatch(SegArgs& a, int gtype, bool vec, hipStream_t st) {
  if (gtype == LM_F32)
    return vec ? dispatch_nv<float, 4, OP>(a, LMZ_SEG_NV_MAX, st)
               : dispatch_nv<float, 1, OP>(a, 4, st);
  return vec ? dispatch_nv<bf16_t, 8, OP>(a, LMZ_SEG_NV_MAX < 2 ? LMZ_SEG_NV_MAX : 2, st)
             : dispatch_nv<bf16_t, 1, OP>(a, 4, st);
}

template <int OP>
static void launch_fix(SegArgs& a, hipStream_t st) {
  const uint32_t fix_blocks = static_cast<uint32_t>((a.nchunks + kFixChunks - 1) / kFixChunks);
  if (a.D % 4 == 0)
    k_segsum_fix<4, LMZ_SEG_FIX_RF, OP>
        <<<dim3(fix_blocks, (a.D + 255) / 256), kFixThreads, 0, st>>>(a);
  else
    k_segsum_fix<1, LMZ_SEG_FIX_RF, OP>
        <<<dim3(fix_blocks, (a.D + 63) / 64), kFixThreads, 0, st>>>(a);
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// Test hook for the failure path of the one-launch form: while set, the
// fix-up workgroups wait for a flag value that no walk writes, so every such
// wait gives up after `limit` polls and raises LM_DEVERR_SPIN; the launch
// still drains and stays inside its buffers. Off by default.
static std::atomic<bool> g_force_wait_failure{false};
static std::atomic<uint32_t> g_forced_spin_limit{kSpinLimit};

void segsum_force_wait_failure(bool enable, uint32_t limit) {
  g_forced_spin_limit.store(limit < 1 ? 1u : limit, std::memory_order_relaxed);
  g_force_wait_failure.store(enable, std::memory_order_relaxed);
}

// The host switch to the two-launch form (lm_segsum_set_two_launches):
// -1 until the first call reads LMZIPF_SEGSUM_TWO_LAUNCHES, then 0 or 1.
static std::atomic<int> g_two_launches{-1};

static bool two_launches() {
  int v = g_two_launches.load(std::memory_order_relaxed);
  if (v < 0) {
    const char* e = std::getenv("LMZIPF_SEGSUM_TWO_LAUNCHES");
    const int from_env = (e && e[0] == '1') ? 1 : 0;
    int expected = -1;
    g_two_launches.compare_exchange_strong(expected, from_env, std::memory_order_relaxed);
    v = g_two_launches.load(std::memory_order_relaxed);
  }
  return v == 1;
}

int segsum_set_two_launches(bool enable) {
  const int prev = two_launches() ? 1 : 0;
  g_two_launches.store(enable ? 1 : 0, std::memory_order_relaxed);
  return prev;
}

int segsum_run(const void* grad, int gtype, int64_t K, int64_t D, int64_t ld_grad,
               const int32_t* perm, const int32_t* inverse, const int32_t* offsets,
               const int64_t* num_unique, int64_t u_cap, float* out, int64_t ld_out,
               int32_t* dev_err, void* ws, size_t ws_bytes, hipStream_t st,
               const void* row_ids, int row_ids64, int64_t out_rows, int op,
               const OptParams& opt, float* m, float* v) {
  const SegLayout L = seg_layout(K, D);
  if (ws_bytes < L.total) return LM_E_WORKSPACE;
  if (K == 0 || D == 0 || u_cap == 0) return LM_OK;
  char* w = static_cast<char*>(ws);
  SegArgs a{};
  a.spin_limit = kSpinLimit;
  a.grad = grad;
  a.ld_grad = ld_grad;
  a.K = static_cast<int>(K);
  a.D = static_cast<int>(D);
  a.perm = perm;
  a.inverse = inverse;
  a.offsets = offsets;
  a.num_unique = num_unique;
  a.u_cap = u_cap;
  a.out = out;
  a.ld_out = ld_out;
  a.row_ids = row_ids;
  a.row_ids64 = row_ids64;
  a.out_rows = row_ids ? out_rows : u_cap;
  a.part_cont = reinterpret_cast<float*>(w + L.cont);
  a.part_start = reinterpret_cast<float*>(w + L.start);
  a.desc = reinterpret_cast<int32_t*>(w + L.desc);
  a.npieces = reinterpret_cast<int32_t*>(w + L.npieces);
  a.R = L.R;
  a.rw = read_cost(gtype);
  a.ww = write_cost(gtype);
  a.nchunks = static_cast<int>(chunks_for(K, L.R, a.rw, a.ww, u_cap));
  a.max_chunks = L.max_chunks;
  a.dev_err = dev_err;
  a.opt = opt;
  a.m = m;
  a.v = v;

  const bool out_vec = al16(out) && ld_out % 4 == 0 && D % 4 == 0;
  const bool vec = gtype == LM_F32 ? out_vec && al16(grad) && ld_grad % 4 == 0
                                   : out_vec && al16(grad) && ld_grad % 8 == 0 && D % 8 == 0;
  // One launch for the walk and the fix-up on the vector path. Measured at
  // K = 1,048,576, D = 2048 fp32 (two column tiles): 1,490 us as the walk
  // and a separate fix-up kernel, 1,411 us in one launch, the fix-up
  // workgroups running in the walk's last round.
  a.fused = LMZ_SEG_FUSED != 0 && vec && D <= LMZ_SEG_FUSED_MAX_D &&
            (LMZ_SEG_NV_MAX >= 4 || gtype != LM_F32) && !two_launches();
  // A captured launch would replay with this call's epoch every time, and a
  // replay could take the previous replay's flags for its own: under stream
  // capture the fix-up is a second launch, which keeps no state across calls.
  if (a.fused) {
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone) {
      (void)hipGetLastError();
      a.fused = 0;
    }
  }
  if (a.fused) {
    static std::atomic<uint64_t> epoch{0x9e3779b97f4a7c15ull};
    a.flags = reinterpret_cast<uint64_t*>(w + L.flags);
    a.epoch = epoch.fetch_add(1, std::memory_order_relaxed) + 1;
    const bool fail = g_force_wait_failure.load(std::memory_order_relaxed);
    a.wait_epoch = fail ? a.epoch ^ (uint64_t(1) << 63) : a.epoch;
    a.spin_limit = fail ? g_forced_spin_limit.load(std::memory_order_relaxed) : kSpinLimit;
    a.fix_tiles = static_cast<int>((D + kFusedCols - 1) / kFusedCols);
  }
  const hipError_t e = op == kOpSgd    ? dispatch<kOpSgd>(a, gtype, vec, st)
                       : op == kOpAdam ? dispatch<kOpAdam>(a, gtype, vec, st)
                                       : dispatch<kOpStore>(a, gtype, vec, st);
  if (e != hipSuccess) return launch_status(e);
  if (a.fused) return LM_OK;
  if (op == kOpSgd) launch_fix<kOpSgd>(a, st);
  else if (op == kOpAdam) launch_fix<kOpAdam>(a, st);
  else launch_fix<kOpStore>(a, st);
  return launch_status(hipGetLastError());
}

}  // namespace lmz
