// Seg-Sum (Sec. III-A step 2): out[u, :] = sum of grad[perm[i], :] over the
// sorted positions i of type u, accumulated in fp32 in a fixed order.
//
// Work partition (no float atomics, run-to-run bit-identical):
//   The K sorted positions are cut into chunks of R positions, one chunk per
//   wave (and per column tile of up to 1024 columns). A segment (the
//   positions of one type) shorter than kLongRows rows belongs entirely to
//   the chunk that holds its first position, even when it runs past the
//   chunk end; a longer one — the heads of the Zipf distribution — is cut at
//   chunk boundaries, each chunk summing its piece into a partial row:
//     part_start[c]  the piece of a long segment that starts in chunk c and
//                    continues past it (desc[c] names that segment),
//     part_cont[c]   the piece of a long segment that started before chunk c.
//   k_segsum_fix then adds, for every desc[c] >= 0, part_start[c] and the
//   part_cont rows of the following chunks the segment covers, in chunk
//   order. A chunk therefore reads at most R + kLongRows - 1 rows, and a
//   head holding 20% of a million tokens is spread over ~400 waves.
//   Each wave gathers whole 16-byte column vectors of RF rows at a time
//   (RF x NV x 1 KiB in flight), adds them in fp32 registers and writes a row
//   as soon as its segment ends; grad is streamed with non-temporal loads.
#include "common.hpp"

namespace lmz {

constexpr int kSegThreads = 256;
constexpr int kSegWaves = kSegThreads / kWave;
constexpr int kLongRows = 64;
constexpr int kTargetChunks = 2048;

struct SegArgs {
  const void* grad;
  int64_t ld_grad;
  int K, D;
  const int32_t* perm;
  const int32_t* offsets;
  const int64_t* num_unique;
  int64_t u_cap;
  float* out;
  int64_t ld_out;
  float* part_cont;
  float* part_start;
  int32_t* desc;
  int R, nchunks;
  int32_t* dev_err;
};

struct SegLayout {
  int R, nchunks;
  size_t cont, start, desc, total;
};

static inline size_t a256(size_t x) { return (x + 255) & ~size_t(255); }

static SegLayout seg_layout(int64_t K, int64_t D) {
  SegLayout L{};
  int64_t r = (K + kTargetChunks - 1) / kTargetChunks;
  r = (r + 63) / 64 * 64;
  L.R = static_cast<int>(r < 64 ? 64 : r);
  L.nchunks = static_cast<int>((K + L.R - 1) / L.R);
  size_t off = LM_UNIQUE_CTRL_BYTES;  // reserved for lm_unique's control block
  L.cont = off;  off += a256(size_t(L.nchunks) * D * 4);
  L.start = off; off += a256(size_t(L.nchunks) * D * 4);
  L.desc = off;  off += a256(size_t(L.nchunks) * 4);
  L.total = off;
  return L;
}

size_t segsum_workspace_bytes(int64_t K, int64_t D) { return seg_layout(K, D).total; }

// Largest s in [0, U) with offsets[s] <= target (offsets ascending, offsets[0]
// = 0). A 64-ary search by the whole wave: ceil(log64 U) dependent loads.
__device__ __forceinline__ int seg_search(const int32_t* __restrict__ offsets, int U, int target) {
  const int lane = lane_id();
  int lo = 0, hi = U;
  while (hi - lo > 1) {
    const int stride = (hi - lo + kWave - 1) / kWave;
    const int idx = lo + lane * stride;
    const bool pred = idx < hi && offsets[idx] <= target;
    int t = __popcll(ballot(pred));
    if (t < 1) t = 1;  // only reachable with non-monotone offsets
    const int nlo = lo + (t - 1) * stride;
    const int nhi = lo + t * stride;
    lo = nlo;
    hi = nhi < hi ? nhi : hi;
  }
  return lo;
}

template <typename GT, int VEC, int NV, int RF>
__global__ __launch_bounds__(kSegThreads) void k_segsum(SegArgs a) {
  using RV = RowVec<GT, VEC>;
  using raw_t = typename RV::raw_t;
  constexpr int kColsPerVec = kWave * VEC;
  constexpr int CT = NV * kColsPerVec;

  const int lane = lane_id();
  const int c = blockIdx.x * kSegWaves + (threadIdx.x >> 6);
  if (c >= a.nchunks) return;
  const int ct = blockIdx.y;
  const int K = a.K, D = a.D, R = a.R;

  int64_t U64 = *a.num_unique;
  if (U64 > a.u_cap) {
    if (c == 0 && ct == 0 && lane == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
  }
  const int U = static_cast<int>(U64 < K ? U64 : K);
  const int p0 = c * R;
  const int p1 = p0 + R < K ? p0 + R : K;
  if (U <= 0 || p0 >= K) {
    if (ct == 0 && lane == 0) a.desc[c] = -1;
    return;
  }
  const int32_t* __restrict__ offsets = a.offsets;
  const int32_t* __restrict__ perm = a.perm;

  const int s_f = seg_search(offsets, U, p0);
  const int s_l = seg_search(offsets, U, p1 - 1);
  const int a_f = offsets[s_f], b_f = offsets[s_f + 1];
  const int a_l = offsets[s_l], b_l = offsets[s_l + 1];
  const bool long_l = b_l - a_l >= kLongRows;
  int s = s_f, q = p0;
  if (a_f < p0 && b_f - a_f < kLongRows) {
    s = s_f + 1;  // a short segment owned by the previous chunk
    q = b_f;
  }
  int q_end = long_l ? p1 : b_l;
  if (q_end > K) q_end = K;
  if (ct == 0 && lane == 0) a.desc[c] = (long_l && a_l >= p0 && b_l > p1) ? s_l : -1;
  if (q >= q_end) return;

  // Columns of this lane.
  const int col0 = ct * CT + lane * VEC;
  bool col_ok[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) col_ok[v] = col0 + v * kColsPerVec < D;

  const GT* __restrict__ grad = static_cast<const GT*>(a.grad) + col0;

  // Windows: perm_cur/perm_nxt hold perm[pw .. pw+128); ends holds
  // offsets[ow+1 .. ow+65) (the end of segments ow .. ow+63).
  int pw = q;
  int perm_cur = pw + lane < K ? perm[pw + lane] : 0;
  int perm_nxt = pw + kWave + lane < K ? perm[pw + kWave + lane] : 0;
  int ow = s;
  int ends = ow + 1 + lane <= U ? offsets[ow + 1 + lane] : K;

  int seg_a = s < U ? offsets[s] : K;
  int seg_b = s < U ? read_lane(ends, 0) : K;
  int run_end = seg_b < q_end ? seg_b : q_end;

  float acc[NV][VEC];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[v][e] = 0.f;

  bool bad_row = false;
  while (q < q_end) {
    const int n = q_end - q < RF ? q_end - q : RF;
    raw_t buf[RF][NV];
#pragma unroll
    for (int r = 0; r < RF; ++r) {
      if (r < n) {
        const int idx = q + r - pw;
        int k = idx < kWave ? read_lane(perm_cur, idx) : read_lane(perm_nxt, idx - kWave);
        if (static_cast<uint32_t>(k) >= static_cast<uint32_t>(K)) { bad_row = true; k = 0; }
        const GT* row = grad + static_cast<int64_t>(k) * a.ld_grad;
#pragma unroll
        for (int v = 0; v < NV; ++v)
          if (col_ok[v]) buf[r][v] = RV::load(row + v * kColsPerVec);
          else buf[r][v] = raw_t{};
      }
    }
#pragma unroll
    for (int r = 0; r < RF; ++r) {
      if (r < n) {
#pragma unroll
        for (int v = 0; v < NV; ++v) RV::add(acc[v], buf[r][v]);
        if (q + r + 1 == run_end) {
          // Segment s (or its piece in this chunk) is complete.
          const bool is_long = seg_b - seg_a >= kLongRows;
          float* dst;
          if (is_long && seg_a < p0) dst = a.part_cont + static_cast<int64_t>(c) * D;
          else if (is_long && seg_b > p1) dst = a.part_start + static_cast<int64_t>(c) * D;
          else dst = s < a.u_cap ? a.out + static_cast<int64_t>(s) * a.ld_out : nullptr;
          if (dst) {
#pragma unroll
            for (int v = 0; v < NV; ++v)
              if (col_ok[v]) store_vec<VEC>(dst + col0 + v * kColsPerVec, acc[v]);
          }
#pragma unroll
          for (int v = 0; v < NV; ++v)
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[v][e] = 0.f;
          ++s;
          if (s < U) {
            seg_a = seg_b;
            if (s - ow >= kWave) {
              ow = s;
              ends = ow + 1 + lane <= U ? offsets[ow + 1 + lane] : K;
            }
            seg_b = read_lane(ends, s - ow);
          } else {
            seg_a = seg_b = K;
          }
          run_end = seg_b < q_end ? seg_b : q_end;
        }
      }
    }
    q += n;
    if (q - pw >= kWave) {
      pw += kWave;
      perm_cur = perm_nxt;
      perm_nxt = pw + kWave + lane < K ? perm[pw + kWave + lane] : 0;
    }
  }
  if (ballot(bad_row) && lane == 0) raise_err(a.dev_err, LM_DEVERR_CAPACITY);
}

// Sum the pieces of every long segment that spans chunks, in chunk order.
// One wave per (starting chunk, 64*VEC columns).
template <int VEC, int RF>
__global__ __launch_bounds__(kSegThreads) void k_segsum_fix(SegArgs a) {
  const int lane = lane_id();
  const int c = blockIdx.x * kSegWaves + (threadIdx.x >> 6);
  if (c >= a.nchunks) return;
  const int s = a.desc[c];
  if (s < 0) return;
  const int U = static_cast<int>(*a.num_unique);
  if (s >= U) return;
  const int b = a.offsets[s + 1];
  int c1 = (b - 1) / a.R;
  if (c1 >= a.nchunks) c1 = a.nchunks - 1;
  const int D = a.D;
  const int col = blockIdx.y * (kWave * VEC) + lane * VEC;
  if (col >= D) return;
  float acc[VEC];
  load_vec<VEC>(a.part_start + static_cast<int64_t>(c) * D + col, acc);
  for (int cc = c + 1; cc <= c1; cc += RF) {
    float buf[RF][VEC];
#pragma unroll
    for (int r = 0; r < RF; ++r)
      if (cc + r <= c1) load_vec<VEC>(a.part_cont + static_cast<int64_t>(cc + r) * D + col, buf[r]);
#pragma unroll
    for (int r = 0; r < RF; ++r)
      if (cc + r <= c1)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += buf[r][e];
  }
  if (s < a.u_cap) store_vec<VEC>(a.out + static_cast<int64_t>(s) * a.ld_out + col, acc);
}

template <typename GT, int VEC, int NV, int RF>
static hipError_t launch_main(const SegArgs& a, hipStream_t st) {
  constexpr int CT = NV * kWave * VEC;
  dim3 grid((a.nchunks + kSegWaves - 1) / kSegWaves, (a.D + CT - 1) / CT);
  k_segsum<GT, VEC, NV, RF><<<grid, kSegThreads, 0, st>>>(a);
  return hipGetLastError();
}

template <typename GT, int VEC>
static hipError_t dispatch_nv(const SegArgs& a, int nv_max, hipStream_t st) {
  const int per = kWave * VEC;
  int nv = (a.D + per - 1) / per;
  if (nv > nv_max) nv = nv_max;
  if (nv <= 1) return launch_main<GT, VEC, 1, 8>(a, st);
  if (nv == 2) return launch_main<GT, VEC, 2, 8>(a, st);
  if constexpr (sizeof(GT) == 4 || VEC == 1) return launch_main<GT, VEC, 4, 4>(a, st);
  return launch_main<GT, VEC, 2, 8>(a, st);
}

static bool al16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

int segsum_run(const void* grad, int gtype, int64_t K, int64_t D, int64_t ld_grad,
               const int32_t* perm, const int32_t* offsets, const int64_t* num_unique,
               int64_t u_cap, float* out, int64_t ld_out, int32_t* dev_err, void* ws,
               size_t ws_bytes, hipStream_t st) {
  const SegLayout L = seg_layout(K, D);
  if (ws_bytes < L.total) return LM_E_WORKSPACE;
  if (K == 0 || D == 0 || u_cap == 0) return LM_OK;
  char* w = static_cast<char*>(ws);
  SegArgs a{};
  a.grad = grad;
  a.ld_grad = ld_grad;
  a.K = static_cast<int>(K);
  a.D = static_cast<int>(D);
  a.perm = perm;
  a.offsets = offsets;
  a.num_unique = num_unique;
  a.u_cap = u_cap;
  a.out = out;
  a.ld_out = ld_out;
  a.part_cont = reinterpret_cast<float*>(w + L.cont);
  a.part_start = reinterpret_cast<float*>(w + L.start);
  a.desc = reinterpret_cast<int32_t*>(w + L.desc);
  a.R = L.R;
  a.nchunks = L.nchunks;
  a.dev_err = dev_err;

  const bool out_vec = al16(out) && ld_out % 4 == 0 && D % 4 == 0;
  hipError_t e;
  if (gtype == LM_F32) {
    const bool vec = out_vec && al16(grad) && ld_grad % 4 == 0;
    e = vec ? dispatch_nv<float, 4>(a, 4, st) : dispatch_nv<float, 1>(a, 4, st);
  } else {
    const bool vec = out_vec && al16(grad) && ld_grad % 8 == 0 && D % 8 == 0;
    e = vec ? dispatch_nv<bf16_t, 8>(a, 2, st) : dispatch_nv<bf16_t, 1>(a, 4, st);
  }
  if (e != hipSuccess) return launch_status(e);

  if (D % 4 == 0) {
    dim3 grid((L.nchunks + kSegWaves - 1) / kSegWaves, (a.D + 255) / 256);
    k_segsum_fix<4, 16><<<grid, kSegThreads, 0, st>>>(a);
  } else {
    dim3 grid((L.nchunks + kSegWaves - 1) / kSegWaves, (a.D + 63) / 64);
    k_segsum_fix<1, 16><<<grid, kSegThreads, 0, st>>>(a);
  }
  return launch_status(hipGetLastError());
}

}  // namespace lmz
