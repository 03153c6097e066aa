// Unique (Sec. III-A steps 1 and 4): the distinct word indices of a batch in
// ascending order, with counts, CSR offsets, the token->type map and the
// stable sort permutation.
//
// Pipeline (all on one stream, no host sync):
//   k_hist      digit histograms of every radix pass in one read of the ids;
//               also clears this call's look-back status words and tickets.
//   k_onesweep  one LSD radix pass per 8-bit digit over only ceil(log2 V) key
//               bits: each 256-thread workgroup ranks a tile of keys with
//               wave64 ballot matching, gets its global digit offsets through
//               a decoupled look-back over tile status words, reorders the
//               tile in LDS and writes it out in digit runs.
//   k_dedup     run-head flags on the sorted keys, a block scan plus a
//               decoupled look-back that carries (number of heads, position of
//               the last head), and writes uniq, offsets, counts, inverse and
//               num_unique; it also re-zeroes the histogram control block.
// Tiles take their index from an atomic ticket, so a tile only ever waits on
// tiles that already hold a workgroup: the look-back always makes progress.
#include "common.hpp"

namespace lmz {

constexpr int kSortThreads = 256;
constexpr int kSortWaves = kSortThreads / kWave;
constexpr int kRadix = 256;
constexpr int kMaxPasses = 8;             // 64-bit keys
constexpr int kSortItems = 16;            // keys per thread in a sort tile
constexpr int kSortTile = kSortThreads * kSortItems;
constexpr int kDedupItems = 16;
constexpr int kDedupTile = kSortThreads * kDedupItems;

// Status words of the sort look-back: 2-bit flag | 30-bit count.
constexpr uint32_t kFlagAgg = 1u << 30, kFlagPrefix = 2u << 30, kValMask = (1u << 30) - 1;
// Status words of the dedup look-back: flag (2) | heads (31) | last head + 1 (31).
constexpr uint64_t kDFlagAgg = 1ull << 62, kDFlagPrefix = 2ull << 62;
constexpr uint64_t kD31 = (1ull << 31) - 1;

struct UniqueLayout {
  size_t hist, tickets, status, dstatus, keys0, keys1, vals0, vals1, total;
  int passes, bits, tiles, dtiles;
};

static inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

static inline int key_bits_for(int64_t V) {
  if (V <= 1) return 0;
  uint64_t m = static_cast<uint64_t>(V - 1);
  return 64 - __builtin_clzll(m);
}

static UniqueLayout unique_layout(int64_t K, int idtype, int64_t V) {
  UniqueLayout L{};
  const size_t ks = idtype == LM_I64 ? 8 : 4;
  L.bits = key_bits_for(V);
  L.passes = L.bits == 0 ? 1 : (L.bits + 7) / 8;
  L.tiles = static_cast<int>((K + kSortTile - 1) / kSortTile);
  L.dtiles = static_cast<int>((K + kDedupTile - 1) / kDedupTile);
  size_t off = 0;
  L.hist = off;    off += LM_UNIQUE_CTRL_BYTES;                      // zero between calls
  L.tickets = off; off += 256;
  L.status = off;  off += align256(size_t(L.passes) * L.tiles * kRadix * 4);
  L.dstatus = off; off += align256(size_t(L.dtiles) * 8);
  L.keys0 = off;   off += align256(size_t(K) * ks);
  L.keys1 = off;   off += align256(size_t(K) * ks);
  L.vals0 = off;   off += align256(size_t(K) * 4);
  L.vals1 = off;   off += align256(size_t(K) * 4);
  L.total = off;
  return L;
}

// ---------------------------------------------------------------------------
// k_hist
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ __launch_bounds__(kSortThreads) void k_hist(
    const KeyT* __restrict__ keys, int K, uint64_t V, int passes, int bits,
    uint32_t* __restrict__ hist, uint32_t* __restrict__ clear, int64_t clear_words,
    int32_t* __restrict__ dev_err) {
  __shared__ uint32_t sh[kMaxPasses][kRadix];
  for (int i = threadIdx.x; i < kMaxPasses * kRadix; i += kSortThreads) (&sh[0][0])[i] = 0;
  // Clear this call's look-back status words and tile tickets.
  for (int64_t i = blockIdx.x * int64_t(kSortThreads) + threadIdx.x; i < clear_words;
       i += int64_t(gridDim.x) * kSortThreads)
    clear[i] = 0;
  __syncthreads();
  bool bad = false;
  for (int64_t i = blockIdx.x * int64_t(kSortThreads) + threadIdx.x; i < K;
       i += int64_t(gridDim.x) * kSortThreads) {
    const uint64_t kb = key_bits(keys[i]);
    bad |= kb >= V;
    for (int p = 0; p < passes; ++p) {
      const int shift = 8 * p;
      const int nb = bits - shift < 8 ? bits - shift : 8;
      const uint32_t d = nb > 0 ? static_cast<uint32_t>(kb >> shift) & ((1u << nb) - 1) : 0u;
      atomicAdd(&sh[p][d], 1u);
    }
  }
  if (ballot(bad) && lane_id() == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
  __syncthreads();
  for (int i = threadIdx.x; i < passes * kRadix; i += kSortThreads) {
    const uint32_t c = (&sh[0][0])[i];
    if (c) add_agent(&hist[i], c);
  }
}

// ---------------------------------------------------------------------------
// k_onesweep: one stable LSD pass over the digit (key >> shift) & (2^nbits-1).
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ __launch_bounds__(kSortThreads) void k_onesweep(
    const KeyT* __restrict__ keys_in, const int32_t* __restrict__ vals_in,
    KeyT* __restrict__ keys_out, int32_t* __restrict__ vals_out, int K, int shift, int nbits,
    const uint32_t* __restrict__ hist, uint32_t* __restrict__ status,
    uint32_t* __restrict__ ticket, int32_t* __restrict__ dev_err) {
  __shared__ KeyT s_keys[kSortTile];
  __shared__ int32_t s_vals[kSortTile];
  __shared__ uint32_t s_cnt[kSortWaves][kRadix];  // per-wave digit counts, then offsets
  __shared__ int32_t s_local[kRadix];             // tile-local start of each digit
  __shared__ int32_t s_shift[kRadix];             // global position - local position
  __shared__ uint32_t s_scan[4];
  __shared__ uint32_t s_tile;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) s_tile = add_agent(ticket, 1u);
  for (int i = tid; i < kSortWaves * kRadix; i += kSortThreads) (&s_cnt[0][0])[i] = 0;
  __syncthreads();
  const int tile = static_cast<int>(s_tile);
  const int64_t base = int64_t(tile) * kSortTile;
  const uint32_t mask = nbits > 0 ? (1u << nbits) - 1 : 0u;

  // Wave w owns tile items [w*16*64, (w+1)*16*64); item i of a lane is
  // base + w*1024 + i*64 + lane, so (wave, i, lane) order is position order.
  KeyT key[kSortItems];
  int32_t val[kSortItems];
  uint32_t dig[kSortItems];
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const int64_t pos = base + int64_t(wave) * (kSortItems * kWave) + i * kWave + lane;
    const bool ok = pos < K;
    key[i] = ok ? keys_in[pos] : KeyT(0);
    val[i] = ok ? (vals_in ? vals_in[pos] : static_cast<int32_t>(pos)) : 0;
    dig[i] = ok ? static_cast<uint32_t>(key_bits(key[i]) >> shift) & mask : kRadix;
  }

  // Rank every key among the equal-digit keys before it in its wave.
  uint32_t rank[kSortItems];
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    const bool ok = dig[i] < kRadix;
    uint64_t peers = ballot(ok);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (dig[i] >> b) & 1u;
      const uint64_t bb = ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    uint32_t prior = 0;
    if (ok) prior = s_cnt[wave][dig[i]];
    rank[i] = prior + popc_below(peers);
    if (ok && popc_below(peers) == 0) s_cnt[wave][dig[i]] = prior + __popcll(peers);
  }
  __syncthreads();

  // Thread d: per-wave exclusive offsets of digit d, tile total of digit d.
  const int d = tid;
  uint32_t tot = 0;
#pragma unroll
  for (int w = 0; w < kSortWaves; ++w) {
    const uint32_t c = s_cnt[w][d];
    s_cnt[w][d] = tot;
    tot += c;
  }
  uint32_t tile_sum;
  const uint32_t local = block256_excl_sum<uint32_t>(tot, s_scan, tile_sum);
  uint32_t hist_sum;
  const uint32_t gbase = block256_excl_sum<uint32_t>(hist[d], s_scan, hist_sum);
  s_local[d] = static_cast<int32_t>(local);

  // Decoupled look-back for digit d.
  uint32_t* my = status + size_t(tile) * kRadix + d;
  uint32_t excl = 0;
  if (tile == 0) {
    st_agent(my, kFlagPrefix | tot);
  } else {
    st_agent(my, kFlagAgg | tot);
    int j = tile - 1;
    uint32_t spins = 0;
    while (true) {
      const uint32_t s = ld_agent(status + size_t(j) * kRadix + d);
      const uint32_t f = s & ~kValMask;
      if (f == 0) {
        if (++spins > kSpinLimit) { raise_err(dev_err, LM_DEVERR_SPIN); break; }
        __builtin_amdgcn_s_sleep(1);
        continue;
      }
      excl += s & kValMask;
      if (f == kFlagPrefix || j == 0) break;
      --j;
    }
    st_agent(my, kFlagPrefix | ((excl + tot) & kValMask));
  }
  s_shift[d] = static_cast<int32_t>(gbase + excl) - static_cast<int32_t>(local);
  __syncthreads();

  // Reorder the tile in LDS by digit (stable), then write digit runs out.
#pragma unroll
  for (int i = 0; i < kSortItems; ++i) {
    if (dig[i] < kRadix) {
      const int lp = s_local[dig[i]] + static_cast<int>(s_cnt[wave][dig[i]] + rank[i]);
      s_keys[lp] = key[i];
      s_vals[lp] = val[i];
    }
  }
  __syncthreads();
  const int n = static_cast<int>(K - base < kSortTile ? K - base : kSortTile);
  for (int j = tid; j < n; j += kSortThreads) {
    const KeyT k = s_keys[j];
    const uint32_t dd = static_cast<uint32_t>(key_bits(k) >> shift) & mask;
    const int gp = s_shift[dd] + j;
    // Only a failed look-back (LM_DEVERR_SPIN already raised) leaves gp out
    // of range; never write outside the buffers.
    if (static_cast<uint32_t>(gp) < static_cast<uint32_t>(K)) {
      keys_out[gp] = k;
      vals_out[gp] = s_vals[j];
    }
  }
}

// ---------------------------------------------------------------------------
// k_dedup
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ __launch_bounds__(kSortThreads) void k_dedup(
    const KeyT* __restrict__ skeys, const int32_t* __restrict__ perm, int K, int cap,
    KeyT* __restrict__ uniq, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ inverse, int64_t* __restrict__ num_unique,
    uint64_t* __restrict__ status, uint32_t* __restrict__ ticket,
    uint32_t* __restrict__ hist, int hist_words, int32_t* __restrict__ dev_err) {
  __shared__ KeyT s_keys[kDedupTile + 2];  // [0]: key before the tile, [n+1]: key after
  __shared__ uint32_t s_scan[4];
  __shared__ int s_maxs[4];
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_excl_heads;
  __shared__ int s_excl_last;

  const int tid = threadIdx.x;
  if (tid == 0) s_tile = add_agent(ticket, 1u);
  __syncthreads();
  const int tile = static_cast<int>(s_tile);
  const int64_t base = int64_t(tile) * kDedupTile;
  const int n = static_cast<int>(K - base < kDedupTile ? K - base : kDedupTile);

  // The histogram control block is no longer needed by this call: leave it
  // zero for the next one.
  if (tile == 0)
    for (int i = tid; i < hist_words; i += kSortThreads) hist[i] = 0;

  for (int j = tid; j < n; j += kSortThreads) s_keys[j + 1] = skeys[base + j];
  if (tid == 0) s_keys[0] = base > 0 ? skeys[base - 1] : KeyT(0);
  if (tid == 1) s_keys[n + 1] = base + n < K ? skeys[base + n] : KeyT(0);
  __syncthreads();

  // Thread t owns positions base + t*16 + i. Run heads and tails become
  // bit masks first (bit i: item i), evaluated without short-circuit
  // branches: ROCm 7.2's compiler dropped `last = p` on the branchy form
  // of this loop when the head was a thread's first item.
  const int first = tid * kDedupItems;
  uint32_t hmask = 0, tmask = 0;
#pragma unroll
  for (int i = 0; i < kDedupItems; ++i) {
    const int j = first + i;
    if (j < n) {
      const int64_t p = base + j;
      const KeyT k = s_keys[j + 1];
      const bool head = (p == 0) | (k != s_keys[j]);
      const bool tail = (p == K - 1) | (s_keys[j + 2] != k);
      hmask |= static_cast<uint32_t>(head) << i;
      tmask |= static_cast<uint32_t>(tail) << i;
    }
  }
  const uint32_t nheads = static_cast<uint32_t>(__popc(hmask));
  const int last_head =
      hmask ? static_cast<int>(base) + first + (31 - __clz(static_cast<int>(hmask))) : -1;
  uint32_t tile_heads;
  const uint32_t heads_before = block256_excl_sum<uint32_t>(nheads, s_scan, tile_heads);
  int tile_last;
  const int last_before = block256_excl_max(last_head, s_maxs, tile_last);

  if (tid == 0) {
    uint64_t* my = status + tile;
    uint32_t eh = 0;
    int el = -1;
    if (tile == 0) {
      st_agent(my, kDFlagPrefix | (uint64_t(tile_heads) << 31) | uint64_t(tile_last + 1));
    } else {
      st_agent(my, kDFlagAgg | (uint64_t(tile_heads) << 31) | uint64_t(tile_last + 1));
      int j = tile - 1;
      uint32_t spins = 0;
      while (true) {
        const uint64_t s = ld_agent(status + j);
        const uint64_t f = s & (3ull << 62);
        if (f == 0) {
          if (++spins > kSpinLimit) { raise_err(dev_err, LM_DEVERR_SPIN); break; }
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        eh += static_cast<uint32_t>((s >> 31) & kD31);
        const int pl = static_cast<int>(s & kD31) - 1;
        if (el < 0) el = pl;
        if (f == kDFlagPrefix || j == 0) break;
        --j;
      }
      const int incl_last = tile_last >= 0 ? tile_last : el;
      st_agent(my, kDFlagPrefix | (uint64_t(eh + tile_heads) << 31) | uint64_t(incl_last + 1));
    }
    s_excl_heads = eh;
    s_excl_last = el;
  }
  __syncthreads();

  // Types can only outnumber cap = min(K, V) when ids lie outside [0, V)
  // (LM_DEVERR_ID_RANGE is raised then): clamp every write to the buffers.
  int seg = static_cast<int>(s_excl_heads + heads_before) - 1;
  int hp = last_before >= 0 ? last_before : s_excl_last;
  bool over = false;
#pragma unroll
  for (int i = 0; i < kDedupItems; ++i) {
    const int j = first + i;
    if (j < n) {
      const int64_t p = base + j;
      const KeyT k = s_keys[j + 1];
      const bool head = (hmask >> i) & 1u;
      seg += head ? 1 : 0;
      hp = head ? static_cast<int>(p) : hp;
      const bool in_cap = static_cast<uint32_t>(seg) < static_cast<uint32_t>(cap);
      over |= !in_cap;
      if (head && in_cap) {
        uniq[seg] = k;
        offsets[seg] = static_cast<int32_t>(p);
      }
      if (((tmask >> i) & 1u) && in_cap) counts[seg] = static_cast<int32_t>(p + 1 - hp);
      const int32_t src = perm[p];
      if (static_cast<uint32_t>(src) < static_cast<uint32_t>(K)) inverse[src] = seg;
      else over = true;
      if (p == K - 1) {
        *num_unique = seg + 1 < cap ? seg + 1 : cap;
        offsets[seg + 1 < cap ? seg + 1 : cap] = K;
      }
    }
  }
  if (ballot(over) && lane_id() == 0) raise_err(dev_err, LM_DEVERR_CAPACITY);
}

__global__ void k_unique_empty(int64_t* num_unique, int32_t* offsets) {
  if (threadIdx.x == 0) {
    *num_unique = 0;
    offsets[0] = 0;
  }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
size_t unique_workspace_bytes(int64_t K, int idtype, int64_t V) {
  return unique_layout(K, idtype, V).total;
}

template <typename KeyT>
static int run_unique(const KeyT* ids, int K, int64_t V, KeyT* uniq, int32_t* counts,
                      int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
                      int32_t* dev_err, char* ws, const UniqueLayout& L, hipStream_t st) {
  if (K == 0) {
    k_unique_empty<<<1, 64, 0, st>>>(num_unique, offsets);
    return launch_status(hipGetLastError());
  }
  uint32_t* hist = reinterpret_cast<uint32_t*>(ws + L.hist);
  uint32_t* tickets = reinterpret_cast<uint32_t*>(ws + L.tickets);
  uint32_t* status = reinterpret_cast<uint32_t*>(ws + L.status);
  uint64_t* dstatus = reinterpret_cast<uint64_t*>(ws + L.dstatus);
  KeyT* kb[2] = {reinterpret_cast<KeyT*>(ws + L.keys0), reinterpret_cast<KeyT*>(ws + L.keys1)};
  int32_t* vb[2] = {reinterpret_cast<int32_t*>(ws + L.vals0), reinterpret_cast<int32_t*>(ws + L.vals1)};

  // tickets .. end of dstatus is contiguous: clear it in k_hist.
  const int64_t clear_words = static_cast<int64_t>((L.keys0 - L.tickets) / 4);
  int hist_blocks = (K + kSortThreads * 16 - 1) / (kSortThreads * 16);
  if (hist_blocks > 1024) hist_blocks = 1024;
  const int64_t clear_blocks = (clear_words + kSortThreads * 8 - 1) / (kSortThreads * 8);
  if (hist_blocks < clear_blocks) hist_blocks = static_cast<int>(clear_blocks < 1024 ? clear_blocks : 1024);
  k_hist<KeyT><<<hist_blocks, kSortThreads, 0, st>>>(ids, K, static_cast<uint64_t>(V), L.passes,
                                                     L.bits, hist, tickets, clear_words, dev_err);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return launch_status(e);

  const KeyT* kin = ids;
  const int32_t* vin = nullptr;
  for (int p = 0; p < L.passes; ++p) {
    const int shift = 8 * p;
    const int nb = L.bits - shift < 8 ? L.bits - shift : 8;
    KeyT* kout = kb[p & 1];
    int32_t* vout = p == L.passes - 1 ? perm : vb[p & 1];
    k_onesweep<KeyT><<<L.tiles, kSortThreads, 0, st>>>(
        kin, vin, kout, vout, K, shift, nb < 0 ? 0 : nb, hist + p * kRadix,
        status + size_t(p) * L.tiles * kRadix, tickets + p, dev_err);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return launch_status(e);
    kin = kout;
    vin = vout;
  }
  k_dedup<KeyT><<<L.dtiles, kSortThreads, 0, st>>>(
      kin, perm, K, static_cast<int>(K < V ? K : V), uniq, counts, offsets, inverse, num_unique,
      dstatus, tickets + kMaxPasses,
      hist, L.passes * kRadix, dev_err);
  return launch_status(hipGetLastError());
}

int unique_run(const void* ids, int idtype, int64_t K, int64_t V, void* uniq, int32_t* counts,
               int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
               int32_t* dev_err, void* ws, size_t ws_bytes, hipStream_t st) {
  const UniqueLayout L = unique_layout(K, idtype, V);
  if (ws_bytes < L.total) return LM_E_WORKSPACE;
  char* w = static_cast<char*>(ws);
  if (idtype == LM_I64)
    return run_unique<int64_t>(static_cast<const int64_t*>(ids), static_cast<int>(K), V,
                               static_cast<int64_t*>(uniq), counts, offsets, inverse, perm,
                               num_unique, dev_err, w, L, st);
  return run_unique<int32_t>(static_cast<const int32_t*>(ids), static_cast<int>(K), V,
                             static_cast<int32_t*>(uniq), counts, offsets, inverse, perm,
                             num_unique, dev_err, w, L, st);
}

}  // namespace lmz
