// Unique (Sec. III-A steps 1 and 4): the distinct word indices of a batch in
// ascending order, with counts, CSR offsets, the token->type map and the
// stable sort permutation.
//
// Inputs of up to LMZ_UNIQUE_BLOCK_MAX_K ids take one workgroup that holds
// every key in LDS (k_unique_block, below). Larger inputs take a pipeline of
// kernels (all on one stream, no host sync; the only atomics are the tile
// tickets):
//   k_hist      digit histograms of every radix pass in one read of the ids,
//               one row per workgroup (4096 ids each, at most 64 rows); also
//               clears this call's tile tickets and look-back status words.
//   k_onesweep  one LSD radix pass over a digit (the ceil(log2 V) key bits
//               are split evenly over the fewest passes). A workgroup of NT
//               threads (256 for inputs of up to LMZ_UNIQUE_SMALL_TILE_MAX_K
//               keys, so that they spread over more CUs, else 1024) ranks a
//               tile of ITEMS * NT keys with
//               wave64 ballot matching, publishes its per-digit counts,
//               learns the counts of the tiles before it through a decoupled
//               look-back, reorders the tile in LDS and writes it out in
//               digit runs.
//   k_dedup     run heads on the sorted keys (4 per thread, one 16-byte load
//               each), a block scan plus a wave-wide decoupled look-back (64
//               predecessors per round) carrying (number of heads, position of
//               the last head), then writes uniq, offsets, counts, inverse and
//               num_unique. From LMZ_UNIQUE_TYPEMAP_MIN_K ids on (vocabularies
//               of up to LMZ_UNIQUE_TYPEMAP_MAX_V ids) it writes each type to
//               a table indexed by id instead of the inverse map, and
//   k_inverse_types  writes inverse[token] = table[ids[token]] in token order.
// Where the ids are narrower (V <= LMZ_UNIQUE_KEYCOUNT_MAX_V), the types
// come from a count per id instead of the sorted keys, and no dedup runs:
//   k_key_hist  the count of every id value in LDS, one row per workgroup;
//               clears the tickets and status words like k_hist.
//   k_key_scan  the rows added up per id, then a block scan and a decoupled
//               look-back over the ids in ascending order give uniq, counts,
//               offsets, num_unique and each id's type (its rank among the
//               ids present); also the digit counts of the radix passes.
//   k_onesweep  the passes as above (8 keys per thread from 512K ids on);
//               the first one, which reads the ids in token order, also
//               writes inverse[token] = rank[id], and the last writes the
//               permutation only (no sorted keys). With two passes over
//               4-byte ids the first writes one word per key, the second
//               pass's digit above the position, which the second reads.
// Tiles take their index from an atomic ticket, so a tile only waits on
// tiles that already hold a workgroup: every look-back makes progress. A
// tile's inputs are fetched for tile = blockIdx.x while the ticket is in
// flight (workgroups are dispatched in order, so the guess almost always
// holds) and fetched again when it does not.
#include <atomic>

#include "common.hpp"

namespace lmz {

#ifndef LMZ_UNIQUE_HIST_RUNS_MIN_K
#define LMZ_UNIQUE_HIST_RUNS_MIN_K (1 << 18)  // above this K, lanes' digit runs share an atomic
#endif
constexpr int kHistThreads = 1024;
#ifndef LMZ_UNIQUE_SMALL_TILE_MAX_K
#define LMZ_UNIQUE_SMALL_TILE_MAX_K (1 << 14)  // up to this K, 256-thread tiles
#endif
#ifndef LMZ_UNIQUE_DIGIT_BITS
#define LMZ_UNIQUE_DIGIT_BITS 8        // widest digit with 256-thread tiles
#endif
#ifndef LMZ_UNIQUE_DIGIT_BITS_LARGE
#define LMZ_UNIQUE_DIGIT_BITS_LARGE 10 // widest digit with 1024-thread tiles
#endif
constexpr int kBlockThreadsHost = 1024;  // threads of k_unique_block
#ifndef LMZ_UNIQUE_BLOCK_MAX_K
#define LMZ_UNIQUE_BLOCK_MAX_K 8192    // up to this K, one workgroup does it all
#endif
#ifndef LMZ_UNIQUE_GATHER
#define LMZ_UNIQUE_GATHER 1            // tile-local passes joined by gathers (see k_sort_local)
#endif
#ifndef LMZ_UNIQUE_GATHER_MAX_TILES
#define LMZ_UNIQUE_GATHER_MAX_TILES 64 // a wave holds one digit's runs of every tile
#endif
#ifndef LMZ_UNIQUE_GATHER_MIN_TILES
#define LMZ_UNIQUE_GATHER_MIN_TILES 12 // fewer tiles: the look-back passes are faster
#endif
#ifndef LMZ_UNIQUE_GATHER_DIGIT_BITS
#define LMZ_UNIQUE_GATHER_DIGIT_BITS 9 // widest digit of the tile-local passes
#endif
#ifndef LMZ_UNIQUE_KEYCOUNT_MAX_V
#define LMZ_UNIQUE_KEYCOUNT_MAX_V (1 << 15)  // up to this V (and past one workgroup), counts per id
#endif
// From this many ids on (and vocabularies of up to LMZ_UNIQUE_TYPEMAP_MAX_V
// ids), the dedup writes each type once to a table indexed by id, and a
// pass in token order writes the inverse map from it, instead of scattering
// one 4-byte store per token to the tokens' positions. Above the largest K
// of lm_unique_noalloc, whose fixed scratch does not hold the table.
#ifndef LMZ_UNIQUE_TYPEMAP_MIN_K
#define LMZ_UNIQUE_TYPEMAP_MIN_K (1 << 19)
#endif
#ifndef LMZ_UNIQUE_TYPEMAP_MAX_V
#define LMZ_UNIQUE_TYPEMAP_MAX_V (int64_t(1) << 24)
#endif
static_assert(LMZ_UNIQUE_TYPEMAP_MIN_K > LM_UNIQUE_NOALLOC_MAX_K,
              "the type table would not fit lm_unique_noalloc's scratch");
#ifndef LMZ_UNIQUE_LOOKBACK_W
#define LMZ_UNIQUE_LOOKBACK_W 4        // predecessor tiles a look-back round reads
#endif
constexpr int kSmallDigitBits = LMZ_UNIQUE_DIGIT_BITS;
constexpr int kLargeDigitBits = LMZ_UNIQUE_DIGIT_BITS_LARGE;
constexpr int kMaxPasses = 8;              // ceil(64 / 8)
constexpr int kGatherSmallTileKeys = 1024;  // keys per 256-thread tile-local workgroup
// Keys per thread of a sort or dedup tile, by input size: bigger tiles mean
// fewer tiles for the look-back to pass, smaller ones spread a small input
// over more CUs. Measured best: with 256-thread tiles, 2 keys up to 16K ids
// (4 above, where 256-thread tiles are no longer the default); with
// 1024-thread tiles, 2 up to 512K, 4 up to 1.5M, 8 above.
#ifndef LMZ_UNIQUE_SMALL_ITEMS2_MAX_K
#define LMZ_UNIQUE_SMALL_ITEMS2_MAX_K (1 << 14)
#endif
#ifndef LMZ_UNIQUE_LARGE_ITEMS2_MAX_K
#define LMZ_UNIQUE_LARGE_ITEMS2_MAX_K (1 << 19)
#endif
#ifndef LMZ_UNIQUE_LARGE_ITEMS4_MAX_K
#define LMZ_UNIQUE_LARGE_ITEMS4_MAX_K (3 << 19)
#endif
static inline int items_for(int64_t K, int nt) {
  if (nt == 256) return K <= LMZ_UNIQUE_SMALL_ITEMS2_MAX_K ? 2 : 4;
  return K <= LMZ_UNIQUE_LARGE_ITEMS2_MAX_K ? 2 : (K <= LMZ_UNIQUE_LARGE_ITEMS4_MAX_K ? 4 : 8);
}
constexpr int kHistItems = 16;             // keys per thread per histogram round
// ids per k_key_scan workgroup: 256 measured 1.2 us faster per call than
// 1024 at 1,048,576 ids over 20K words (80 workgroups against 20)
constexpr int kKeyScanThreads = 256;
// Histogram workgroups: about K / 2048 of them, 8 to 32, up to 2^18 ids
// (measured best: 8 at 8K ids, 32 at 64K and 262K), 64 above (larger
// blocks serialise on LDS atomics at the Zipf heads).
#ifndef LMZ_UNIQUE_HIST_RULE
#define LMZ_UNIQUE_HIST_RULE 1
#endif
#ifndef LMZ_UNIQUE_HIST_KEYS
#define LMZ_UNIQUE_HIST_KEYS 4096      // ids per histogram workgroup without the rule
#endif
constexpr int kHistKeysPerBlock = LMZ_UNIQUE_HIST_KEYS;
static inline int hist_blocks_for(int64_t K) {
  if (LMZ_UNIQUE_HIST_RULE) {
    if (K > (int64_t(1) << 18)) return 64;
    const int64_t b = K / 2048;
    return static_cast<int>(b < 8 ? 8 : (b > 32 ? 32 : b));
  }
  const int64_t hb = (K + kHistKeysPerBlock - 1) / kHistKeysPerBlock;
  return static_cast<int>(hb < 1 ? 1 : (hb > 64 ? 64 : hb));
}

// Status words of the sort look-back: 2-bit flag | 30-bit count.
constexpr uint32_t kFlagAgg = 1u << 30, kFlagPrefix = 2u << 30, kValMask = (1u << 30) - 1;
// Status words of the dedup look-back: flag (2) | heads (31) | last head + 1 (31).
constexpr uint64_t kDFlagAgg = 1ull << 62, kDFlagPrefix = 2ull << 62, kDFlags = 3ull << 62;
constexpr uint64_t kD31 = (1ull << 31) - 1;

struct UniqueLayout {
  size_t bhist, tickets, status, dstatus, keys0, keys1, vals0, vals1, total;
  int passes, bits, tiles, hist_blocks, nt, items;
  int block_items;  // > 0: one workgroup (k_unique_block) with this many keys per thread
  int block_rb;     // its digit width (8, 9 or 10): the widest digit of its passes
  int gather;       // 1: tile-local passes (k_sort_local) and a gathering dedup; the
                    // histogram region then holds the runs of each pass and tile
  int keycount;     // 1: a count per id (k_key_hist, k_key_scan) instead of k_hist
                    // and k_dedup; bhist then holds a row per k_key_scan tile
  int typemap;      // 1: the dedup writes each id's type to a table (rank) and
                    // k_inverse_types writes the inverse map in token order
  int key_blocks;   // k_key_hist workgroups (rows of khist)
  int scan_tiles;   // k_key_scan workgroups, kKeyScanThreads ids each
  size_t khist, rank;
  int rstride;  // digit slots per pass in the histogram rows and status arrays
  int shift[kMaxPasses], nbits[kMaxPasses];
};

static inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

static inline int key_bits_for(int64_t V) {
  if (V <= 1) return 0;
  const uint64_t m = static_cast<uint64_t>(V - 1);
  return 64 - __builtin_clzll(m);
}

static UniqueLayout unique_layout(int64_t K, int idtype, int64_t V) {
  UniqueLayout L{};
  const size_t ks = idtype == LM_I64 ? 8 : 4;
  L.bits = key_bits_for(V);
  // Workgroups of 256 threads take 8-bit digits; 1024-thread workgroups take
  // digits of up to 10 bits where that saves a pass (20-bit keys: two passes
  // instead of three), with fewer tiles for the look-back to pass. Measured
  // per call: 256-thread tiles are faster up to 16K ids (4K ids at V = 800K:
  // 26 against 29 us), 1024-thread tiles above (64K ids: 37 against 43 us;
  // 131K ids: 43 against 51 us).
  L.nt = K <= LMZ_UNIQUE_SMALL_TILE_MAX_K ? 256 : 1024;
  // One workgroup holds up to 1024 * 8 keys (8 per thread keep the ranking
  // and dedup state in registers).
  L.block_items = 0;
  if (K <= LMZ_UNIQUE_BLOCK_MAX_K && K <= 8 * kBlockThreadsHost) {
    L.block_items = 1;
    while (int64_t(L.block_items) * 1024 < K) L.block_items *= 2;
  }
  L.items = items_for(K, L.nt);
  const int64_t tile_keys = int64_t(L.nt) * L.items;
  L.tiles = static_cast<int>((K + tile_keys - 1) / tile_keys);
  // Tile-local passes joined by gathers (k_sort_local) from 12 to 64 tiles,
  // with digits of at most 9 bits: a gather adds up every tile's count of
  // each digit, which 10-bit digits made the larger cost. Measured per call
  // (us, look-back passes / gathers): 65,536 ids at V = 800K 37.1 / 32.0
  // (10-bit digits: 38.1), 131,072 ids 43.0 / 33.7, 24,576 ids 32.6 / 31.5;
  // at 9 tiles (16,385 ids, V = 262,144) 31.9 / 36.2.
  L.gather = LMZ_UNIQUE_GATHER && !L.block_items && L.nt == 1024 && L.items == 2 &&
             L.tiles <= LMZ_UNIQUE_GATHER_MAX_TILES && L.tiles >= LMZ_UNIQUE_GATHER_MIN_TILES;
  // Where tiles of 1024 keys still number at most 64 (up to 65,536 ids),
  // 256-thread workgroups take them, with digits of at most 8 bits so that
  // every gathering workgroup has a thread per digit of the pass before.
  // Four-wave workgroups fit beside the one-wave Seg-Sum and update
  // workgroups of an earlier step when Unique runs on a stream of its own:
  // measured at 65,536 ids over 800K words, 34 -> 36 us per call alone, and
  // the overlapped word step 143.6 -> 129.6 us.
  if (L.gather) {
    const int64_t small_tiles = (K + kGatherSmallTileKeys - 1) / kGatherSmallTileKeys;
    if (small_tiles <= LMZ_UNIQUE_GATHER_MAX_TILES) {
      L.nt = 256;
      L.items = kGatherSmallTileKeys / 256;
      L.tiles = static_cast<int>(small_tiles);
    }
  }
  const int narrow = kSmallDigitBits < kLargeDigitBits ? kSmallDigitBits : kLargeDigitBits;
  // The one workgroup takes digits of up to 10 bits (a thread per digit):
  // the fewest passes, with the narrowest digits that reach them (17-bit
  // keys: 9 + 8 bits). Measured at 8,192 ids: 21.2 against 24.1 us for three
  // 8-bit passes at 17-bit keys, 24.2 against 25.8 us at 20-bit keys; where
  // wider digits save no pass (15 and 31 bits) 8-bit ones stay faster.
  const int widest = L.block_items ? kLargeDigitBits
                     : L.gather  ? (L.nt == 256 ? kSmallDigitBits : LMZ_UNIQUE_GATHER_DIGIT_BITS)
                                 : (L.nt == 256 ? kSmallDigitBits : kLargeDigitBits);
  const int p_narrow = (L.bits + narrow - 1) / narrow, p_wide = (L.bits + widest - 1) / widest;
  L.passes = L.bits == 0 ? 1 : (p_wide < p_narrow ? p_wide : p_narrow);
  // Split the key bits evenly: the low passes take the extra bit.
  int sh = 0;
  for (int p = 0; p < L.passes; ++p) {
    const int nb = L.bits / L.passes + (p < L.bits % L.passes ? 1 : 0);
    L.shift[p] = sh;
    L.nbits[p] = nb;
    sh += nb;
  }
  L.block_rb = kSmallDigitBits;
  for (int p = 0; p < L.passes; ++p)
    if (L.block_items && L.nbits[p] > L.block_rb) L.block_rb = L.nbits[p];
  L.hist_blocks = hist_blocks_for(K);
  if (L.gather) L.hist_blocks = L.tiles;  // one row of runs per pass and tile
  L.keycount = !L.block_items && !L.gather && V <= LMZ_UNIQUE_KEYCOUNT_MAX_V;
  // With the counts per id, tiles of 8 keys per thread from 512K ids on.
  // Alone the call times the same as with 4 (1,048,576 ids over 20K words:
  // 54.7 against 53.9 us), but beside the Seg-Sum walk (Unique on CUs of
  // its own) the sort passes' scattered digit runs slow the walk, and tiles
  // twice as large write half as many runs and pass half as many tiles in
  // the look-back: 1,434 -> 1,426 us per overlapped step at that workload.
  if (L.keycount && L.nt == 1024 && L.items == 4) {
    L.items = 8;
    L.tiles = static_cast<int>((K + int64_t(L.nt) * L.items - 1) / (int64_t(L.nt) * L.items));
  }
  L.typemap = !L.block_items && !L.gather && !L.keycount && K >= LMZ_UNIQUE_TYPEMAP_MIN_K &&
              V <= LMZ_UNIQUE_TYPEMAP_MAX_V;
  if (L.keycount) {
    L.key_blocks = L.hist_blocks;
    L.scan_tiles = static_cast<int>((V + kKeyScanThreads - 1) / kKeyScanThreads);
    L.hist_blocks = L.scan_tiles;  // the passes add up one row per scan tile
  }
  size_t off = 0;
  L.rstride = 1 << kSmallDigitBits;
  for (int p = 0; p < L.passes; ++p)
    if (L.nbits[p] > kSmallDigitBits) L.rstride = 1 << kLargeDigitBits;
  L.bhist = off;   off += align256(size_t(L.hist_blocks) * L.passes * L.rstride * 4);
  L.tickets = off; off += 256;
  L.status = off;  // the look-backs' words (none when the passes gather)
  if (!L.gather) off += align256(size_t(L.passes) * L.tiles * L.rstride * 4);
  L.dstatus = off;  // the dedup's (or the key scan's) look-back words
  off += align256(size_t(L.tiles > L.scan_tiles ? L.tiles : L.scan_tiles) * 8);
  L.keys0 = off;   off += align256(size_t(K) * ks);
  L.keys1 = off;   off += align256(size_t(K) * ks);
  L.vals0 = off;   off += align256(size_t(K) * 4);
  L.vals1 = off;   off += align256(size_t(K) * 4);
  if (L.keycount) {
    L.khist = off; off += align256(size_t(L.key_blocks) * V * 4);
  }
  if (L.keycount || L.typemap) {
    L.rank = off;  off += align256(size_t(V) * 4);
  }
  L.total = off;
  return L;
}

template <int N>
using I = std::integral_constant<int, N>;

// The look-backs' bounded waits: polls before giving up (LM_DEVERR_SPIN),
// and the test hook for that path (every predecessor read as not ready).
struct WaitCfg {
  uint32_t spin_limit;
  int force_fail;
};
// Two-pass sorts with the counts per id and 4-byte ids: the first pass
// writes, for each key, one word holding the second pass's digit above the
// token's position (mode 1), and the second pass reads that word as its key
// and the position from its low pos_bits bits (mode 2). That halves the
// first pass's scattered writes and the second pass's reads.
struct PackCfg {
  int mode;      // 0: keys and positions apart; 1: write packed words; 2: read them
  int shift;     // mode 1: the second pass's digit within the key
  int nbits;     //         and its width
  int pos_bits;  // bits of the position in a packed word
};
static std::atomic<bool> g_force_wait_failure{false};
static std::atomic<uint32_t> g_forced_spin_limit{kSpinLimit};

void unique_force_wait_failure(bool enable, uint32_t limit) {
  g_forced_spin_limit.store(limit < 1 ? 1u : limit, std::memory_order_relaxed);
  g_force_wait_failure.store(enable, std::memory_order_relaxed);
}

static WaitCfg wait_cfg() {
  const bool fail = g_force_wait_failure.load(std::memory_order_relaxed);
  return WaitCfg{fail ? g_forced_spin_limit.load(std::memory_order_relaxed) : kSpinLimit,
                 fail ? 1 : 0};
}

struct PassBits {
  int shift[kMaxPasses], nbits[kMaxPasses];
};

template <typename KeyT>
__device__ __forceinline__ uint32_t digit_of(KeyT k, int shift, uint32_t mask) {
  return static_cast<uint32_t>(key_bits(k) >> shift) & mask;
}

// gfx950's three-input bitwise op: bit (a << 2 | b << 1 | c) of the
// immediate is the result for input bits a, b, c. This one is a & ~(b ^ c).
constexpr int kBitop3AndXnor = (1 << 4) | (1 << 7);

// The lanes of this wave whose digit equals this lane's, among the lanes of
// `valid`: one ballot per digit bit, and a lane keeps the lanes whose bit
// agrees with its own, peers &= ~(bits ^ mine) with its bit spread over the
// word (0 or ~0). Digits have no bits at or above RB on valid lanes, so bits
// past a pass's width (zero in every lane) leave the mask unchanged and the
// loop needs no bound of its own. Four instructions per bit: the bit field
// extract, the compare that is the ballot, and one three-input op per half
// (the loop with a runtime bound and a select per half took about twice as
// many, with a branch per bit).
template <int RB>
__device__ __forceinline__ uint64_t match_digit(uint32_t dig, uint64_t valid) {
  uint32_t lo = static_cast<uint32_t>(valid), hi = static_cast<uint32_t>(valid >> 32);
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    uint32_t mine = static_cast<uint32_t>(__builtin_amdgcn_sbfe(static_cast<int>(dig), b, 1));
    // Opaque to the optimiser, so that the ballot compares this value
    // instead of deriving the bit again with a shift and a compare.
    __asm__("" : "+v"(mine));
    const uint64_t bits = ballot(mine != 0u);
    lo = __builtin_amdgcn_bitop3_b32(lo, static_cast<uint32_t>(bits), mine, kBitop3AndXnor);
    hi = __builtin_amdgcn_bitop3_b32(hi, static_cast<uint32_t>(bits >> 32), mine, kBitop3AndXnor);
  }
  return (uint64_t(hi) << 32) | lo;
}

// Wave and block scans for Unique's kernels. Within a wave they use DPP
// (lanes read other lanes' registers inside the ALU op: row shifts by 1, 2
// and 3, then by 4 and 8 on the upper banks of each 16-lane row, then the
// broadcasts of lanes 15 and 31 to the rows after them), not LDS permutes:
// a 64-lane scan is seven dependent ALU ops instead of six LDS round trips.
// `id` is the operation's identity, which a lane takes where its source
// lies outside its row or its row or bank is masked off.
struct OpAdd {
  __device__ int operator()(int a, int b) const { return a + b; }
};
struct OpMax {
  __device__ int operator()(int a, int b) const { return a > b ? a : b; }
};

template <typename Op>
__device__ __forceinline__ int dpp_incl_scan(int v, Op op, int id) {
  int a = op(v, __builtin_amdgcn_update_dpp(id, v, 0x111, 0xf, 0xf, false));  // row_shr:1
  a = op(a, __builtin_amdgcn_update_dpp(id, v, 0x112, 0xf, 0xf, false));      // row_shr:2
  a = op(a, __builtin_amdgcn_update_dpp(id, v, 0x113, 0xf, 0xf, false));      // row_shr:3
  a = op(a, __builtin_amdgcn_update_dpp(id, a, 0x114, 0xf, 0xe, false));      // row_shr:4
  a = op(a, __builtin_amdgcn_update_dpp(id, a, 0x118, 0xf, 0xc, false));      // row_shr:8
  a = op(a, __builtin_amdgcn_update_dpp(id, a, 0x142, 0xa, 0xf, false));      // row_bcast:15
  a = op(a, __builtin_amdgcn_update_dpp(id, a, 0x143, 0xc, 0xf, false));      // row_bcast:31
  return a;
}

// The value of the lane below this one (`id` on lane 0): DPP wave_shr:1.
__device__ __forceinline__ int dpp_lane_below(int v, int id) {
  return __builtin_amdgcn_update_dpp(id, v, 0x138, 0xf, 0xf, false);
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
  return static_cast<uint32_t>(
      read_lane(dpp_incl_scan(static_cast<int>(v), OpAdd(), 0), kWave - 1));
}

// Exclusive sums over a block of NW waves of two values at once (one pair
// of barriers for both); lds holds 2 * NW words. t0, t1: the block totals.
template <int NW>
__device__ __forceinline__ void blk_excl_sum2(uint32_t v0, uint32_t v1, uint32_t* lds,
                                              uint32_t& e0, uint32_t& t0, uint32_t& e1,
                                              uint32_t& t1) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t i0 = static_cast<uint32_t>(dpp_incl_scan(static_cast<int>(v0), OpAdd(), 0));
  const uint32_t i1 = static_cast<uint32_t>(dpp_incl_scan(static_cast<int>(v1), OpAdd(), 0));
  if (lane == kWave - 1) {
    lds[wave] = i0;
    lds[NW + wave] = i1;
  }
  __syncthreads();
  uint32_t b0 = 0, b1 = 0, a0 = 0, a1 = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint32_t x0 = lds[w], x1 = lds[NW + w];
    b0 += w < wave ? x0 : 0u;
    b1 += w < wave ? x1 : 0u;
    a0 += x0;
    a1 += x1;
  }
  __syncthreads();
  e0 = b0 + i0 - v0;
  e1 = b1 + i1 - v1;
  t0 = a0;
  t1 = a1;
}

// Exclusive sum over a block of NW waves; lds holds NW words.
template <int NW>
__device__ __forceinline__ uint32_t blk_excl_sum(uint32_t v, uint32_t* lds, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t incl = static_cast<uint32_t>(dpp_incl_scan(static_cast<int>(v), OpAdd(), 0));
  if (lane == kWave - 1) lds[wave] = incl;
  __syncthreads();
  uint32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint32_t x = lds[w];
    before += w < wave ? x : 0u;
    all += x;
  }
  __syncthreads();
  total = all;
  return before + incl - v;
}

// An exclusive sum (s) and an exclusive maximum (m, values >= -1, -1 before
// the first thread) over a block of NW waves with one pair of barriers.
template <int NW>
__device__ __forceinline__ void blk_excl_sum_max(uint32_t s, int m, uint32_t* lds_s, int* lds_m,
                                                 uint32_t& es, uint32_t& ts, int& em, int& tm) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t is = static_cast<uint32_t>(dpp_incl_scan(static_cast<int>(s), OpAdd(), 0));
  const int im = dpp_incl_scan(m, OpMax(), -1);
  const int prev = dpp_lane_below(im, -1);
  if (lane == kWave - 1) {
    lds_s[wave] = is;
    lds_m[wave] = im;
  }
  __syncthreads();
  uint32_t bs = 0, as = 0;
  int bm = -1, am = -1;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const uint32_t x = lds_s[w];
    const int y = lds_m[w];
    bs += w < wave ? x : 0u;
    as += x;
    if (w < wave && y > bm) bm = y;
    if (y > am) am = y;
  }
  __syncthreads();
  es = bs + is - s;
  ts = as;
  em = prev > bm ? prev : bm;
  tm = am;
}

// Exclusive maximum (values >= -1; -1 before the first thread) over a block
// of NW waves; lds holds NW words.
template <int NW>
__device__ __forceinline__ int blk_excl_max(int v, int* lds, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int incl = dpp_incl_scan(v, OpMax(), -1);
  const int prev = dpp_lane_below(incl, -1);
  if (lane == kWave - 1) lds[wave] = incl;
  __syncthreads();
  int before = -1, all = -1;
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const int x = lds[w];
    if (w < wave && x > before) before = x;
    if (x > all) all = x;
  }
  __syncthreads();
  total = all;
  return prev > before ? prev : before;
}

// ---------------------------------------------------------------------------
// k_hist: bhist[b][p][d] = number of keys read by workgroup b whose digit of
// pass p is d (rows of rstride slots per pass). Also clears the tickets and the
// look-back status words of this call.
// ---------------------------------------------------------------------------
template <typename KeyT, bool RUNS>
__global__ __launch_bounds__(kHistThreads) void k_hist(
    const KeyT* __restrict__ keys, int K, uint64_t V, int passes, int rstride, PassBits pb,
    uint32_t* __restrict__ bhist, uint32_t* __restrict__ clear, int64_t clear_words,
    int32_t* __restrict__ dev_err) {
  extern __shared__ uint32_t sh[];  // passes * rstride
  for (int i = threadIdx.x; i < passes * rstride; i += kHistThreads) sh[i] = 0;
  for (int64_t i = blockIdx.x * int64_t(kHistThreads) + threadIdx.x; i < clear_words;
       i += int64_t(gridDim.x) * kHistThreads)
    clear[i] = 0;
  __syncthreads();
  bool bad = false;
  const int64_t stride = int64_t(gridDim.x) * kHistThreads;
  for (int64_t i0 = blockIdx.x * int64_t(kHistThreads) + threadIdx.x; i0 < K;
       i0 += stride * kHistItems) {
    KeyT kv[kHistItems];  // all loads of a round in flight together
#pragma unroll
    for (int j = 0; j < kHistItems; ++j) {
      const int64_t i = i0 + j * stride;
      kv[j] = i < K ? keys[i] : KeyT(0);
    }
#pragma unroll
    for (int j = 0; j < kHistItems; ++j) {
      const bool in = i0 + j * stride < K;
      const uint64_t kb = key_bits(kv[j]);
      bad |= in && kb >= V;
      // the lanes past K are the last ones of the wave
      const int nact = RUNS ? __popcll(ballot(in)) : 0;
      for (int p = 0; p < passes; ++p) {
        const uint32_t d = static_cast<uint32_t>(kb >> pb.shift[p]) & ((1u << pb.nbits[p]) - 1);
        if constexpr (RUNS) {
          // Lanes hold consecutive ids: a run of lanes with the same digit
          // adds its length with one atomic. Zipf heads put long runs of the
          // heaviest digit on adjacent lanes, whose LDS atomics on one address
          // would otherwise serialise: measured at 1,048,576 ids over 20K
          // words 78.3 -> 71.4 us per Unique call, 2M ids 126.6 -> 124.4 us;
          // at 262,144 ids (32 workgroups, less skew) 60.0 -> 62.0 us, so
          // only inputs above LMZ_UNIQUE_HIST_RUNS_MIN_K take it.
          const uint32_t up = static_cast<uint32_t>(dpp_lane_below(static_cast<int>(d), static_cast<int>(d)));
          const int ln = lane_id();
          const bool head = in && (ln == 0 || up != d);
          const uint64_t heads = ballot(head);
          if (head) {
            const uint64_t above = ln < 63 ? heads & ~((2ull << ln) - 1ull) : 0ull;
            const int next = above ? __builtin_ctzll(above) : nact;
            atomicAdd(&sh[p * rstride + d], static_cast<uint32_t>(next - ln));
          }
        } else if (in) {
          atomicAdd(&sh[p * rstride + d], 1u);
        }
      }
    }
  }
  if (ballot(bad) && lane_id() == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
  __syncthreads();
  uint32_t* row = bhist + size_t(blockIdx.x) * passes * rstride;
  for (int i = threadIdx.x; i < passes * rstride; i += kHistThreads) row[i] = sh[i];
}

// ---------------------------------------------------------------------------
// k_key_hist: khist[b][v] = number of keys read by workgroup b equal to v,
// for every v < V (V <= LMZ_UNIQUE_KEYCOUNT_MAX_V: a counter per id in LDS).
// Like k_hist, lanes hold consecutive ids and a run of lanes with the same
// id adds its length with one atomic; it also clears the call's tickets and
// look-back status words. Ids outside [0, V) raise LM_DEVERR_ID_RANGE and
// are not counted.
// ---------------------------------------------------------------------------
template <typename KeyT>
__global__ __launch_bounds__(kHistThreads) void k_key_hist(
    const KeyT* __restrict__ keys, int K, int V, uint32_t* __restrict__ khist,
    uint32_t* __restrict__ clear, int64_t clear_words, int32_t* __restrict__ dev_err) {
  extern __shared__ uint32_t sh[];  // V counters (at most 128 KiB)
  for (int i = threadIdx.x; i < V; i += kHistThreads) sh[i] = 0;
  for (int64_t i = blockIdx.x * int64_t(kHistThreads) + threadIdx.x; i < clear_words;
       i += int64_t(gridDim.x) * kHistThreads)
    clear[i] = 0;
  __syncthreads();
  bool bad = false;
  const int ln = lane_id();
  const int64_t stride = int64_t(gridDim.x) * kHistThreads;
  for (int64_t i0 = blockIdx.x * int64_t(kHistThreads) + threadIdx.x; i0 < K;
       i0 += stride * kHistItems) {
    KeyT kv[kHistItems];  // all loads of a round in flight together
#pragma unroll
    for (int j = 0; j < kHistItems; ++j) {
      const int64_t i = i0 + j * stride;
      kv[j] = i < K ? keys[i] : KeyT(0);
    }
#pragma unroll
    for (int j = 0; j < kHistItems; ++j) {
      const bool in = i0 + j * stride < K;
      const uint64_t kb = key_bits(kv[j]);
      bad |= in && kb >= static_cast<uint64_t>(V);
      const bool ok = in && kb < static_cast<uint64_t>(V);
      const int v = ok ? static_cast<int>(kb) : -1;
      const int up = dpp_lane_below(v, -2);
      const bool head = ok && up != v;
      // a run ends before the next head or the next lane that counts nothing
      const uint64_t stops = ballot(head) | ~ballot(ok);
      if (head) {
        const uint64_t above = ln < 63 ? stops & ~((2ull << ln) - 1ull) : 0ull;
        const int next = above ? __builtin_ctzll(above) : kWave;
        atomicAdd(&sh[v], static_cast<uint32_t>(next - ln));
      }
    }
  }
  if (ballot(bad) && ln == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
  __syncthreads();
  uint32_t* row = khist + size_t(blockIdx.x) * V;
  for (int i = threadIdx.x; i < V; i += kHistThreads) row[i] = sh[i];
}

// ---------------------------------------------------------------------------
// k_key_scan: tile `tile` (by ticket) owns the ids v = tile * NT + tid. An
// id's count is the sum of its khist rows; the ids with a count are the
// types, in ascending order. A block scan of (count, has a count) and a
// decoupled look-back over the tiles (64 predecessors per round, the pair
// (types, tokens) before each tile in one 64-bit status word) give every
// type its index and CSR offset: uniq, counts, offsets, rank[v] = the type
// of id v, num_unique and offsets[U] = K. Each workgroup also writes its
// ids' counts per digit of every radix pass as a row of bhist, which the
// passes add up like k_hist's rows.
// ---------------------------------------------------------------------------
template <typename KeyT, int NT>
__global__ __launch_bounds__(NT) void k_key_scan(
    const uint32_t* __restrict__ khist, int rows, int V, int K, int passes, int rstride,
    PassBits pb, uint32_t* __restrict__ bhist, KeyT* __restrict__ uniq,
    int32_t* __restrict__ counts, int32_t* __restrict__ offsets, int32_t* __restrict__ rank,
    int64_t* __restrict__ num_unique, uint64_t* __restrict__ status,
    uint32_t* __restrict__ ticket, int32_t* __restrict__ dev_err, WaitCfg wc) {
  constexpr int kWaves = NT / kWave;
  constexpr int kDigSlots = 2 * (1 << kLargeDigitBits);  // passes * rstride at most
  __shared__ uint32_t s_dig[kDigSlots];
  __shared__ uint32_t s_scan[2 * kWaves];
  __shared__ uint32_t s_tile, s_excl_types, s_excl_tokens;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);
  if (tid == 0) s_tile = add_agent(ticket, 1u);
  for (int i = tid; i < passes * rstride; i += NT) s_dig[i] = 0;
  __syncthreads();
  const int tile = first_lane(static_cast<int>(s_tile));
  const int v = tile * NT + tid;

  // This id's count: its rows, 16 loads in flight per round.
  uint32_t c = 0;
  if (v < V) {
    constexpr int kRows = 16;
    for (int b = 0; b < rows; b += kRows) {
      uint32_t h[kRows];
#pragma unroll
      for (int r = 0; r < kRows; ++r) h[r] = khist[size_t(b + r < rows ? b + r : b) * V + v];
#pragma unroll
      for (int r = 0; r < kRows; ++r) c += b + r < rows ? h[r] : 0u;
    }
  }
  if (c > 0)
    for (int p = 0; p < passes; ++p)
      atomicAdd(&s_dig[p * rstride + ((static_cast<uint32_t>(v) >> pb.shift[p]) &
                                      ((1u << pb.nbits[p]) - 1))],
                c);
  const uint32_t nz = c > 0 ? 1u : 0u;
  uint32_t c_before, tile_tokens, t_before, tile_types;
  blk_excl_sum2<kWaves>(c, nz, s_scan, c_before, tile_tokens, t_before, tile_types);
  uint32_t* row = bhist + size_t(blockIdx.x) * passes * rstride;
  for (int i = tid; i < passes * rstride; i += NT) row[i] = s_dig[i];

  // Wave 0: publish the tile aggregate, then look back 64 tiles per round.
  if (wave == 0) {
    uint64_t* my = status + tile;
    const uint64_t agg = (uint64_t(tile_types) << 31) | uint64_t(tile_tokens);
    if (lane == 0) st_agent(my, (tile == 0 ? kDFlagPrefix : kDFlagAgg) | agg);
    uint32_t et = 0, ek = 0;
    if (tile > 0) {
      int j = tile - 1;
      uint32_t spins = 0;
      while (true) {
        const int pos = j - lane;
        const uint64_t st = pos >= 0 ? ld_agent(status + pos) : kDFlagPrefix;
        const uint64_t f = wc.force_fail ? 0 : st & kDFlags;
        const uint64_t notready = ballot(f == 0);
        const uint64_t prefix = ballot(f == kDFlagPrefix);
        const int first_nr = notready ? __builtin_ctzll(notready) : kWave;
        const int first_px = prefix ? __builtin_ctzll(prefix) : kWave;
        const bool done = first_px < first_nr;
        const int take = done ? first_px + 1 : first_nr;  // lanes [0, take) are consumed
        const bool mine = lane < take;
        et += wave_sum(mine ? static_cast<uint32_t>((st >> 31) & kD31) : 0u);
        ek += wave_sum(mine ? static_cast<uint32_t>(st & kD31) : 0u);
        if (done) break;
        j -= take;
        if (take == 0) {
          if (++spins > wc.spin_limit) {
            if (lane == 0) raise_err(dev_err, LM_DEVERR_SPIN);
            break;
          }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      if (lane == 0)
        st_agent(my, kDFlagPrefix | ((uint64_t(et + tile_types) & kD31) << 31) |
                         ((uint64_t(ek) + tile_tokens) & kD31));
    }
    if (lane == 0) {
      s_excl_types = et;
      s_excl_tokens = ek;
    }
  }
  __syncthreads();
  const uint32_t types_before = s_excl_types, tokens_before = s_excl_tokens;
  if (nz) {
    const int seg = static_cast<int>(types_before + t_before);
    uniq[seg] = static_cast<KeyT>(v);
    counts[seg] = static_cast<int32_t>(c);
    offsets[seg] = static_cast<int32_t>(tokens_before + c_before);
    rank[v] = seg;
  }
  if (tile == static_cast<int>(gridDim.x) - 1 && tid == 0) {
    const uint32_t U = types_before + tile_types;
    *num_unique = U;
    offsets[U] = K;
  }
}

// ---------------------------------------------------------------------------
// k_onesweep: one stable LSD pass over the digit (key >> shift) & (2^nbits-1),
// nbits <= RB. Thread t answers for digits t*DPT .. t*DPT+DPT-1 (DPT = 2 for
// 11-bit digits; for 8-bit digits threads 0..255 answer for one each).
// ---------------------------------------------------------------------------
template <typename KeyT, int RB, int NT, int ITEMS>
__global__ __launch_bounds__(NT) void k_onesweep(
    const KeyT* __restrict__ keys_in, const int32_t* __restrict__ vals_in,
    KeyT* __restrict__ keys_out, int32_t* __restrict__ vals_out, int K, int shift, int nbits,
    const uint32_t* __restrict__ bhist, int hist_blocks, int hist_stride,
    uint32_t* __restrict__ status, uint32_t* __restrict__ ticket, int32_t* __restrict__ dev_err,
    WaitCfg wc, const int32_t* __restrict__ type_of_id, uint32_t n_ids,
    int32_t* __restrict__ inverse, PackCfg pk) {
  constexpr int kWaves = NT / kWave;
  constexpr int kItems = ITEMS;
  constexpr int kTile = NT * kItems;
  constexpr int kRadix = 1 << RB;
  constexpr int DPT = kRadix >= NT ? kRadix / NT : 1;
  constexpr int kDigitThreads = kRadix / DPT;        // threads that own digits
  constexpr int W = LMZ_UNIQUE_LOOKBACK_W;           // predecessors per look-back round
  __shared__ KeyT s_keys[kTile];
  __shared__ int32_t s_vals[kTile];
  __shared__ uint16_t s_cnt[kWaves][kRadix];         // per-wave digit counts, then offsets
  __shared__ int32_t s_shift[kRadix];                // global position - local position
  __shared__ int32_t s_local[kRadix];                // tile-local start of each digit
  __shared__ uint32_t s_scan[2 * kWaves];  // two block sums at once
  __shared__ uint32_t s_tile;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);
  const bool owner = tid < kDigitThreads;
  if (tid == 0) s_tile = add_agent(ticket, 1u);
  const uint32_t mask = nbits > 0 ? (1u << nbits) - 1 : 0u;

  // Item i of a lane is base + wave*256 + i*64 + lane: (wave, i, lane) order
  // is position order. Fetched for tile blockIdx.x while the ticket flies.
  KeyT key[kItems];
  int32_t val[kItems];
  auto fetch = [&](int64_t base) {
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int64_t pos = base + int64_t(wave) * (kItems * kWave) + i * kWave + lane;
      const bool ok = pos < K;
      key[i] = ok ? keys_in[pos] : KeyT(0);
      val[i] = ok ? (vals_in ? vals_in[pos] : static_cast<int32_t>(pos)) : 0;
    }
    if (pk.mode == 2) {  // the position is the packed word's low bits
      const uint32_t pm = (1u << pk.pos_bits) - 1u;
#pragma unroll
      for (int i = 0; i < kItems; ++i) val[i] = static_cast<int32_t>(static_cast<uint32_t>(key_bits(key[i])) & pm);
    }
  };
  fetch(int64_t(blockIdx.x) * kTile);
  // Totals of this thread's digits over the whole input (the histogram
  // rows of every k_hist workgroup). Where the threads outnumber the digits
  // (8-bit digits on 1024 threads), kRowGroups threads share a digit, each
  // summing every kRowGroups-th row, so the rows take one round of loads
  // instead of two: measured 72.0 -> 69.9 us per call at 1,048,576 ids over
  // 20K words (64 rows, 8-bit digits).
  constexpr int kRowGroups = kDigitThreads < NT ? NT / kDigitThreads : 1;
  __shared__ uint32_t s_rows[kRowGroups > 1 ? kRowGroups : 1][kRowGroups > 1 ? kDigitThreads : 1];
  uint32_t dig_total[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) dig_total[i] = 0;
  if constexpr (kRowGroups > 1) {
    const int d = tid % kDigitThreads, g = tid / kDigitThreads;
    constexpr int kHistRows = 16;  // rows in flight per round
    uint32_t part = 0;
    for (int b = g; b < hist_blocks; b += kRowGroups * kHistRows) {
      uint32_t h[kHistRows];
#pragma unroll
      for (int r = 0; r < kHistRows; ++r) {
        const int br = b + r * kRowGroups < hist_blocks ? b + r * kRowGroups : g;  // valid, unused
        h[r] = bhist[size_t(br) * hist_stride + d];
      }
#pragma unroll
      for (int r = 0; r < kHistRows; ++r) part += b + r * kRowGroups < hist_blocks ? h[r] : 0u;
    }
    s_rows[g][d] = part;
  } else if (owner) {
    // Rows in flight per round: 16 with 256-thread tiles (at most 32 rows),
    // 32 with 1024-thread tiles (32 or 64 rows).
    constexpr int kHistRows = NT == 256 ? 16 : 32;
    for (int b = 0; b < hist_blocks; b += kHistRows) {
      uint32_t h[kHistRows][DPT];
#pragma unroll
      for (int r = 0; r < kHistRows; ++r)
#pragma unroll
        for (int i = 0; i < DPT; ++i) {
          const int br = b + r < hist_blocks ? b + r : b;  // repeat a valid row, unused
          h[r][i] = bhist[size_t(br) * hist_stride + tid * DPT + i];
        }
#pragma unroll
      for (int r = 0; r < kHistRows; ++r)
#pragma unroll
        for (int i = 0; i < DPT; ++i) dig_total[i] += b + r < hist_blocks ? h[r][i] : 0u;
    }
  }
  for (int i = tid; i < kWaves * kRadix / 2; i += NT)
    reinterpret_cast<uint32_t*>(&s_cnt[0][0])[i] = 0;
  __syncthreads();
  if constexpr (kRowGroups > 1) {
    if (owner)
#pragma unroll
      for (int g = 0; g < kRowGroups; ++g) dig_total[0] += s_rows[g][tid];
  }
  const int tile = first_lane(static_cast<int>(s_tile));
  const int64_t base = int64_t(tile) * kTile;
  if (tile != static_cast<int>(blockIdx.x)) fetch(base);

  uint32_t dig[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t pos = base + int64_t(wave) * (kItems * kWave) + i * kWave + lane;
    dig[i] = pos < K ? digit_of(key[i], shift, mask) : kRadix;
  }
  // With the key counts (the first pass, ids in token order): each token's
  // type, loaded now and stored at the end, so that the loads fly during
  // the ranking and the look-back.
  int32_t type_of[kItems];
  if (inverse) {
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int64_t pos = base + int64_t(wave) * (kItems * kWave) + i * kWave + lane;
      const uint64_t kb = key_bits(key[i]);
      type_of[i] = pos < K && kb < n_ids ? type_of_id[kb] : 0;
    }
  }

  // Rank every key among the equal-digit keys before it in its wave.
  uint32_t rank[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const bool ok = dig[i] < kRadix;
    const uint64_t peers = match_digit<RB>(dig[i], ballot(ok));
    uint32_t prior = 0;
    if (ok) prior = s_cnt[wave][dig[i]];
    const uint32_t below = popc_below(peers);
    rank[i] = prior + below;
    if (ok && below == 0) s_cnt[wave][dig[i]] = static_cast<uint16_t>(prior + __popcll(peers));
  }
  __syncthreads();

  // Per-wave exclusive offsets and tile counts of this thread's digits,
  // published at once for the tiles after this one.
  uint32_t tot[DPT];
  uint32_t tsum = 0, gsum = 0;
#pragma unroll
  for (int i = 0; i < DPT; ++i) {
    tot[i] = 0;
    if (owner) {
      const int d = tid * DPT + i;
      uint32_t t = 0;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const uint32_t c = s_cnt[w][d];
        s_cnt[w][d] = static_cast<uint16_t>(t);
        t += c;
      }
      tot[i] = t;
      tsum += t;
      gsum += dig_total[i];
      st_agent(status + size_t(tile) * kRadix + d, (tile == 0 ? kFlagPrefix : kFlagAgg) | t);
    }
  }
  uint32_t tile_sum, all_sum, local, gbase;
  blk_excl_sum2<kWaves>(tsum, gsum, s_scan, local, tile_sum, gbase, all_sum);

  // Decoupled look-back for this thread's digits, W predecessors per round.
  uint32_t excl[DPT];
#pragma unroll
  for (int i = 0; i < DPT; ++i) excl[i] = 0;
  if (tile > 0 && owner) {
    int j[DPT];
    bool done[DPT];
#pragma unroll
    for (int i = 0; i < DPT; ++i) { j[i] = tile - 1; done[i] = false; }
    uint32_t spins = 0;
    while (true) {
      bool all_done = true, stalled = false;
      uint32_t s[DPT][W];
#pragma unroll
      for (int i = 0; i < DPT; ++i)
#pragma unroll
        for (int r = 0; r < W; ++r)
          s[i][r] = (!done[i] && j[i] - r >= 0)
                        ? ld_agent(status + size_t(j[i] - r) * kRadix + tid * DPT + i)
                        : kFlagPrefix;
#pragma unroll
      for (int i = 0; i < DPT; ++i) {
        if (done[i]) continue;
        bool stop = false;
        int used = 0;
#pragma unroll
        for (int r = 0; r < W; ++r) {
          if (!stop) {
            const uint32_t f = wc.force_fail ? 0u : s[i][r] & ~kValMask;
            if (f == 0) {
              stop = true;
              stalled = true;
            } else {
              excl[i] += s[i][r] & kValMask;
              ++used;
              if (f == kFlagPrefix) { stop = true; done[i] = true; }
            }
          }
        }
        j[i] -= used;
        all_done &= done[i];
      }
      if (all_done) break;
      if (stalled) {
        if (++spins > wc.spin_limit) { raise_err(dev_err, LM_DEVERR_SPIN); break; }
        __builtin_amdgcn_s_sleep(1);
      }
    }
#pragma unroll
    for (int i = 0; i < DPT; ++i)
      st_agent(status + size_t(tile) * kRadix + tid * DPT + i,
               kFlagPrefix | ((excl[i] + tot[i]) & kValMask));
  }
  if (owner) {
#pragma unroll
    for (int i = 0; i < DPT; ++i) {
      const int d = tid * DPT + i;
      s_local[d] = static_cast<int32_t>(local);
      s_shift[d] = static_cast<int32_t>(gbase + excl[i]) - static_cast<int32_t>(local);
      local += tot[i];
      gbase += dig_total[i];
    }
  }
  __syncthreads();

  // Reorder the tile in LDS by digit (stable), then write digit runs out.
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (dig[i] < kRadix) {
      const int lp = s_local[dig[i]] + static_cast<int>(s_cnt[wave][dig[i]]) + static_cast<int>(rank[i]);
      s_keys[lp] = key[i];
      s_vals[lp] = val[i];
    }
  }
  __syncthreads();
  const int n = static_cast<int>(K - base < kTile ? K - base : kTile);
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int jj = tid + i * NT;
    if (jj < n) {
      const KeyT k = s_keys[jj];
      const int gp = s_shift[digit_of(k, shift, mask)] + jj;
      // Only a look-back that gave up (LM_DEVERR_SPIN) leaves gp out of
      // range; never write outside the buffers.
      if (static_cast<uint32_t>(gp) < static_cast<uint32_t>(K)) {
        if (keys_out) keys_out[gp] = k;
        int32_t v = s_vals[jj];
        if (pk.mode == 1)
          v = static_cast<int32_t>((digit_of(k, pk.shift, (1u << pk.nbits) - 1) << pk.pos_bits) |
                                   static_cast<uint32_t>(v));
        vals_out[gp] = v;
      }
    }
  }
  if (inverse) {
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int64_t pos = base + int64_t(wave) * (kItems * kWave) + i * kWave + lane;
      if (pos < K) inverse[pos] = type_of[i];
    }
  }
}

// ---------------------------------------------------------------------------
// Tile-local passes. Where an input takes at most 64 tiles, each radix pass
// sorts its tile by the pass's digit in LDS and writes it back over the
// tile's own range, publishing for every digit d one word,
// (start of d within the tile) << 16 | (keys of d in the tile). The pass's
// global (stable) order is then implied: the keys of digit d from tile t
// begin at D(d) + the counts of d in the tiles before t, where D(d) counts
// the keys of smaller digits. The next pass, and the dedup after the last,
// gather the range of that order they own from the tiles' runs. No pass waits
// on another workgroup and no histogram kernel runs first: each workgroup
// adds up the counts of every tile (one column of words per digit) instead.
// ---------------------------------------------------------------------------
constexpr uint32_t kRunCountMask = 0xFFFFu;
#ifndef LMZ_UNIQUE_RUN_U
#define LMZ_UNIQUE_RUN_U 16            // run words a thread loads per round in run_total
#endif

// Keys of digit d over every tile of the previous pass, for thread d < R (0
// for the others); R is a power of two. The threads split the rows: thread
// tid adds up rows g, g + G, ... of digit tid % R (g = tid / R, G = the
// number of such groups, at most 16), and thread d then adds the G sums.
template <int NT>
__device__ __forceinline__ uint32_t run_total(const uint32_t* __restrict__ runs, int tiles,
                                              int rstride, int R, uint32_t* s_part) {
  const int tid = threadIdx.x;
  const int G = NT / R < 16 ? NT / R : 16;
  const int d = tid & (R - 1), g = tid / R;
  uint32_t part = 0;
  if (g < G) {
    // Loads in flight per round: 16 measured 1.6 us faster per call than 8
    // at 65,536 ids (three gathering kernels), 32 slower than 8.
    constexpr int kU = LMZ_UNIQUE_RUN_U;
    for (int t0 = g; t0 < tiles; t0 += kU * G) {
      uint32_t w[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int t = t0 + u * G < tiles ? t0 + u * G : t0;  // repeat a valid row, unused
        w[u] = runs[size_t(t) * rstride + d];
      }
#pragma unroll
      for (int u = 0; u < kU; ++u) part += t0 + u * G < tiles ? (w[u] & kRunCountMask) : 0u;
    }
    s_part[g * R + d] = part;
  }
  __syncthreads();
  uint32_t tot = 0;
  if (tid < R)
    for (int j = 0; j < G; ++j) tot += s_part[j * R + tid];
  return tot;
}

// Marks where each (digit, tile) run starts among the positions gs .. gs+m-1
// (m >= 1) of the previous pass's order: s_mark[e] = e at the first position
// e of a run within the range (the caller set -1 everywhere before), s_src[e]
// = the index that position is read from. Thread d < R holds digit d's total
// `tot` and its start D(d); the caller set s_lohi to {0, -1} before a barrier.
// The digits that reach into the range form one interval, from the digit
// holding position gs to the one holding gs+m-1. A wave takes one digit of it
// at a time, lane t the run of tile t (tiles <= 64), and a wave prefix sum
// places the runs.
template <int NT>
__device__ __forceinline__ void mark_runs(const uint32_t* __restrict__ runs, int tiles,
                                          int rstride, int tile_keys, int R, uint32_t tot,
                                          uint32_t start, int64_t gs, int m, int* s_mark,
                                          int* s_src, uint32_t* s_dstart, int* s_lohi) {
  constexpr int kWaves = NT / kWave;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);
  if (tid < R) {
    s_dstart[tid] = start;
    if (tot > 0 && int64_t(start) <= gs && int64_t(start) + tot > gs) s_lohi[0] = tid;
    if (tot > 0 && int64_t(start) < gs + m && int64_t(start) + tot >= gs + m) s_lohi[1] = tid;
  }
  __syncthreads();
  const int dlo = first_lane(s_lohi[0]);
  const int dhi = first_lane(s_lohi[1] < R ? s_lohi[1] : R - 1);
  auto place = [&](uint32_t w, uint32_t dstart) {
    const uint32_t c = w & kRunCountMask;
    const int64_t g =
        int64_t(dstart) + (static_cast<uint32_t>(dpp_incl_scan(static_cast<int>(c), OpAdd(), 0)) - c);
    const int64_t lo = g > gs ? g : gs;
    const int64_t hi = g + c < gs + m ? g + c : gs + m;
    if (lo < hi) {
      const int e = static_cast<int>(lo - gs);
      s_mark[e] = e;
      s_src[e] = lane * tile_keys + static_cast<int>(w >> 16) + static_cast<int>(lo - g);
    }
  };
  // Two digits per round: their loads fly together.
  for (int d0 = dlo + wave; d0 <= dhi; d0 += 2 * kWaves) {
    const int d1 = d0 + kWaves;
    const bool two = d1 <= dhi;
    const uint32_t w0 = lane < tiles ? runs[size_t(lane) * rstride + d0] : 0u;
    const uint32_t w1 = two && lane < tiles ? runs[size_t(lane) * rstride + d1] : 0u;
    place(w0, s_dstart[d0]);
    if (two) place(w1, s_dstart[d1]);
  }
  __syncthreads();
}

// s_mark[e] = the start of the run that holds position e (the last mark at
// or before e), for e < m; thread t takes positions t*CH .. t*CH + CH - 1.
template <int NT, int CH>
__device__ __forceinline__ void spread_marks(int* s_mark, int m, int* s_maxs) {
  constexpr int kWaves = NT / kWave;
  const int e0 = static_cast<int>(threadIdx.x) * CH;
  int v[CH];
  int run = -1;
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    v[c] = e0 + c < m ? s_mark[e0 + c] : -1;
    run = v[c] > run ? v[c] : run;
  }
  int total;
  int before = blk_excl_max<kWaves>(run, s_maxs, total);
#pragma unroll
  for (int c = 0; c < CH; ++c) {
    before = v[c] > before ? v[c] : before;
    if (e0 + c < m) s_mark[e0 + c] = before;
  }
  __syncthreads();
}

// The index position e of the range is read from. Counts that do not add up
// (never for counts a pass published) set `bad` and give index 0.
__device__ __forceinline__ int run_src(const int* s_mark, const int* s_src, int e, int K,
                                       bool& bad) {
  const int h = s_mark[e];
  const int src = h >= 0 ? s_src[h] + (e - h) : -1;
  const bool ok = static_cast<uint32_t>(src) < static_cast<uint32_t>(K);
  bad |= !ok;
  return ok ? src : 0;
}

// ---------------------------------------------------------------------------
// k_sort_local: one stable radix pass over the digit (key >> shift) &
// (2^nbits - 1), nbits <= RB, within tile blockIdx.x. The first pass
// (GATHER = false) reads the ids, checks their range and clears the dedup's
// ticket and look-back words; later passes gather their tile's positions of
// the previous pass's order. Ranking as in k_onesweep (ballot matching, per-
// wave counters), then the tile is reordered in LDS and written back over
// the tile's range, and each digit's run word is published.
// ---------------------------------------------------------------------------
template <typename KeyT, int RB, int NT, int ITEMS, bool GATHER>
__global__ __launch_bounds__(NT) void k_sort_local(
    const KeyT* __restrict__ keys_in, const int32_t* __restrict__ vals_in, int K, uint64_t V,
    int shift, int nbits, const uint32_t* __restrict__ prev_runs, int prev_nbits,
    KeyT* __restrict__ keys_out, int32_t* __restrict__ vals_out, uint32_t* __restrict__ runs,
    int rstride, uint32_t* __restrict__ clear, int64_t clear_words,
    int32_t* __restrict__ dev_err) {
  constexpr int kWaves = NT / kWave;
  constexpr int kItems = ITEMS;
  constexpr int kTile = NT * kItems;
  constexpr int kRadix = 1 << RB;
  static_assert(kRadix <= NT, "a thread per digit");
  static_assert(kTile <= int(kRunCountMask), "run starts and counts fit 16 bits");
  constexpr int kG = GATHER ? 1 : 0;
  __shared__ KeyT s_keys[kTile];
  __shared__ int32_t s_vals[kTile];
  __shared__ uint16_t s_cnt[kWaves][kRadix];  // per-wave digit counts, then offsets
  __shared__ int32_t s_local[kRadix];         // tile-local start of each digit
  __shared__ uint32_t s_scan[kWaves];
  __shared__ int s_maxs[kWaves];
  __shared__ int s_mark[kG * kTile + 1];
  __shared__ int s_src[kG * kTile + 1];
  __shared__ uint32_t s_dstart[kG * NT + 1];  // also the partial totals
  __shared__ int s_lohi[2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);
  const int tile = blockIdx.x;
  const int64_t base = int64_t(tile) * kTile;
  const int n = static_cast<int>(K - base < kTile ? K - base : kTile);
  const uint32_t mask = nbits > 0 ? (1u << nbits) - 1 : 0u;
  for (int i = tid; i < kWaves * kRadix / 2; i += NT)
    reinterpret_cast<uint32_t*>(&s_cnt[0][0])[i] = 0;

  // Item i of a lane is tile position wave*64*ITEMS + i*64 + lane: (wave, i,
  // lane) order is position order.
  KeyT key[kItems];
  int32_t val[kItems];
  if constexpr (!GATHER) {
    for (int64_t i = int64_t(blockIdx.x) * NT + tid; i < clear_words; i += int64_t(gridDim.x) * NT)
      clear[i] = 0;
    bool bad = false;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int64_t pos = base + int64_t(wave) * (kItems * kWave) + i * kWave + lane;
      const bool ok = pos < K;
      key[i] = ok ? keys_in[pos] : KeyT(0);
      val[i] = static_cast<int32_t>(pos);
      bad |= ok && key_bits(key[i]) >= V;
    }
    if (ballot(bad) && lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
  } else {
    for (int e = tid; e < n; e += NT) s_mark[e] = -1;
    if (tid == 0) { s_lohi[0] = 0; s_lohi[1] = -1; }
    const int R = 1 << prev_nbits;
    const uint32_t tot = run_total<NT>(prev_runs, gridDim.x, rstride, R, s_dstart);
    uint32_t all;
    const uint32_t start = blk_excl_sum<kWaves>(tot, s_scan, all);
    mark_runs<NT>(prev_runs, gridDim.x, rstride, kTile, R, tot, start, base, n, s_mark, s_src,
                  s_dstart, s_lohi);
    spread_marks<NT, kItems>(s_mark, n, s_maxs);
    bool bad = false;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int e = wave * (kItems * kWave) + i * kWave + lane;
      key[i] = KeyT(0);
      val[i] = 0;
      if (e < n) {
        const int src = run_src(s_mark, s_src, e, K, bad);
        key[i] = keys_in[src];
        val[i] = vals_in[src];
      }
    }
    if (ballot(bad) && lane == 0) raise_err(dev_err, LM_DEVERR_CAPACITY);
  }
  __syncthreads();

  uint32_t dig[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int e = wave * (kItems * kWave) + i * kWave + lane;
    dig[i] = e < n ? digit_of(key[i], shift, mask) : kRadix;
  }
  uint32_t rank[kItems];
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const bool ok = dig[i] < kRadix;
    const uint64_t peers = match_digit<RB>(dig[i], ballot(ok));
    uint32_t prior = 0;
    if (ok) prior = s_cnt[wave][dig[i]];
    const uint32_t below = popc_below(peers);
    rank[i] = prior + below;
    if (ok && below == 0) s_cnt[wave][dig[i]] = static_cast<uint16_t>(prior + __popcll(peers));
  }
  __syncthreads();

  // Per-wave exclusive offsets of digit tid, its tile count and start.
  uint32_t tot = 0;
  if (tid < kRadix) {
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const uint32_t c = s_cnt[w][tid];
      s_cnt[w][tid] = static_cast<uint16_t>(tot);
      tot += c;
    }
  }
  uint32_t tile_sum;
  const uint32_t local = blk_excl_sum<kWaves>(tot, s_scan, tile_sum);
  if (tid < kRadix) {
    s_local[tid] = static_cast<int32_t>(local);
    runs[size_t(tile) * rstride + tid] = (local << 16) | tot;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    if (dig[i] < kRadix) {
      const int lp = s_local[dig[i]] + static_cast<int>(s_cnt[wave][dig[i]]) + static_cast<int>(rank[i]);
      s_keys[lp] = key[i];
      s_vals[lp] = val[i];
    }
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int jj = tid + i * NT;
    if (jj < n) {
      keys_out[base + jj] = s_keys[jj];
      vals_out[base + jj] = s_vals[jj];
    }
  }
}

// ---------------------------------------------------------------------------
// A thread's run of N consecutive elements from p (aligned to the run's
// bytes) in 16- or 8-byte loads: the scalar form spread each load
// instruction of a wave over 64 runs, one line each, and the compiler cannot
// widen it without knowing the alignment.
// ---------------------------------------------------------------------------
template <typename T, int N>
__device__ __forceinline__ void load_run(const T* __restrict__ p, T (&out)[N]) {
  constexpr int kBytes = N * static_cast<int>(sizeof(T));
  if constexpr (kBytes % 16 == 0) {
    constexpr int kPer = 16 / sizeof(T);
#pragma unroll
    for (int c = 0; c < N / kPer; ++c) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(p + c * kPer);
      const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
      __builtin_memcpy(&out[c * kPer], w, 16);
    }
  } else if constexpr (kBytes == 8) {
    const uint64_t v = *reinterpret_cast<const uint64_t*>(p);
    __builtin_memcpy(&out[0], &v, 8);
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) out[i] = p[i];
  }
}

// ---------------------------------------------------------------------------
// k_dedup: thread t of tile `tile` owns the ITEMS sorted positions
// base + ITEMS*t .. base + ITEMS*t + ITEMS - 1 (runs read in 16-byte loads;
// the permutation too when the caller's buffer is 16-byte aligned). With
// GATHER, skeys and perm hold the last tile-local pass (k_sort_local), whose
// runs words are `runs`: the tile gathers its positions (and the one on
// either side) from them and writes the permutation to perm_out.
// ---------------------------------------------------------------------------
template <typename KeyT, int NT, int ITEMS, bool PERM_RUNS, bool GATHER>
__global__ __launch_bounds__(NT) void k_dedup(
    const KeyT* __restrict__ skeys, const int32_t* __restrict__ perm, int K, int cap,
    KeyT* __restrict__ uniq, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ inverse, int64_t* __restrict__ num_unique,
    uint64_t* __restrict__ status, uint32_t* __restrict__ ticket, int32_t* __restrict__ dev_err,
    WaitCfg wc, const uint32_t* __restrict__ runs, int runs_nbits, int rstride,
    int32_t* __restrict__ perm_out, int32_t* __restrict__ type_of_id, uint64_t n_ids) {
  constexpr int kWaves = NT / kWave;
  constexpr int kItems = ITEMS;
  constexpr int kTile = NT * kItems;
  constexpr int kG = GATHER ? 1 : 0;
  __shared__ uint32_t s_scan[kWaves];
  __shared__ int s_maxs[kWaves];
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_excl_heads;
  __shared__ int s_excl_last;
  __shared__ int s_mark[kG * (kTile + 2) + 1];
  __shared__ int s_src[kG * (kTile + 2) + 1];
  __shared__ uint32_t s_dstart[kG * NT + 1];  // also the partial totals
  __shared__ int s_lohi[2];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);
  if (tid == 0) s_tile = add_agent(ticket, 1u);
  KeyT k[kItems], kprev, knext;
  int32_t src[kItems];
  int tile;
  if constexpr (GATHER) {
    // Positions base-1 .. base+kTile of the last pass's order (within [0, K)).
    for (int e = tid; e < kTile + 2; e += NT) s_mark[e] = -1;
    if (tid == 0) { s_lohi[0] = 0; s_lohi[1] = -1; }
    const int R = 1 << runs_nbits;
    const uint32_t tot = run_total<NT>(runs, gridDim.x, rstride, R, s_dstart);
    uint32_t all;
    const uint32_t start = blk_excl_sum<kWaves>(tot, s_scan, all);
    tile = first_lane(static_cast<int>(s_tile));
    const int64_t base = int64_t(tile) * kTile;
    const int64_t gs = base > 0 ? base - 1 : 0;
    const int64_t ge = base + kTile + 1 < K ? base + kTile + 1 : K;
    const int m = static_cast<int>(ge - gs);
    mark_runs<NT>(runs, gridDim.x, rstride, kTile, R, tot, start, gs, m, s_mark, s_src, s_dstart,
                  s_lohi);
    spread_marks<NT, kItems + 1>(s_mark, m, s_maxs);
    const int64_t p0 = base + int64_t(tid) * kItems;
    bool bad = false;
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      k[i] = KeyT(0);
      src[i] = 0;
      if (p0 + i < K) {
        const int j = run_src(s_mark, s_src, static_cast<int>(p0 + i - gs), K, bad);
        k[i] = skeys[j];
        src[i] = perm[j];
      }
    }
    kprev = KeyT(0);
    knext = KeyT(0);
    if (p0 > 0 && p0 - 1 < K) kprev = skeys[run_src(s_mark, s_src, static_cast<int>(p0 - 1 - gs), K, bad)];
    if (p0 + kItems < K) knext = skeys[run_src(s_mark, s_src, static_cast<int>(p0 + kItems - gs), K, bad)];
    if (ballot(bad) && lane == 0) raise_err(dev_err, LM_DEVERR_CAPACITY);
  } else {
  auto fetch = [&](int64_t base) {
    const int64_t p0 = base + int64_t(tid) * kItems;
    if (p0 + kItems <= K) {  // a whole run: the workspace keys are 256-byte aligned
      load_run<KeyT, kItems>(skeys + p0, k);
      if constexpr (PERM_RUNS) {
        load_run<int32_t, kItems>(perm + p0, src);
      } else {
#pragma unroll
        for (int i = 0; i < kItems; ++i) src[i] = perm[p0 + i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < kItems; ++i) {
        const bool ok = p0 + i < K;
        k[i] = ok ? skeys[p0 + i] : KeyT(0);
        src[i] = ok ? perm[p0 + i] : 0;
      }
    }
    kprev = p0 > 0 && p0 - 1 < K ? skeys[p0 - 1] : KeyT(0);
    knext = p0 + kItems < K ? skeys[p0 + kItems] : KeyT(0);
  };
  fetch(int64_t(blockIdx.x) * kTile);
  __syncthreads();
  tile = first_lane(static_cast<int>(s_tile));
  if (tile != static_cast<int>(blockIdx.x)) fetch(int64_t(tile) * kTile);
  }
  const int64_t base = int64_t(tile) * kTile;
  const int64_t p0 = base + int64_t(tid) * kItems;

  // Run heads and tails as bit masks (bit i: item i), evaluated without
  // short-circuit branches: ROCm 7.2's compiler dropped `last = p` on the
  // branchy form of this loop when the head was a thread's first item.
  uint32_t hmask = 0, tmask = 0;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t p = p0 + i;
    if (p < K) {
      const KeyT prev = i == 0 ? kprev : k[i - 1];
      const KeyT next = i + 1 < kItems ? k[i + 1] : knext;
      const bool head = (p == 0) | (k[i] != prev);
      const bool tail = (p == K - 1) | (next != k[i]);
      hmask |= static_cast<uint32_t>(head) << i;
      tmask |= static_cast<uint32_t>(tail) << i;
    }
  }
  const uint32_t nheads = static_cast<uint32_t>(__popc(hmask));
  const int last_head = hmask ? static_cast<int>(p0) + (31 - __clz(static_cast<int>(hmask))) : -1;
  uint32_t tile_heads, heads_before;
  int tile_last, last_before;
  blk_excl_sum_max<kWaves>(nheads, last_head, s_scan, s_maxs, heads_before, tile_heads,
                           last_before, tile_last);

  // Wave 0: publish the tile aggregate, then look back 64 tiles per round.
  if (wave == 0) {
    uint64_t* my = status + tile;
    const uint64_t agg = (uint64_t(tile_heads) << 31) | uint64_t(tile_last + 1);
    if (lane == 0) st_agent(my, (tile == 0 ? kDFlagPrefix : kDFlagAgg) | agg);
    uint32_t eh = 0;
    int el = -1;
    if (tile > 0) {
      int j = tile - 1;
      uint32_t spins = 0;
      while (true) {
        const int pos = j - lane;
        const uint64_t s = pos >= 0 ? ld_agent(status + pos) : kDFlagPrefix;
        const uint64_t f = wc.force_fail ? 0 : s & kDFlags;
        const uint64_t notready = ballot(f == 0);
        const uint64_t prefix = ballot(f == kDFlagPrefix);
        const int first_nr = notready ? __builtin_ctzll(notready) : kWave;
        const int first_px = prefix ? __builtin_ctzll(prefix) : kWave;
        const bool done = first_px < first_nr;
        const int take = done ? first_px + 1 : first_nr;  // lanes [0, take) are consumed
        const bool mine = lane < take;
        uint32_t h = mine ? static_cast<uint32_t>((s >> 31) & kD31) : 0u;
        eh += wave_sum(h);
        // the nearest consumed predecessor that has a head holds the last one
        const int pl = static_cast<int>(s & kD31) - 1;
        const uint64_t has = ballot(mine && pl >= 0);
        if (el < 0 && has) el = read_lane(pl, __builtin_ctzll(has));
        if (done) break;
        j -= take;
        if (take == 0) {
          if (++spins > wc.spin_limit) { raise_err(dev_err, LM_DEVERR_SPIN); break; }
          __builtin_amdgcn_s_sleep(1);
        }
      }
      const int incl_last = tile_last >= 0 ? tile_last : el;
      if (lane == 0)
        st_agent(my, kDFlagPrefix | (uint64_t(eh + tile_heads) << 31) | uint64_t(incl_last + 1));
    }
    if (lane == 0) {
      s_excl_heads = eh;
      s_excl_last = el;
    }
  }
  __syncthreads();

  // Types can only outnumber cap = min(K, V) when ids lie outside [0, V)
  // (LM_DEVERR_ID_RANGE is raised then): clamp every write to the buffers.
  int seg = static_cast<int>(s_excl_heads + heads_before) - 1;
  int hp = last_before >= 0 ? last_before : s_excl_last;
  bool over = false;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t p = p0 + i;
    if (p < K) {
      const bool head = (hmask >> i) & 1u;
      seg += head ? 1 : 0;
      hp = head ? static_cast<int>(p) : hp;
      const bool in_cap = static_cast<uint32_t>(seg) < static_cast<uint32_t>(cap);
      over |= !in_cap;
      if (head && in_cap) {
        uniq[seg] = k[i];
        offsets[seg] = static_cast<int32_t>(p);
      }
      if (((tmask >> i) & 1u) && in_cap) counts[seg] = static_cast<int32_t>(p + 1 - hp);
      if (static_cast<uint32_t>(src[i]) >= static_cast<uint32_t>(K)) over = true;
      else if (!type_of_id) inverse[src[i]] = seg;
      else if (head && in_cap && key_bits(k[i]) < n_ids) type_of_id[key_bits(k[i])] = seg;
      if constexpr (GATHER) perm_out[p] = src[i];
      if (p == K - 1) {
        *num_unique = seg + 1 < cap ? seg + 1 : cap;
        offsets[seg + 1 < cap ? seg + 1 : cap] = K;
      }
    }
  }
  if (ballot(over) && lane_id() == 0) raise_err(dev_err, LM_DEVERR_CAPACITY);
}

// ---------------------------------------------------------------------------
// k_unique_block: the whole of Unique in one workgroup of 1024 threads, for
// inputs of up to 1024 * ITEMS keys. The keys stay in LDS through every
// radix pass (RB-bit digits, RB = 8..10, ranked by wave64 ballot matching as in
// k_onesweep, with digit offsets from a block scan instead of a look-back)
// and through the dedup (run heads by ballot, a scan of the head counts
// over the 16 waves), so the call is one launch with no waits between
// workgroups: a small batch is bound by latency, not by bytes. The inverse
// map, the type ids and the offsets are staged in LDS and written out
// coalesced: one CU issuing a scattered 4-byte store per token took longer
// than all the passes.
// ---------------------------------------------------------------------------
constexpr int kBlockThreads = kBlockThreadsHost;
constexpr int kBlockWaves = kBlockThreads / kWave;
constexpr size_t kLdsBytes = 160 * 1024 - 4096;  // gfx950's 160 KiB, less a margin

// The one workgroup's keys and values in LDS (N of each, and one value
// more). With 4-byte keys a key and its value sit side by side, so that the
// reorder, the read-back and the dedup move a pair with one 8-byte access;
// 8-byte keys keep two arrays.
template <typename KeyT, int N>
struct BlockPairs {
  KeyT keys[N];
  int32_t vals[N + 1];
  __device__ void put(int i, KeyT k, int32_t v) { keys[i] = k; vals[i] = v; }
  __device__ void get(int i, KeyT& k, int32_t& v) const { k = keys[i]; v = vals[i]; }
  __device__ KeyT& key(int i) { return keys[i]; }
  __device__ int32_t& val(int i) { return vals[i]; }
};
template <int N>
struct BlockPairs<int32_t, N> {
  int2 kv[N + 1];
  __device__ void put(int i, int32_t k, int32_t v) { kv[i] = make_int2(k, v); }
  __device__ void get(int i, int32_t& k, int32_t& v) const {
    const int2 t = kv[i];
    k = t.x;
    v = t.y;
  }
  __device__ int32_t& key(int i) { return kv[i].x; }
  __device__ int32_t& val(int i) { return kv[i].y; }
};

template <typename KeyT, int ITEMS, int RB>
__global__ __launch_bounds__(kBlockThreads) void k_unique_block(
    const KeyT* __restrict__ ids, int K, uint64_t V, int passes, PassBits pb, int cap,
    KeyT* __restrict__ uniq, int32_t* __restrict__ counts, int32_t* __restrict__ offsets,
    int32_t* __restrict__ inverse, int32_t* __restrict__ perm, int64_t* __restrict__ num_unique,
    int32_t* __restrict__ dev_err) {
  constexpr int kRadix = 1 << RB;
  static_assert(kRadix <= kBlockThreads, "one thread per digit");
  constexpr int kN = kBlockThreads * ITEMS;
  __shared__ BlockPairs<KeyT, kN> s_kv;  // + 1 value: the end offset of the last type
  // Per-wave digit counts, then offsets. Where the LDS holds two sets, pass
  // p uses set p & 1 and the next pass's counters are cleared while this
  // pass still runs; otherwise each pass clears the one set first.
  constexpr size_t kCntBytes = sizeof(uint16_t) * kBlockWaves * kRadix;
  constexpr size_t kLdsRest = sizeof(KeyT) * kN + sizeof(int32_t) * (kN + 1) +
                              sizeof(uint32_t) * (kRadix + kBlockWaves);
  constexpr int kCntSets = kLdsRest + 2 * kCntBytes <= kLdsBytes ? 2 : 1;
  __shared__ uint16_t s_cnt[kCntSets][kBlockWaves][kRadix];
  // The dedup's offsets get an array of their own where the LDS has room
  // beside the counter sets, so that they are staged together with the
  // inverse map and the type ids (one barrier and one pass fewer).
  constexpr bool kOffLds = kLdsRest + kCntSets * kCntBytes + sizeof(int32_t) * (kN + 1) <= kLdsBytes;
  __shared__ int32_t s_off[kOffLds ? kN + 1 : 1];
  __shared__ uint32_t s_start[kRadix];             // first sorted position of each digit
  __shared__ uint32_t s_scan[kBlockWaves];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = first_lane(tid >> 6);

  // Item i of a lane is position wave * 64 * ITEMS + i * 64 + lane: (wave, i,
  // lane) order is position order, which keeps every pass stable.
  KeyT key[ITEMS];
  int32_t val[ITEMS];
  bool bad = false;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
    key[i] = pos < K ? ids[pos] : KeyT(0);
    val[i] = pos;
  }
  // The first pass's counters, cleared while the ids are in flight.
  for (int j = tid; j < kBlockWaves * kRadix / 2; j += kBlockThreads)
    reinterpret_cast<uint32_t*>(&s_cnt[0][0][0])[j] = 0;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
    bad |= pos < K && key_bits(key[i]) >= V;
  }
  if (ballot(bad) && lane == 0) raise_err(dev_err, LM_DEVERR_ID_RANGE);
  __syncthreads();

  for (int p = 0; p < passes; ++p) {
    const int shift = pb.shift[p], nbits = pb.nbits[p];
    const uint32_t mask = nbits > 0 ? (1u << nbits) - 1 : 0u;
    uint16_t (*cnt)[kRadix] = s_cnt[p % kCntSets];
    if (kCntSets == 1 && p > 0) {
      for (int j = tid; j < kBlockWaves * kRadix / 2; j += kBlockThreads)
        reinterpret_cast<uint32_t*>(&cnt[0][0])[j] = 0;
      __syncthreads();
    }
    uint32_t dig[ITEMS], rank[ITEMS];
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
      dig[i] = pos < K ? digit_of(key[i], shift, mask) : kRadix;
    }
    // Rank every key among the equal-digit keys before it in its wave.
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      const bool ok = dig[i] < kRadix;
      const uint64_t peers = match_digit<RB>(dig[i], ballot(ok));
      uint32_t prior = 0;
      if (ok) prior = cnt[wave][dig[i]];
      const uint32_t below = popc_below(peers);
      rank[i] = prior + below;
      if (ok && below == 0) cnt[wave][dig[i]] = static_cast<uint16_t>(prior + __popcll(peers));
    }
    // The next pass's counters: their last reader, the pass before this
    // one, finished before this pass began.
    if (kCntSets == 2 && p + 1 < passes)
      for (int j = tid; j < kBlockWaves * kRadix / 2; j += kBlockThreads)
        reinterpret_cast<uint32_t*>(&s_cnt[(p + 1) % kCntSets][0][0])[j] = 0;
    __syncthreads();
    // Thread d < kRadix: per-wave offsets within digit d and its total; a
    // block scan of the totals gives each digit's first sorted position.
    uint32_t tot = 0;
    if (tid < kRadix) {
#pragma unroll
      for (int w = 0; w < kBlockWaves; ++w) {
        const uint32_t c = cnt[w][tid];
        cnt[w][tid] = static_cast<uint16_t>(tot);
        tot += c;
      }
    }
    uint32_t all;
    const uint32_t start = blk_excl_sum<kBlockWaves>(tot, s_scan, all);
    if (tid < kRadix) s_start[tid] = start;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < ITEMS; ++i) {
      if (dig[i] < kRadix) {
        const int dst = static_cast<int>(s_start[dig[i]] + cnt[wave][dig[i]] + rank[i]);
        s_kv.put(dst, key[i], val[i]);
      }
    }
    __syncthreads();
    if (p + 1 < passes) {
#pragma unroll
      for (int i = 0; i < ITEMS; ++i) {
        const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
        s_kv.get(pos, key[i], val[i]);
      }
      __syncthreads();  // every read done before the next pass overwrites
    }
  }

  // Dedup, in the same (wave, i, lane) order: position pos is a run head when
  // its key differs from the one before. The perm goes out as it is read.
  KeyT k[ITEMS];
  int32_t src[ITEMS];
  uint64_t hm[ITEMS];
  uint32_t wave_heads = 0;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
    const bool ok = pos < K;
    k[i] = KeyT(0);
    src[i] = 0;
    if (ok) s_kv.get(pos, k[i], src[i]);
    const KeyT before = ok && pos > 0 ? s_kv.key(pos - 1) : KeyT(0);
    hm[i] = ballot(ok && (pos == 0 || k[i] != before));
    wave_heads += static_cast<uint32_t>(__popcll(hm[i]));
    if (ok) perm[pos] = src[i];
  }
  if (lane == 0) s_scan[wave] = wave_heads;
  __syncthreads();  // also: every read of the pairs is done
  uint32_t heads_before = 0, U = 0;
#pragma unroll
  for (int w = 0; w < kBlockWaves; ++w) {
    const uint32_t x = s_scan[w];
    heads_before += w < wave ? x : 0u;
    U += x;
  }
  // Types can only outnumber cap = min(K, V) when ids lie outside [0, V)
  // (LM_DEVERR_ID_RANGE is raised then): every write stays in the buffers.
  const int Uc = static_cast<int>(U) < cap ? static_cast<int>(U) : cap;
  // seg[i]: the type of position pos (heads up to and including it, minus 1).
  int seg[ITEMS];
  uint32_t run = heads_before;
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const bool head = (hm[i] >> lane) & 1u;
    seg[i] = static_cast<int>(run + popc_below(hm[i]) + (head ? 1u : 0u)) - 1;
    run += static_cast<uint32_t>(__popcll(hm[i]));
  }
  // Stage the inverse map (by token) and the type ids in LDS (and, with
  // kOffLds, the first position of every type), then write them out
  // coalesced.
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
    if (pos < K) {
      const bool head = (hm[i] >> lane) & 1u;
      s_kv.val(src[i]) = seg[i];
      if (head && seg[i] < Uc) s_kv.key(seg[i]) = k[i];
      if constexpr (kOffLds)
        if (head && seg[i] <= Uc) s_off[seg[i]] = pos;
    }
  }
  if constexpr (kOffLds) {
    if (tid == 0 && static_cast<int>(U) == Uc) s_off[Uc] = K;
    __syncthreads();
    for (int j = tid; j < K; j += kBlockThreads) inverse[j] = s_kv.val(j);
    for (int j = tid; j < Uc; j += kBlockThreads) {
      const int o = s_off[j];
      uniq[j] = s_kv.key(j);
      offsets[j] = o;
      counts[j] = s_off[j + 1] - o;
    }
    if (tid == 0) {
      offsets[Uc] = K;
      *num_unique = Uc;
      if (static_cast<int>(U) > cap) raise_err(dev_err, LM_DEVERR_CAPACITY);
    }
    return;
  }
  __syncthreads();
  for (int j = tid; j < K; j += kBlockThreads) inverse[j] = s_kv.val(j);
  for (int j = tid; j < Uc; j += kBlockThreads) uniq[j] = s_kv.key(j);
  __syncthreads();
  // Stage the first position of every type, then write offsets and counts.
#pragma unroll
  for (int i = 0; i < ITEMS; ++i) {
    const int pos = wave * (ITEMS * kWave) + i * kWave + lane;
    if (pos < K && ((hm[i] >> lane) & 1u) && seg[i] <= Uc) s_kv.val(seg[i]) = pos;
  }
  if (tid == 0 && static_cast<int>(U) == Uc) s_kv.val(Uc) = K;
  __syncthreads();
  for (int j = tid; j < Uc; j += kBlockThreads) {
    const int o = s_kv.val(j);
    offsets[j] = o;
    counts[j] = s_kv.val(j + 1) - o;
  }
  if (tid == 0) {
    offsets[Uc] = K;
    *num_unique = Uc;
    if (static_cast<int>(U) > cap) raise_err(dev_err, LM_DEVERR_CAPACITY);
  }
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

// k_inverse_types: inverse[i] = type_of_id[ids[i]] in token order (after a
// dedup that wrote each id's type to type_of_id). Four ids per thread per
// round, with 16-byte loads and stores where ids and inverse are 16-byte
// aligned; ids outside [0, n_ids) (an error already raised by the
// histogram) read no table entry.
constexpr int kInvThreads = 256;
constexpr int kInvItems = 4;
constexpr int kInvMaxBlocks = 2048;
template <typename KeyT, bool VEC>
__global__ __launch_bounds__(kInvThreads) void k_inverse_types(
    const KeyT* __restrict__ ids, int K, uint64_t n_ids, const int32_t* __restrict__ type_of_id,
    int32_t* __restrict__ inverse) {
  const int64_t stride = int64_t(gridDim.x) * kInvThreads * kInvItems;
  for (int64_t i0 = (int64_t(blockIdx.x) * kInvThreads + threadIdx.x) * kInvItems; i0 < K;
       i0 += stride) {
    if (VEC && i0 + kInvItems <= K) {
      KeyT k[kInvItems];
      load_run<KeyT, kInvItems>(ids + i0, k);
      int32_t t[kInvItems];
#pragma unroll
      for (int j = 0; j < kInvItems; ++j) {
        const uint64_t kb = key_bits(k[j]);
        t[j] = kb < n_ids ? type_of_id[kb] : 0;
      }
      *reinterpret_cast<int4*>(inverse + i0) = make_int4(t[0], t[1], t[2], t[3]);
    } else {
      for (int j = 0; j < kInvItems && i0 + j < K; ++j) {
        const uint64_t kb = key_bits(ids[i0 + j]);
        inverse[i0 + j] = kb < n_ids ? type_of_id[kb] : 0;
      }
    }
  }
}

template <typename KeyT, int RB, int NT, int ITEMS>
static hipError_t launch_pass(const UniqueLayout& L, int p, const KeyT* kin, const int32_t* vin,
                              KeyT* kout, int32_t* vout, int K, uint32_t* bhist,
                              uint32_t* status, uint32_t* tickets, int32_t* dev_err,
                              const int32_t* type_of_id, uint32_t n_ids, int32_t* inverse,
                              int shift, PackCfg pk, hipStream_t st) {
  k_onesweep<KeyT, RB, NT, ITEMS><<<L.tiles, NT, 0, st>>>(
      kin, vin, kout, vout, K, shift, L.nbits[p], bhist + size_t(p) * L.rstride,
      L.hist_blocks, L.passes * L.rstride, status + size_t(p) * L.tiles * L.rstride, tickets + p,
      dev_err, wait_cfg(), type_of_id, n_ids, inverse, pk);
  return hipGetLastError();
}

template <typename KeyT>
static int run_unique(const KeyT* ids, int K, int64_t V, KeyT* uniq, int32_t* counts,
                      int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
                      int32_t* dev_err, char* ws, const UniqueLayout& L, hipStream_t st) {
  if (K == 0) {
    k_unique_empty<<<1, 64, 0, st>>>(num_unique, offsets);
    return launch_status(hipGetLastError());
  }
  PassBits pb{};
  for (int p = 0; p < L.passes; ++p) {
    pb.shift[p] = L.shift[p];
    pb.nbits[p] = L.nbits[p];
  }
  const int cap = static_cast<int>(K < V ? K : V);
  if (L.block_items > 0) {
    auto launch = [&](auto items, auto rb) {
      k_unique_block<KeyT, decltype(items)::value, decltype(rb)::value>
          <<<1, kBlockThreads, 0, st>>>(ids, K, static_cast<uint64_t>(V), L.passes, pb, cap, uniq,
                                        counts, offsets, inverse, perm, num_unique, dev_err);
    };
    auto block = [&](auto items) {
      if (L.block_rb <= 8) launch(items, I<8>{});
      else if (L.block_rb == 9) launch(items, I<9>{});
      else launch(items, I<10>{});
    };
    switch (L.block_items) {
      case 1: block(I<1>{}); break;
      case 2: block(I<2>{}); break;
      case 4: block(I<4>{}); break;
      default: block(I<8>{}); break;
    }
    return launch_status(hipGetLastError());
  }
  uint32_t* bhist = reinterpret_cast<uint32_t*>(ws + L.bhist);
  uint32_t* tickets = reinterpret_cast<uint32_t*>(ws + L.tickets);
  uint32_t* status = reinterpret_cast<uint32_t*>(ws + L.status);
  uint64_t* dstatus = reinterpret_cast<uint64_t*>(ws + L.dstatus);
  KeyT* kb[2] = {reinterpret_cast<KeyT*>(ws + L.keys0), reinterpret_cast<KeyT*>(ws + L.keys1)};
  int32_t* vb[2] = {reinterpret_cast<int32_t*>(ws + L.vals0), reinterpret_cast<int32_t*>(ws + L.vals1)};

  // tickets .. end of dstatus is contiguous: k_hist (or the first
  // tile-local pass) clears it.
  const int64_t clear_words = static_cast<int64_t>((L.keys0 - L.tickets) / 4);
  if (L.gather) {
    // Tile-local passes (1024 threads and 2 keys each, or 256 threads and 4
    // keys each with digits of at most 8 bits); the runs words of pass p and
    // tile t sit in the histogram region at row p * tiles + t.
    auto passes = [&](auto nt) -> hipError_t {
      constexpr int kNT = decltype(nt)::value;
      constexpr int kIT = kNT == 256 ? kGatherSmallTileKeys / 256 : 2;
      for (int p = 0; p < L.passes; ++p) {
        const KeyT* kin = p == 0 ? ids : kb[(p - 1) & 1];
        const int32_t* vin = p == 0 ? nullptr : vb[(p - 1) & 1];
        const uint32_t* prev = p == 0 ? nullptr : bhist + size_t(p - 1) * L.tiles * L.rstride;
        const int prev_nbits = p == 0 ? 0 : L.nbits[p - 1];
        uint32_t* runs = bhist + size_t(p) * L.tiles * L.rstride;
        auto pass = [&](auto rb, auto gather) {
          k_sort_local<KeyT, decltype(rb)::value, kNT, kIT, decltype(gather)::value>
              <<<L.tiles, kNT, 0, st>>>(kin, vin, K, static_cast<uint64_t>(V), L.shift[p],
                                        L.nbits[p], prev, prev_nbits, kb[p & 1], vb[p & 1], runs,
                                        L.rstride, tickets, clear_words, dev_err);
        };
        const bool narrow = L.nbits[p] <= kSmallDigitBits;
        if constexpr (kNT == 1024) {
          if (p == 0) {
            if (narrow) pass(I<kSmallDigitBits>{}, std::false_type{});
            else pass(I<kLargeDigitBits>{}, std::false_type{});
          } else {
            if (narrow) pass(I<kSmallDigitBits>{}, std::true_type{});
            else pass(I<kLargeDigitBits>{}, std::true_type{});
          }
        } else {
          if (!narrow) return hipErrorInvalidValue;  // the layout keeps digits to 8 bits here
          if (p == 0) pass(I<kSmallDigitBits>{}, std::false_type{});
          else pass(I<kSmallDigitBits>{}, std::true_type{});
        }
        if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
      }
      const int q = L.passes - 1;
      k_dedup<KeyT, kNT, kIT, false, true><<<L.tiles, kNT, 0, st>>>(
          kb[q & 1], vb[q & 1], K, cap, uniq, counts, offsets, inverse, num_unique, dstatus,
          tickets + kMaxPasses, dev_err, wait_cfg(), bhist + size_t(q) * L.tiles * L.rstride,
          L.nbits[q], L.rstride, perm, nullptr, 0);
      return hipGetLastError();
    };
    return launch_status(L.nt == 256 ? passes(I<256>{}) : passes(I<1024>{}));
  }
  int32_t* type_of_id = nullptr;
  if (L.keycount) {
    // Counts per id, then the types and each id's type; the first pass
    // writes the inverse map and no dedup runs.
    if (L.passes * L.rstride > 2 * (1 << kLargeDigitBits)) return LM_E_UNSUPPORTED;
    uint32_t* khist = reinterpret_cast<uint32_t*>(ws + L.khist);
    type_of_id = reinterpret_cast<int32_t*>(ws + L.rank);
    k_key_hist<KeyT><<<L.key_blocks, kHistThreads, size_t(V) * 4, st>>>(
        ids, K, static_cast<int>(V), khist, tickets, clear_words, dev_err);
    k_key_scan<KeyT, kKeyScanThreads><<<L.scan_tiles, kKeyScanThreads, 0, st>>>(
        khist, L.key_blocks, static_cast<int>(V), K, L.passes, L.rstride, pb, bhist, uniq, counts,
        offsets, type_of_id, num_unique, dstatus, tickets + kMaxPasses + 1, dev_err, wait_cfg());
  } else {
    const size_t hist_lds = size_t(L.passes) * L.rstride * 4;
    if (K > LMZ_UNIQUE_HIST_RUNS_MIN_K)
      k_hist<KeyT, true><<<L.hist_blocks, kHistThreads, hist_lds, st>>>(
          ids, K, static_cast<uint64_t>(V), L.passes, L.rstride, pb, bhist, tickets, clear_words,
          dev_err);
    else
      k_hist<KeyT, false><<<L.hist_blocks, kHistThreads, hist_lds, st>>>(
          ids, K, static_cast<uint64_t>(V), L.passes, L.rstride, pb, bhist, tickets, clear_words,
          dev_err);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return launch_status(e);

  const KeyT* kin = ids;
  const int32_t* vin = nullptr;
  // Counts per id, two passes and 4-byte ids: the first pass writes the
  // second pass's digit and the position as one word (PackCfg).
  const int pos_bits = L.passes == 2 ? 32 - L.nbits[1] : 0;
  const bool packed = L.keycount && L.passes == 2 && sizeof(KeyT) == 4 && pos_bits < 32 &&
                      int64_t(K) <= (int64_t(1) << pos_bits);
  for (int p = 0; p < L.passes; ++p) {
    // The last pass with the counts per id writes the permutation only: the
    // types came from the counts, so nothing reads its sorted keys.
    KeyT* kout = (L.keycount && p == L.passes - 1) || (packed && p == 0) ? nullptr : kb[p & 1];
    int32_t* vout = p == L.passes - 1 ? perm : vb[p & 1];
    int shift = L.shift[p];
    PackCfg pk{0, 0, 0, 0};
    if (packed) {
      pk = p == 0 ? PackCfg{1, L.shift[1], L.nbits[1], pos_bits} : PackCfg{2, 0, 0, pos_bits};
      if (p == 1) shift = pos_bits;  // the digit sits above the position
    }
    // The narrowest compiled digit that holds this pass's bits.
    const bool narrow = L.nbits[p] <= kSmallDigitBits;
    const bool first = p == 0 && type_of_id;
    auto pass = [&](auto rb, auto nt, auto items) {
      return launch_pass<KeyT, decltype(rb)::value, decltype(nt)::value, decltype(items)::value>(
          L, p, kin, vin, kout, vout, K, bhist, status, tickets, dev_err,
          first ? type_of_id : nullptr, static_cast<uint32_t>(V), first ? inverse : nullptr,
          shift, pk, st);
    };
    auto by_items = [&](auto rb, auto nt) {
      if constexpr (decltype(nt)::value == 256)
        return L.items == 2 ? pass(rb, nt, I<2>{}) : pass(rb, nt, I<4>{});
      else
        return L.items == 2 ? pass(rb, nt, I<2>{})
                            : (L.items == 4 ? pass(rb, nt, I<4>{}) : pass(rb, nt, I<8>{}));
    };
    hipError_t e;
    if (L.nt == 256)
      e = narrow ? by_items(I<kSmallDigitBits>{}, I<256>{}) : by_items(I<kLargeDigitBits>{}, I<256>{});
    else
      e = narrow ? by_items(I<kSmallDigitBits>{}, I<1024>{})
                 : by_items(I<kLargeDigitBits>{}, I<1024>{});
    if (e != hipSuccess) return launch_status(e);
    kin = packed && p == 0 ? reinterpret_cast<const KeyT*>(vout) : kout;  // the packed words
    vin = packed && p == 0 ? nullptr : vout;
  }
  if (L.keycount)  // the scan wrote the types, the first pass the inverse map
    return launch_status(hipGetLastError());
  const bool perm_runs = (reinterpret_cast<uintptr_t>(perm) & 15) == 0;
  int32_t* tmap = L.typemap ? reinterpret_cast<int32_t*>(ws + L.rank) : nullptr;
  auto dedup = [&](auto nt, auto items) {
    constexpr int NT = decltype(nt)::value, IT = decltype(items)::value;
    if (perm_runs)
      k_dedup<KeyT, NT, IT, true, false><<<L.tiles, NT, 0, st>>>(
          kin, perm, K, cap, uniq, counts, offsets, inverse, num_unique, dstatus,
          tickets + kMaxPasses, dev_err, wait_cfg(), nullptr, 0, 0, nullptr, tmap,
          static_cast<uint64_t>(V));
    else
      k_dedup<KeyT, NT, IT, false, false><<<L.tiles, NT, 0, st>>>(
          kin, perm, K, cap, uniq, counts, offsets, inverse, num_unique, dstatus,
          tickets + kMaxPasses, dev_err, wait_cfg(), nullptr, 0, 0, nullptr, tmap,
          static_cast<uint64_t>(V));
  };
  if (L.nt == 256) {
    if (L.items == 2) dedup(I<256>{}, I<2>{});
    else dedup(I<256>{}, I<4>{});
  } else {
    if (L.items == 2) dedup(I<1024>{}, I<2>{});
    else if (L.items == 4) dedup(I<1024>{}, I<4>{});
    else dedup(I<1024>{}, I<8>{});
  }
  if (tmap) {
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return launch_status(e);
    const int64_t per_block = int64_t(kInvThreads) * kInvItems;
    int64_t blocks = (K + per_block - 1) / per_block;
    if (blocks > kInvMaxBlocks) blocks = kInvMaxBlocks;
    const bool vec = ((reinterpret_cast<uintptr_t>(ids) | reinterpret_cast<uintptr_t>(inverse)) & 15) == 0;
    if (vec)
      k_inverse_types<KeyT, true><<<static_cast<int>(blocks), kInvThreads, 0, st>>>(
          ids, K, static_cast<uint64_t>(V), tmap, inverse);
    else
      k_inverse_types<KeyT, false><<<static_cast<int>(blocks), kInvThreads, 0, st>>>(
          ids, K, static_cast<uint64_t>(V), tmap, inverse);
  }
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
