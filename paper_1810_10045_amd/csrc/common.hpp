// Device-side building blocks shared by the lmzipf kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/lmzipf.h"

namespace lmz {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Wave-level primitives
// ---------------------------------------------------------------------------

__device__ __forceinline__ int lane_id() {
  return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

// Number of set bits of `mask` in lanes below this one.
__device__ __forceinline__ int popc_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ int read_lane(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

__device__ __forceinline__ int first_lane(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ int first_lane(unsigned v) { return first_lane(static_cast<int>(v)); }

__device__ __forceinline__ int64_t read_lane(int64_t v, int lane) {
  const uint64_t u = static_cast<uint64_t>(v);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u), lane));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(u >> 32), lane));
  return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

__device__ __forceinline__ int64_t first_lane(int64_t v) {
  const uint64_t u = static_cast<uint64_t>(v);
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(u)));
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(u >> 32)));
  return static_cast<int64_t>((uint64_t(hi) << 32) | lo);
}

// Inclusive prefix sum over the 64 lanes of a wave.
template <typename T>
__device__ __forceinline__ T wave_incl_sum(T v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    T t = __shfl_up(v, off, kWave);
    if (lane >= off) v += t;
  }
  return v;
}

// Inclusive prefix maximum over the 64 lanes of a wave.
__device__ __forceinline__ int wave_incl_max(int v) {
  const int lane = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    int t = __shfl_up(v, off, kWave);
    if (lane >= off && t > v) v = t;
  }
  return v;
}

// Exclusive prefix sum over a block of NW waves. `lds` holds NW entries.
// Returns this thread's exclusive prefix; `total` gets the block sum.
template <int NW, typename T>
__device__ __forceinline__ T block_excl_sum(T v, T* lds, T& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  T incl = wave_incl_sum(v);
  if (lane == 63) lds[wave] = incl;
  __syncthreads();
  T before = T(0), all = T(0);
#pragma unroll
  for (int w = 0; w < NW; ++w) {
    const T x = lds[w];
    before += w < wave ? x : T(0);
    all += x;
  }
  __syncthreads();
  total = all;
  return before + incl - v;
}

template <typename T>
__device__ __forceinline__ T block256_excl_sum(T v, T* lds, T& total) {
  return block_excl_sum<4, T>(v, lds, total);
}

// Exclusive prefix maximum over a block of NW waves (-1 for thread 0).
template <int NW>
__device__ __forceinline__ int block_excl_max(int v, int* lds, int& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = wave_incl_max(v);
  int prev = __shfl_up(incl, 1, kWave);
  if (lane == 0) prev = -1;
  if (lane == 63) lds[wave] = incl;
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

__device__ __forceinline__ int block256_excl_max(int v, int* lds, int& total) {
  return block_excl_max<4>(v, lds, total);
}

// ---------------------------------------------------------------------------
// Inter-workgroup communication. The 8 XCDs of an MI355X each have their own
// L2, so every flag another workgroup polls is accessed with agent-scope
// atomics (the compiler then bypasses the non-coherent caches).
// ---------------------------------------------------------------------------

template <typename T>
__device__ __forceinline__ T ld_agent(const T* p) {
  return __hip_atomic_load(const_cast<T*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T>
__device__ __forceinline__ T add_agent(T* p, T v) {
  return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void raise_err(int32_t* dev_err, int bit) {
  if (dev_err) __hip_atomic_fetch_or(dev_err, bit, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Upper bound on polls of another workgroup's status word before giving up
// with LM_DEVERR_SPIN (every legitimate wait ends within microseconds).
constexpr uint32_t kSpinLimit = 1u << 20;

// ---------------------------------------------------------------------------
// Row loads: VEC consecutive gradient values as fp32.
// ---------------------------------------------------------------------------

struct bf16_t {
  uint16_t bits;
};

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Gradient rows are read exactly once: stream them past the caches.
#ifndef LMZ_STREAM_LOADS
#define LMZ_STREAM_LOADS 1
#endif
template <typename T>
__device__ __forceinline__ T stream_load(const T* p) {
#if LMZ_STREAM_LOADS
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

template <typename GT, int VEC>
struct RowVec;

template <>
struct RowVec<float, 4> {
  using raw_t = f32x4;
  static __device__ __forceinline__ raw_t load(const float* p) {
    return stream_load(reinterpret_cast<const f32x4*>(p));
  }
  static __device__ __forceinline__ void add(float* acc, const raw_t& r) {
    acc[0] += r.x; acc[1] += r.y; acc[2] += r.z; acc[3] += r.w;
  }
};

template <>
struct RowVec<float, 1> {
  using raw_t = float;
  static __device__ __forceinline__ raw_t load(const float* p) { return stream_load(p); }
  static __device__ __forceinline__ void add(float* acc, const raw_t& r) { acc[0] += r; }
};

template <>
struct RowVec<bf16_t, 8> {
  using raw_t = u32x4;
  static __device__ __forceinline__ raw_t load(const bf16_t* p) {
    return stream_load(reinterpret_cast<const u32x4*>(p));
  }
  static __device__ __forceinline__ void add(float* acc, const raw_t& r) {
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      acc[2 * i] += __uint_as_float(w[i] << 16);
      acc[2 * i + 1] += __uint_as_float(w[i] & 0xffff0000u);
    }
  }
};

template <>
struct RowVec<bf16_t, 1> {
  using raw_t = uint32_t;
  static __device__ __forceinline__ raw_t load(const bf16_t* p) {
    return static_cast<uint32_t>(stream_load(&p->bits));
  }
  static __device__ __forceinline__ void add(float* acc, const raw_t& r) {
    acc[0] += bf16_to_f32(r);
  }
};

// Store VEC fp32 values (16-byte stores when VEC is a multiple of 4).
template <int VEC>
__device__ __forceinline__ void store_vec(float* p, const float* v) {
  if constexpr (VEC % 4 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 4)
      *reinterpret_cast<float4*>(p + i) = make_float4(v[i], v[i + 1], v[i + 2], v[i + 3]);
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) p[i] = v[i];
  }
}

// ---------------------------------------------------------------------------
// binary16 payload (Sec. III-C): VEC values per lane, 8 per 16-byte vector.
// The casts are v_cvt_f16_f32 (round to nearest even, binary16 subnormals
// kept) and v_cvt_f32_f16 (exact). The scaling is an fp32 multiply whose
// result is held opaque (mul_rounded): folded into the cast
// (v_fma_mixlo_f16), the product would be rounded once to binary16 instead
// of first to fp32.
// ---------------------------------------------------------------------------
typedef _Float16 h16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ bool half_nonfinite(uint16_t b) { return (b & 0x7c00u) == 0x7c00u; }

// p[i] = binary16(v[i] * s); returns true if any stored value is inf or NaN.
// fp32 product of a and b, rounded to fp32 and opaque to the optimizer (an
// empty asm statement holds it in a VGPR), so no later cast can absorb it.
__device__ __forceinline__ float mul_rounded(float a, float b) {
  float t = __fmul_rn(a, b);
  asm volatile("" : "+v"(t));
  return t;
}

template <int VEC>
__device__ __forceinline__ bool store_half_scaled(uint16_t* p, const float* v, float s) {
  bool bad = false;
  if constexpr (VEC % 8 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 8) {
      h16x8 h;
#pragma unroll
      for (int k = 0; k < 8; ++k) h[k] = static_cast<_Float16>(mul_rounded(v[i + k], s));
      const u32x4 w = __builtin_bit_cast(u32x4, h);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        bad |= half_nonfinite(static_cast<uint16_t>(w[k]));
        bad |= half_nonfinite(static_cast<uint16_t>(w[k] >> 16));
      }
      *reinterpret_cast<u32x4*>(p + i) = w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) {
      const uint16_t b = __builtin_bit_cast(uint16_t, static_cast<_Float16>(mul_rounded(v[i], s)));
      bad |= half_nonfinite(b);
      p[i] = b;
    }
  }
  return bad;
}

// v[i] = fp32(p[i]) * s.
template <int VEC>
__device__ __forceinline__ void load_half_scaled(const uint16_t* p, float* v, float s) {
  if constexpr (VEC % 8 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 8) {
      const h16x8 h = __builtin_bit_cast(h16x8, *reinterpret_cast<const u32x4*>(p + i));
#pragma unroll
      for (int k = 0; k < 8; ++k) v[i + k] = mul_rounded(static_cast<float>(h[k]), s);
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i)
      v[i] = mul_rounded(static_cast<float>(__builtin_bit_cast(_Float16, p[i])), s);
  }
}

template <int VEC>
__device__ __forceinline__ void store_half_zero(uint16_t* p) {
  if constexpr (VEC % 8 == 0) {
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < VEC; i += 8) __builtin_nontemporal_store(z, reinterpret_cast<u32x4*>(p + i));
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) p[i] = 0;
  }
}

// Streaming store (non-temporal): for rows nothing reads back soon.
template <int VEC>
__device__ __forceinline__ void store_vec_nt(float* p, const float* v) {
  if constexpr (VEC % 4 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 4) {
      f32x4 t = {v[i], v[i + 1], v[i + 2], v[i + 3]};
      __builtin_nontemporal_store(t, reinterpret_cast<f32x4*>(p + i));
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) __builtin_nontemporal_store(v[i], p + i);
  }
}

template <int VEC>
__device__ __forceinline__ void load_vec(const float* p, float* v) {
  if constexpr (VEC % 4 == 0) {
#pragma unroll
    for (int i = 0; i < VEC; i += 4) {
      float4 t = *reinterpret_cast<const float4*>(p + i);
      v[i] = t.x; v[i + 1] = t.y; v[i + 2] = t.z; v[i + 3] = t.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < VEC; ++i) v[i] = p[i];
  }
}

// Widen a word index of dtype KeyT to int64 / its raw unsigned bits.
template <typename KeyT>
__device__ __forceinline__ uint64_t key_bits(KeyT k) {
  if constexpr (sizeof(KeyT) == 4) return static_cast<uint32_t>(k);
  else return static_cast<uint64_t>(k);
}

// First index in [0, n) with a[i] >= x (n if none), over an ascending list.
template <typename KeyT>
__device__ __forceinline__ int64_t lower_bound_dev(const KeyT* a, int64_t n, KeyT x) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// lower_bound for a wave-uniform key x: the 64 lanes probe 64 evenly spaced
// positions per round (log64 n rounds of one gather instead of log2 n
// dependent loads). Every lane returns the same first index i with a[i] >= x.
template <typename KeyT>
__device__ __forceinline__ int64_t lower_bound_wave(const KeyT* a, int64_t n, KeyT x) {
  const int lane = lane_id();
  int64_t lo = 0, len = n;  // answer in [lo, lo + len]
  while (len > 0) {
    const int64_t step = (len + kWave) / (kWave + 1) > 0 ? (len + kWave) / (kWave + 1) : 1;
    const int64_t pos = lo + (lane + 1) * step - 1;  // probe a[pos] < x
    const bool lt = pos < lo + len && a[pos] < x;
    const int cnt = __popcll(ballot(lt));
    lo += int64_t(cnt) * step;
    const int64_t rem = len - int64_t(cnt) * step;
    len = cnt < kWave ? (step - 1 < rem ? step - 1 : rem) : rem;
  }
  return lo;
}

// ---------------------------------------------------------------------------
// The update of Sec. III-A step 7 on one fp32 value. lm_sparse_apply and the
// Seg-Sum entry points that apply their sums themselves call these same
// functions, so they round alike, bit for bit.
// ---------------------------------------------------------------------------
#ifndef LMZ_ADAM_HW_MATH
#define LMZ_ADAM_HW_MATH 0
#endif

struct OptParams {
  float lr, b1, b2, eps, wd, inv_c1, inv_c2, g_scale;
};

// Every multiply-add is an explicit fused one: left to the compiler, a sum
// of two products (b1 * m + (1 - b1) * g) may be fused either way round, and
// the choice can differ between the kernels that inline these functions.
__device__ __forceinline__ void sgd_value(float& p, float g, const OptParams& o) {
  p = __builtin_fmaf(-o.lr, g, p);
}

// Lazy Adam on a touched value: the moments, then the bias-corrected step
// with decoupled weight decay (inv_c1, inv_c2: 1 / (1 - beta^t)).
__device__ __forceinline__ void adam_value(float& p, float& m, float& v, float g,
                                           const OptParams& o) {
  m = __builtin_fmaf(o.b1, m, (1.f - o.b1) * g);
  v = __builtin_fmaf(o.b2, v, (1.f - o.b2) * g * g);
  const float mhat = m * o.inv_c1;
  const float vhat = v * o.inv_c2;
#if LMZ_ADAM_HW_MATH
  // v_sqrt_f32 and v_rcp_f32 (about 1 ulp each) instead of the correctly
  // rounded sequences.
  const float step = mhat * __builtin_amdgcn_rcpf(__builtin_amdgcn_sqrtf(vhat) + o.eps);
#else
  const float step = mhat / (sqrtf(vhat) + o.eps);
#endif
  p = __builtin_fmaf(-o.lr, __builtin_fmaf(o.wd, p, step), p);
}

// The step's parameters; the bias corrections are computed once on the host
// in double.
static inline OptParams make_opt_params(bool adam, float lr, float beta1, float beta2, float eps,
                                        float weight_decay, int64_t step, float g_scale) {
  OptParams o{};
  o.lr = lr;
  o.b1 = beta1;
  o.b2 = beta2;
  o.eps = eps;
  o.wd = weight_decay;
  o.g_scale = g_scale;
  if (adam) {
    o.inv_c1 = static_cast<float>(
        1.0 / (1.0 - __builtin_pow(static_cast<double>(beta1), static_cast<double>(step))));
    o.inv_c2 = static_cast<float>(
        1.0 / (1.0 - __builtin_pow(static_cast<double>(beta2), static_cast<double>(step))));
  }
  return o;
}

}  // namespace lmz

// Host-side launch helpers (defined in lmzipf_api.hip).
namespace lmz {
int launch_status(hipError_t e);
}
