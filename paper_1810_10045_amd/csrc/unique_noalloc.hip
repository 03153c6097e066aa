// lm_unique_noalloc: lm_unique with its workspace in a device array of the
// library itself, for callers that cannot allocate device memory (code under
// graph capture, tight serving loops, harnesses that forbid hipMalloc).
//
// The array is a file-scope device variable, so every GPU the library runs
// on holds its own copy from module load until the process ends. Host code
// never uses the array's name as a device address: on the first call on a
// device, hipGetSymbolAddress gives that device's address, which is kept per
// device and is what the kernels receive. Unique's first kernel clears what
// the call needs of its workspace, so the array needs no initial contents;
// calls that overlap on one GPU share it and race.
#include <atomic>
#include <mutex>

#include "common.hpp"

namespace lmz {
size_t unique_workspace_bytes(int64_t K, int idtype, int64_t V);
int unique_run(const void* ids, int idtype, int64_t K, int64_t V, void* uniq, int32_t* counts,
               int32_t* offsets, int32_t* inverse, int32_t* perm, int64_t* num_unique,
               int32_t* dev_err, void* ws, size_t ws_bytes, hipStream_t st);
}  // namespace lmz

// 12 MiB: the largest workspace lm_unique needs for LM_UNIQUE_NOALLOC_MAX_K
// ids is 10.7 MiB (int64 ids with V = 32,768, counted per id; 61-bit int64
// keys need 10.4 MiB); the call checks its own need against this size all
// the same.
constexpr size_t kScratchBytes = size_t(12) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// This device's address of `scratch`, looked up once per device (with that
// device current), or nullptr with *status set.
void* scratch_on_current_device(int* status) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    *status = LM_E_HIP;
    return nullptr;
  }
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    void* addr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !addr || (reinterpret_cast<uintptr_t>(addr) & 255)) {
      (void)hipGetLastError();
      *status = LM_E_HIP;
      return nullptr;
    }
    p = addr;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  return p;
}
}  // namespace

extern "C" int lm_unique_noalloc(const void* ids, int32_t idtype, int64_t K, int64_t V,
                                 void* uniq, int32_t* counts, int32_t* offsets,
                                 int32_t* inverse, int32_t* perm, int64_t* num_unique,
                                 int32_t* dev_err, void* stream) {
  if (idtype != LM_I32 && idtype != LM_I64) return LM_E_UNSUPPORTED;
  if (K < 0 || V < 1) return LM_E_INVAL;
  if (K > LM_UNIQUE_NOALLOC_MAX_K) return LM_E_UNSUPPORTED;
  if (!offsets || !num_unique) return LM_E_INVAL;
  if (K > 0 && (!ids || !uniq || !counts || !inverse || !perm || !dev_err)) return LM_E_INVAL;
  if (lmz::unique_workspace_bytes(K, idtype, V) > kScratchBytes) return LM_E_UNSUPPORTED;
  int status = LM_OK;
  void* ws = scratch_on_current_device(&status);
  if (!ws) return status;
  return lmz::unique_run(ids, idtype, K, V, uniq, counts, offsets, inverse, perm, num_unique,
                         dev_err, ws, kScratchBytes, static_cast<hipStream_t>(stream));
}
