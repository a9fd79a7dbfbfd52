// Status strings, the thread-local error message and launch checking for the C ABI.
#include "fl_common.h"

#include <atomic>
#include <cstdlib>
#include <cstring>
#include <vector>

namespace fl {

// index-list checks: off unless FL_CHECK_INDICES is set to a non-zero value, or fl_set_index_checks(1)
static std::atomic<int> g_checks{-1};

bool index_checks_on() {
  int v = g_checks.load(std::memory_order_relaxed);
  if (v < 0) {
    const char* e = std::getenv("FL_CHECK_INDICES");
    v = (e && *e && std::strcmp(e, "0") != 0) ? 1 : 0;
    int expect = -1;
    g_checks.compare_exchange_strong(expect, v);
    v = g_checks.load(std::memory_order_relaxed);
  }
  return v > 0;
}

int check_index_lists(const char* fn, const char* name, const int32_t* list, int64_t n_lists, int len, int lo,
                      int hi, hipStream_t st) {
  if (!index_checks_on() || list == nullptr || n_lists <= 0 || len <= 0) return FL_OK;
  hipError_t e = hipStreamSynchronize(st);
  FL_REQUIRE(e == hipSuccess, FL_E_HIP, "%s: index check: stream synchronization failed: %s", fn,
             hipGetErrorString(e));
  std::vector<int32_t> h((size_t)n_lists * (size_t)len);
  e = hipMemcpy(h.data(), list, h.size() * sizeof(int32_t), hipMemcpyDeviceToHost);
  FL_REQUIRE(e == hipSuccess, FL_E_HIP, "%s: index check: copy of %s failed: %s", fn, name, hipGetErrorString(e));
  for (int64_t r = 0; r < n_lists; ++r) {
    const int32_t* p = h.data() + r * len;
    for (int i = 0; i < len; ++i) {
      FL_REQUIRE(p[i] >= lo && p[i] < hi, FL_E_RANGE, "%s: %s[%lld][%d] = %d outside [%d, %d)", fn, name,
                 (long long)r, i, p[i], lo, hi);
      FL_REQUIRE(i == 0 || p[i] > p[i - 1], FL_E_RANGE, "%s: %s[%lld] is not strictly ascending at %d (%d after %d)",
                 fn, name, (long long)r, i, p[i], p[i - 1]);
    }
  }
  return FL_OK;
}

// Largest bf16 magnitude pattern (sign cleared) seen by the range check below; patterns order like the
// magnitudes they encode.
static __device__ unsigned int g_bf16_max_mag;

__global__ __launch_bounds__(256) void bf16_max_mag_kernel(const uint16_t* __restrict__ x, int64_t n) {
  unsigned int m = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    m = max(m, (unsigned int)(x[i] & 0x7FFFu));
  for (int off = 32; off > 0; off >>= 1) m = max(m, (unsigned int)__shfl_xor((int)m, off, 64));
  if ((threadIdx.x & 63) == 0) atomicMax(&g_bf16_max_mag, m);
}

int check_f16_range(const char* fn, const char* name, const uint16_t* x, int64_t n, hipStream_t st) {
  if (!index_checks_on() || x == nullptr || n <= 0) return FL_OK;
  // (synchronous like the list checks: the stream is drained, the device word reset, the reduction run
  // on the stream, and the word read back once the stream has finished)
  hipError_t e = hipStreamSynchronize(st);
  const unsigned int zero = 0;
  if (e == hipSuccess) e = hipMemcpyToSymbol(HIP_SYMBOL(g_bf16_max_mag), &zero, sizeof(zero), 0, hipMemcpyHostToDevice);
  FL_REQUIRE(e == hipSuccess, FL_E_HIP, "%s: range check: reset failed: %s", fn, hipGetErrorString(e));
  const int64_t blocks64 = (n + 255) / 256;
  const unsigned int blocks = (unsigned int)(blocks64 < 4096 ? blocks64 : 4096);
  bf16_max_mag_kernel<<<blocks, 256, 0, st>>>(x, n);
  int rc = check_launch("bf16_max_mag_kernel");
  if (rc != FL_OK) return rc;
  unsigned int m = 0;
  e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipMemcpyFromSymbol(&m, HIP_SYMBOL(g_bf16_max_mag), sizeof(m), 0, hipMemcpyDeviceToHost);
  FL_REQUIRE(e == hipSuccess, FL_E_HIP, "%s: range check: read-back failed: %s", fn, hipGetErrorString(e));
  // 0x4780 is bf16 65536: every smaller finite bf16 magnitude is at most 65280 and fits fp16 (<= 65504)
  FL_REQUIRE(m < 0x4780u, FL_E_RANGE, "%s: %s holds a value of magnitude %s (bf16 bits 0x%04x): the fp16 "
             "product path needs |v| <= 65504", fn, name, m >= 0x7F80u ? "inf/NaN" : "> 65504", m);
  return FL_OK;
}

static thread_local char g_last_error[512] = "";

int set_error(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return set_error(FL_E_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return FL_OK;
}

}  // namespace fl

extern "C" const char* fl_status_str(int status) {
  switch (status) {
    case FL_OK: return "FL_OK";
    case FL_E_NULL: return "FL_E_NULL: a required pointer is NULL";
    case FL_E_SHAPE: return "FL_E_SHAPE: inconsistent or unsupported sizes";
    case FL_E_RANGE: return "FL_E_RANGE: a count is out of range";
    case FL_E_UNSUPPORTED: return "FL_E_UNSUPPORTED: unsupported bit width, axis, mode or flag";
    case FL_E_WORKSPACE: return "FL_E_WORKSPACE: workspace missing or too small";
    case FL_E_HIP: return "FL_E_HIP: the HIP runtime rejected a launch";
    case FL_E_INTERNAL: return "FL_E_INTERNAL: internal error";
    default: return "unknown status";
  }
}

extern "C" const char* fl_last_error(void) { return fl::g_last_error; }

extern "C" int fl_abi_version(void) { return FL_ABI_VERSION; }

extern "C" void fl_set_index_checks(int on) { fl::g_checks.store(on ? 1 : 0, std::memory_order_relaxed); }
