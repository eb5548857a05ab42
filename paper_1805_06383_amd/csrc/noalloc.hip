// Exclusive scan without any allocation (fstc_exclusive_scan_u64_noalloc).
//
// The single-pass scan (scan.hip) needs scratch memory beside its input and
// output: one tile counter, one error word and the look-back state of every
// tile (its aggregate, inclusive prefix and state word).  fstc_exclusive_scan_u64
// allocates them per call; this entry point takes them from `scratch`, a
// file-scope device array each GPU holds once, so that callers that cannot
// allocate device memory can still run the scan.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is looked up with hipGetSymbolAddress once per device (with
// that device current) at the first call there, kept per device, and only
// that address is handed to kernels and fills.  Calls on one GPU share its
// array; calls that overlap on one GPU race.
#include <array>
#include <cstring>
#include <mutex>

#include "common.hpp"

namespace fstc {
namespace {

// Largest input of the no-allocation scan, and the scratch it needs: the
// counter and error words, then the look-back state of ceil(n / 2048) tiles
// (136 bytes a tile, status words rounded up to 256-byte lines, plus 256
// bytes of slack: scan_lb_state_bytes).
constexpr u64 kNoAllocMaxN = 1ull << 28;
constexpr size_t kScratchWords = 256;  // counter, error word; the state starts 256 bytes in
constexpr size_t kScratchStateBytes = ((kNoAllocMaxN + 2047) / 2048) * 136 + 256 + 256;
constexpr size_t kScratchBytes = kScratchWords + kScratchStateBytes;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

struct DeviceScratch {
  std::once_flag once;
  void *ptr = nullptr;   // device address of this device's `scratch`
  hipError_t rc = hipSuccess;
};
std::array<DeviceScratch, kMaxDevices> g_scratch;

__global__ void k_zero_words(u32 *p, u64 n) {
  for (u64 i = (u64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (u64)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// This device's scratch address; at the first call on the device, the
// symbol lookup and one clearing of the whole array on `s` (the scan's
// state words must not hold the current epoch by chance).
void *device_scratch(hipStream_t s) {
  int dev = 0;
  FSTC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) throw Error(FSTC_ERR_INVALID_ARG, "device index too large");
  DeviceScratch &d = g_scratch[dev];
  std::call_once(d.once, [&] {
    void *p = nullptr;
    d.rc = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (d.rc != hipSuccess) return;
    const u64 words = kScratchBytes / 4;
    hipLaunchKernelGGL(k_zero_words, dim3((unsigned)std::min<u64>(ceil_div(words, 256), 4096)),
                       dim3(256), 0, s, static_cast<u32 *>(p), words);
    d.rc = hipGetLastError();
    if (d.rc == hipSuccess) d.rc = hipStreamSynchronize(s);
    if (d.rc == hipSuccess) d.ptr = p;
  });
  if (d.rc != hipSuccess)
    throw Error(FSTC_ERR_HIP, std::string("scratch setup: ") + hipGetErrorString(d.rc));
  return d.ptr;
}

}  // namespace

u64 noalloc_scan_max_n() { return kNoAllocMaxN; }

// Exclusive scan of n u64 values into out[0..n] with the device's scratch
// array; no allocation.  Synchronises `s` to read the scan's error word.
void noalloc_scan(const u64 *in, u64 *out, u64 n, hipStream_t s) {
  if (n > kNoAllocMaxN) throw Error(FSTC_ERR_RANGE, "n exceeds the scratch capacity (2^28)");
  static_assert(kScratchStateBytes >= 256, "state region");
  char *base = static_cast<char *>(device_scratch(s));
  u32 *words = reinterpret_cast<u32 *>(base);  // [0] tile counter, [1] error word
  void *state = base + kScratchWords;
  if (scan_lb_state_bytes(n) > kScratchStateBytes)
    throw Error(FSTC_ERR_INTERNAL, "scan state does not fit the scratch array");
  // the counter is left 0 by every scan; the error word is cleared here
  hipLaunchKernelGGL(k_zero_words, dim3(1), dim3(64), 0, s, words + 1, (u64)1);
  const ScanJob job{in, true, out};
  exclusive_scan_lb(&job, 1, n, state, words, words + 1, s);
  u32 err = 0;
  FSTC_HIP(hipGetLastError());
  FSTC_HIP(hipMemcpyAsync(&err, words + 1, 4, hipMemcpyDeviceToHost, s));
  FSTC_HIP(hipStreamSynchronize(s));
  if (err) throw Error(FSTC_ERR_INTERNAL, "a single-pass scan timed out waiting for a predecessor tile");
}

}  // namespace fstc
