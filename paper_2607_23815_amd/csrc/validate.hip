// Opt-in validation of the device-side metadata of a call (PKV_DEBUG_VALIDATE): block ids
// within the pool, lengths within the host maxima and the table, offsets that start at 0,
// never decrease and end at the host's total. The kernels themselves only bound what they
// index (a bad id reads a stand-in block, a length past the table stops at its end), so bad
// metadata gives finite but wrong results; with validation on, such a call is refused before
// anything else is launched.
//
// One thread per sequence checks its lengths and every table entry the call would read or
// write, and ORs what it finds into a device word (the first offending sequence goes into a
// second word); the host waits for the stream and reads both.
#include <limits.h>

#include <mutex>

#include "launch.h"

namespace pkv {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(64) void validate_reset_kernel(uint32_t* word) {
  if (threadIdx.x == 0) {
    word[0] = 0u;
    word[1] = (uint32_t)INT_MAX;
  }
}

__global__ __launch_bounds__(kThreads) void validate_kernel(MetaCheck c, uint32_t* word) {
  const int i = blockIdx.x * kThreads + threadIdx.x;
  if (i >= c.num_seqs) return;
  uint32_t bad = 0u;
  int64_t e0 = 0, e1 = 0;  // table entries [e0, e1) the call touches
  if (c.mode == kMetaDecode) {
    const int64_t len = c.lens[i];
    if (len < 1 || len > c.max_len) bad |= kMetaBadLength;
    e1 = (len + 15) / 16;
  } else {
    const int64_t a = c.cu[i], b = c.cu[i + 1];
    if (i == 0 && a != 0) bad |= kMetaBadOffsets;
    if (b < a) bad |= kMetaBadOffsets;
    if (i == c.num_seqs - 1 && c.total >= 0 && b != c.total) bad |= kMetaBadOffsets;
    const int64_t n = b - a;
    const int64_t p = c.lens[i];
    if (c.mode == kMetaGather) {
      // lens[i] tokens gathered into rows cu[i] ..
      if (p < 0 || p > c.max_len || n != p) bad |= kMetaBadLength;
      e1 = (p + 15) / 16;
    } else {
      // cached prefix p, n new tokens (append / prefill)
      if (p < 0 || n > c.max_len || p + n > c.max_total) bad |= kMetaBadLength;
      if (n > 0) {
        e0 = c.mode == kMetaAppend ? p / 16 : 0;
        e1 = (p + n + 15) / 16;
      }
    }
  }
  if (e1 > c.max_blocks) {  // entries past the table: the length overruns it
    bad |= kMetaBadLength;
    e1 = c.max_blocks;
  }
  if (e0 < 0) e0 = 0;
  const int32_t* row = c.tables + (size_t)i * c.max_blocks;
  for (int64_t e = e0; e < e1; ++e) {
    const int32_t t = row[e];
    if (t < 0 || t >= c.num_blocks) {
      bad |= kMetaBadBlockId;
      break;
    }
  }
  if (bad) {
    atomicOr(&word[0], bad);
    atomicMin(reinterpret_cast<int*>(&word[1]), i);
  }
}

// The result words: one pair per GPU, in the code object; the address is looked up once per
// device (the symbol's name in host code is a host-side stand-in).
static __device__ __align__(16) uint32_t validate_word[4];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_word_ptr[kMaxDevices] = {};

hipError_t word_ptr(uint32_t** out) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (g_word_ptr[dev] == nullptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(validate_word));
    if (err != hipSuccess) return err;
    g_word_ptr[dev] = p;
  }
  *out = static_cast<uint32_t*>(g_word_ptr[dev]);
  return hipSuccess;
}

}  // namespace

hipError_t validate_metadata(const MetaCheck* checks, int n_checks, hipStream_t stream,
                             uint32_t* bad, int32_t* first_seq, int32_t* which) {
  std::lock_guard<std::mutex> lock(g_mu);  // one word per GPU: checks run one at a time
  *bad = 0u;
  *first_seq = -1;
  *which = -1;
  uint32_t* w = nullptr;
  hipError_t err = word_ptr(&w);
  if (err != hipSuccess) return err;
  for (int k = 0; k < n_checks; ++k) {
    const MetaCheck& c = checks[k];
    if (c.num_seqs <= 0) continue;
    hipLaunchKernelGGL(validate_reset_kernel, dim3(1), dim3(64), 0, stream, w);
    hipLaunchKernelGGL(validate_kernel, dim3((unsigned)((c.num_seqs + kThreads - 1) / kThreads)),
                       dim3(kThreads), 0, stream, c, w);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    uint32_t host[2] = {0u, 0u};
    if ((err = hipMemcpyAsync(host, w, sizeof(host), hipMemcpyDeviceToHost, stream)) !=
        hipSuccess)
      return err;
    if ((err = hipStreamSynchronize(stream)) != hipSuccess) return err;
    if (host[0] != 0u) {
      *bad = host[0];
      *first_seq = (int32_t)host[1];
      *which = k;
      return hipSuccess;
    }
  }
  return hipSuccess;
}

}  // namespace pkv
