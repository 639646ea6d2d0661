// rollout_sample_noalloc: the token draw of rollout_sample for callers that cannot allocate device memory
// (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).  It runs the same
// sampler kernels; their scratch (the exp values of the rows and the per-chunk maxima, masses and
// histograms) lives in a file-scope device array of fixed size instead of a context's arena.
//
// Host code never passes the array's name to a kernel or a copy: the name is a host-side stand-in.  The
// array's device address is looked up once per device (hipGetSymbolAddress, with that device current) and
// kept; every GPU holds its own copy of the array, at its own address, until the process ends.
//
// Every call on a device shares that device's array: calls that overlap on one device (two streams, two
// threads) race on it and must be serialised by the caller.  The sampler writes every scratch word it reads
// within one call, so nothing has to be cleared between calls.
#include <mutex>
#include <string>

#include "internal.h"

using namespace rollout;

namespace {

constexpr size_t kScratchBytes = ROLLOUT_SAMPLE_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device, once looked up

rollout_status fail(rollout_status st, const std::string& msg) {
  set_last_error(msg);
  return st;
}

}  // namespace

extern "C" rollout_status rollout_sample_noalloc(const float* d_logits, int32_t n_seqs, int32_t vocab,
                                                 float temperature, float top_p, const float* d_uniforms,
                                                 int32_t* d_tokens_out, void* hip_stream) {
  // arguments first: nothing below touches the device until they are all valid
  if (!d_logits || !d_uniforms || !d_tokens_out) return fail(ROLLOUT_EINVAL, "NULL buffer");
  if (n_seqs < 1 || vocab < 2) return fail(ROLLOUT_EINVAL, "n_seqs must be >= 1 and vocab >= 2");
  if (!(temperature >= 0.f) || !std::isfinite(temperature)) return fail(ROLLOUT_EINVAL, "temperature must be >= 0");
  if (!(top_p > 0.f && top_p <= 1.f)) return fail(ROLLOUT_EINVAL, "top_p must be in (0, 1]");
  const int rows = sample_rows_fitting(kScratchBytes, vocab);
  if (rows < 1)
    return fail(ROLLOUT_ENOMEM, "one row of " + std::to_string(vocab) + " logits needs " +
                                    std::to_string(sample_scratch_bytes(1, vocab)) + " bytes of sampler scratch; the "
                                    "fixed scratch holds " + std::to_string(kScratchBytes));
  hipStream_t stream = (hipStream_t)hip_stream;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ROLLOUT_EDEVICE, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(ROLLOUT_EDEVICE, "device index beyond the supported count");
  if (stream) {
    int sdev = -1;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return fail(ROLLOUT_EDEVICE, std::string("hipStreamGetDevice: ") + hipGetErrorString(e));
    if (sdev != dev) return fail(ROLLOUT_EINVAL, "the stream belongs to another device than the current one");
  }
  void* base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
      // the current device is `dev`: its own copy of the array
      e = hipGetSymbolAddress(&g_scratch[dev], HIP_SYMBOL(scratch));
      if (e != hipSuccess) {
        g_scratch[dev] = nullptr;
        return fail(ROLLOUT_EDEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
      }
    }
    base = g_scratch[dev];
  }
  // rows in batches that fit the fixed scratch, in order
  for (int r0 = 0; r0 < n_seqs; r0 += rows) {
    const int n = std::min(rows, n_seqs - r0);
    e = launch_sample(stream, d_logits + (size_t)r0 * vocab, n, vocab, temperature, top_p, d_uniforms + r0, 1, nullptr,
                      d_tokens_out + r0, 1, base);
    if (e != hipSuccess) return fail(ROLLOUT_EDEVICE, std::string("sample: ") + hipGetErrorString(e));
  }
  return ROLLOUT_OK;
}
