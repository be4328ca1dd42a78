// seedq_compress_noalloc: seedq_compress for callers that cannot allocate
// device memory (code under stream capture, serving loops, hosts that forbid
// hipMalloc). Its only scratch, the per-rung block lists of a multi-rung call,
// lives in a fixed device array of this translation unit instead of a
// caller-supplied workspace; the kernels are the same as seedq_compress's.
//
// The array is a module-scope device variable: each GPU the library runs on
// holds its own copy for the rest of the process. Host code never passes the
// array's name to a kernel (on the host that name is only a stand-in for the
// symbol); it passes the device address that hipGetSymbolAddress returns, looked
// up once per device, with that device current, on the first call there.
#include <mutex>

#include "seedq_internal.h"

namespace seedq {
namespace {

static __device__ __align__(256) unsigned char scratch[SEEDQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex scratch_mutex;
void* scratch_ptr[kMaxDevices];   // device address of `scratch` per device, once looked up

// Device address of this device's scratch array, SEEDQ_OK or SEEDQ_EHIP.
int current_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SEEDQ_EHIP;
  std::lock_guard<std::mutex> lock(scratch_mutex);
  if (!scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SEEDQ_EHIP;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return SEEDQ_OK;
}

}  // namespace
}  // namespace seedq

using namespace seedq;

extern "C" int seedq_compress_noalloc(const float* d_W, int64_t nrows, int64_t ncols, int32_t C,
                                      const uint8_t* d_rung_of_block, int32_t nrungs,
                                      const seedq_bases* bases, uint32_t* d_seed, uint8_t* d_exp,
                                      int8_t* d_q, float* d_err, void* hip_stream) {
  const int rc = check_compress_args(d_W, nrows, ncols, C, d_rung_of_block, nrungs, bases, d_seed,
                                     d_exp, d_q);
  if (rc != SEEDQ_OK) return rc;
  void* ws = nullptr;
  if (nrungs > 1) {
    // every word of the lists that a search reads is written by the compaction
    // of the same call, so nothing in the array has to start at zero
    if (compaction_workspace_bytes(nrows * (ncols / kC), nrungs) > size_t(SEEDQ_NOALLOC_SCRATCH_BYTES))
      return SEEDQ_ESCRATCH;
    const int sr = current_scratch(&ws);
    if (sr != SEEDQ_OK) return sr;
  }
  return run_compress(d_W, nrows, ncols, d_rung_of_block, nrungs, bases, d_seed, d_exp, d_q, d_err,
                      ws, static_cast<hipStream_t>(hip_stream));
}
