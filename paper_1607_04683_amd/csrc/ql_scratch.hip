// ql_scratch.hip -- the stream step for callers that cannot allocate: the
// model forward of one chunk of a stream (Section 4) on a scratch buffer held
// by the library in a static device array, instead of a caller workspace.
//
// The array's name is a host-side stand-in in host code: the first call on a
// device resolves its device address there with hipGetSymbolAddress (that
// device current) and keeps it; only that address is ever handed to kernels.
#include "../../include/qlstm.h"

#include <hip/hip_runtime.h>

#include <mutex>

#include "ql_exchange.h"

namespace {

constexpr size_t kScratchBytes = QL_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

void *g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each device, once resolved
std::mutex g_scratch_mu;

// Device address of this device's scratch array (resolved on first use).
ql_status scratch_for_current_device(void **out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QL_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return QL_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return QL_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return QL_OK;
}

// The forward's timeout flag (in the scratch header) to the caller's word.
__global__ void k_report_timeout(const int *flag, int32_t *out) {
  if (threadIdx.x == 0) *out = *flag ? 1 : 0;
}

}  // namespace

extern "C" ql_status ql_acoustic_model_forward_stream_noalloc(
    const ql_model *M, const float *feats, int64_t T, int64_t B, const ql_lstm_state *state_in,
    const ql_lstm_state *state_out, float *post, int32_t *timed_out, void *stream) {
  if (!M || !M->layers || M->nlayers <= 0) return QL_EINVAL;
  if (T < 0 || B < 0) return QL_ESHAPE;
  if (ql_acoustic_model_workspace(M, T, B) > kScratchBytes) return QL_ESCRATCH;
  void *ws = nullptr;
  ql_status st = scratch_for_current_device(&ws);
  if (st != QL_OK) return st;
  st = ql_acoustic_model_forward_stream(M, feats, T, B, state_in, state_out, post, nullptr, ws,
                                        kScratchBytes, stream);
  if (st != QL_OK || !timed_out) return st;
  hipLaunchKernelGGL(k_report_timeout, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream),
                     static_cast<const int *>(ws) + ql::kHdrFlag, timed_out);
  return hipGetLastError() == hipSuccess ? QL_OK : QL_EHIP;
}
