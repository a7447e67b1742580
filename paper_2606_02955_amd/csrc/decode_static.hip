// decode_static.hip -- fdllm_decode_step for callers that cannot allocate.
//
// Some callers cannot call hipMalloc (code under HIP graph capture, tight
// serving loops, harnesses that forbid allocation), so they cannot provide
// the decode step's workspace.  This entry point runs the very same step
// (same plans, same kernels, same bits) with its scratch in a file-scope
// device array instead: one FDLLM_STATIC_SCRATCH_BYTES array per GPU, held
// until the process ends.
//
// In host code the array's name only stands for the variable; the device
// address differs per GPU.  The first call on a device, with that device
// current, looks the address up with hipGetSymbolAddress and keeps it; every
// later use (the kernels' workspace argument) goes through that pointer.
// Calls that overlap on one GPU share its array and race.
#include <hip/hip_runtime.h>

#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "fdllm.h"
#include "pass_common.h"

namespace {

static __device__ __align__(256) unsigned char scratch[FDLLM_STATIC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];   // device address of `scratch`, per device id

// Device address of the current GPU's scratch; nullptr with *st set on failure.
void* scratch_on_current_device(fdllm_status* st) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    *st = FDLLM_ERR_HIP;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      *st = FDLLM_ERR_HIP;
      return nullptr;
    }
    g_ptr[dev] = p;
  }
  return g_ptr[dev];
}

}  // namespace

extern "C" fdllm_status fdllm_decode_step_static(
    const void* logits, fdllm_dtype dtype, int B, int L, int V, uint8_t* mask,
    const int32_t* block_start, const int32_t* block_end, int32_t* x, fdllm_selector sel,
    float param, const float* eta, float eta_uniform, int32_t* tokens, float* conf, float* eps,
    float* lse, uint8_t* commit, int32_t* n_commit, fdllm_stream stream) {
  // the workspace fdllm_decode_step would use for the same sizes (its plan
  // with the full workspace); refuse what the static array cannot hold
  size_t need = 0;
  fdllm_status st = fdllm_workspace_size(B, L, V, dtype, &need);
  if (st != FDLLM_OK) return st;
  // argument errors first, as fdllm_decode_step reports them, before any HIP call
  if (sel != FDLLM_SEL_THRESHOLD && sel != FDLLM_SEL_FACTOR && sel != FDLLM_SEL_PROFILE &&
      sel != FDLLM_SEL_ROBUST)
    return FDLLM_ERR_INVALID_ARG;
  if (!(eta_uniform == eta_uniform)) return FDLLM_ERR_INVALID_ARG;
  if (B > 0 && (!logits || !mask || !block_start || !block_end || !x)) return FDLLM_ERR_INVALID_ARG;
  if (need > (size_t)FDLLM_STATIC_SCRATCH_BYTES) return FDLLM_ERR_SCRATCH;
  void* ws = nullptr;
  if (need > 0 && B > 0) {
    ws = scratch_on_current_device(&st);
    if (!ws) return st;
  }
  // a large batch's last sequences run after its one-kernel part on `stream`
  // (no side stream, no events), with the same bits
  return fdllm::decode_step(logits, dtype, B, L, V, mask, block_start, block_end, x, sel, param, eta,
                            eta_uniform, tokens, conf, eps, lse, commit, n_commit, ws, need, stream,
                            false);
}
