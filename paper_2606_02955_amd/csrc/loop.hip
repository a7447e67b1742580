// loop.hip -- the decoding loop around one step, kept on the device
// (arXiv 2606.02955, Alg. 1 outer loops: for every block, repeat model call,
// step, until the block has no masked position).
//
//   * k_synth: the synthetic stand-in for the model call.  It writes the
//     logits of every sequence's active block from a counter-based generator
//     (Philox4x32-10, Salmon et al., SC 2011), so a step needs no host work.
//     The recipe is stated in include/fdllm.h.  Integer arithmetic and
//     individually rounded float32 operations only, so the bits are the ones
//     any IEEE implementation of the recipe produces.
//   * k_advance: a sequence whose active block has no masked position left
//     moves on to its next block; a finished sequence gets an empty window.
//   * a generation object captures `chunk` steps (producer, fdllm_decode_step,
//     advance, step counter) into one HIP graph and replays it; the host reads
//     the number of active sequences once per chunk, one chunk behind the
//     device, and stops when it reaches zero.
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "fdllm.h"

namespace fdllm_loop {

constexpr int kWave = 64;
constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;   // Philox4x32 multipliers
constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;   // Philox4x32 key increments
constexpr uint32_t kTokC0 = 0xFFFFFFFFu, kTokC3 = 0xFFFFFFFFu, kHeightC0 = 0xFFFFFFFEu;

__device__ __forceinline__ void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += kW0;
      k1 += kW1;
    }
    const uint32_t hi0 = __umulhi(kM0, c[0]), lo0 = kM0 * c[0];
    const uint32_t hi1 = __umulhi(kM1, c[2]), lo1 = kM1 * c[2];
    const uint32_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__device__ __forceinline__ float background(uint32_t w) {
  const int s = (int)(w & 0xFFu) + (int)((w >> 8) & 0xFFu) + (int)((w >> 16) & 0xFFu) + (int)(w >> 24);
  return __fmul_rn((float)(s - 510), 0.0078125f);   // exact: |s - 510| <= 510
}

// Logits rows of every sequence's active block at step t.  One row per
// blockIdx.x (b = x / blk, slot = x % blk); blockIdx.y covers the vocabulary
// in groups of 4 entries per thread (one Philox call each).
__global__ void __launch_bounds__(256)
k_synth(uint16_t* __restrict__ logits, int B, int L, int V, int blk,
        const int32_t* __restrict__ bstart, const int32_t* __restrict__ bend, uint32_t k0,
        uint32_t k1, const int32_t* __restrict__ step_dev, int step_host,
        const int32_t* __restrict__ active) {
  __shared__ int s_tok;
  __shared__ float s_h;
  if (active && *active == 0) return;
  const int b = blockIdx.x / blk;
  const int i = bstart[b] + blockIdx.x % blk;
  const int e = bend[b];
  if (bstart[b] < 0 || e > L || i >= e) return;
  const uint32_t t = (uint32_t)(step_dev ? *step_dev : step_host);
  if (threadIdx.x == 0) {
    uint32_t c[4] = {kTokC0, (uint32_t)i, (uint32_t)b, kTokC3};
    philox4x32_10(c, k0, k1);
    s_tok = (int)(c[0] % (uint32_t)V);
    uint32_t y[4] = {kHeightC0, (uint32_t)i, (uint32_t)b, t};
    philox4x32_10(y, k0, k1);
    const float u1 = __fmul_rn((float)(y[0] >> 8), 5.9604644775390625e-08f);   // 2^-24
    const float u2 = __fmul_rn((float)(y[1] >> 8), 5.9604644775390625e-08f);
    const float six_u2 = __fmul_rn(6.0f, u2);
    s_h = u1 < 0.6f ? __fadd_rn(8.0f, six_u2) : six_u2;
  }
  __syncthreads();
  const int q = blockIdx.y * blockDim.x + threadIdx.x;   // vocabulary group
  const int v0 = 4 * q;
  if (v0 >= V) return;
  uint32_t c[4] = {(uint32_t)q, (uint32_t)i, (uint32_t)b, t};
  philox4x32_10(c, k0, k1);
  uint16_t out[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float x = background(c[j]);
    if (v0 + j == s_tok) x = __fadd_rn(x, s_h);
    out[j] = bf16_rne(x);
  }
  uint16_t* row = logits + ((size_t)b * L + i) * (size_t)V;
  if (v0 + 4 <= V && ((((uintptr_t)(row + v0)) & 7u) == 0)) {
    const uint2 packed = make_uint2((uint32_t)out[0] | ((uint32_t)out[1] << 16),
                                    (uint32_t)out[2] | ((uint32_t)out[3] << 16));
    *reinterpret_cast<uint2*>(row + v0) = packed;
  } else {
    for (int j = 0; j < 4 && v0 + j < V; ++j) row[v0 + j] = out[j];
  }
}

struct GenState {
  int32_t t;             // steps taken (steps in which some sequence had an active block)
  int32_t active;        // sequences with an active block at the start of the current step
  int32_t active_next;   // counted by k_advance for the next step
  int32_t pad;
};

// One wavefront per sequence: advance to the first block, from the current
// one on, that still has a masked position.  Optionally records this step's
// n_commit and counts the sequences left active.
__global__ void __launch_bounds__(256)
k_advance(const uint8_t* __restrict__ mask, int32_t* __restrict__ bstart,
          int32_t* __restrict__ bend, int B, int G, int blk, GenState* st,
          const int32_t* __restrict__ n_commit, int32_t* __restrict__ hist, int hist_steps,
          int32_t* __restrict__ n_active) {
  const int lane = threadIdx.x % kWave;
  const int b = blockIdx.x * 4 + threadIdx.x / kWave;
  if (b >= B) return;
  const bool worked = st == nullptr || st->active > 0;
  int s = bstart[b];
  if (s < 0 || s > G) s = G;
  while (s < G) {
    const int e = s + blk < G ? s + blk : G;
    bool any = false;
    for (int p = s + lane; p < e; p += kWave) any |= mask[(size_t)b * G + p] != 0;
    if (__ballot(any) != 0ull) break;
    s += blk;
  }
  if (lane != 0) return;
  if (st && hist && worked && st->t < hist_steps) hist[(size_t)st->t * B + b] = n_commit[b];
  if (s < G) {
    bstart[b] = s;
    bend[b] = s + blk < G ? s + blk : G;
    if (st) atomicAdd(&st->active_next, 1);
    if (n_active) atomicAdd(n_active, 1);
  } else {
    bstart[b] = G;
    bend[b] = G;
  }
}

__global__ void k_step_end(GenState* st) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  if (st->active > 0) st->t += 1;
  st->active = st->active_next;
  st->active_next = 0;
}

__global__ void k_zero_i32(int32_t* p, int n) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < n) p[k] = 0;
}

// Every position of the span masked, x = -1, first block active, counters reset.
__global__ void __launch_bounds__(256)
k_init(uint8_t* __restrict__ mask, int32_t* __restrict__ x, int32_t* __restrict__ bstart,
       int32_t* __restrict__ bend, int B, int G, int blk, GenState* st) {
  const long long n = (long long)B * G;
  for (long long k = (long long)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (long long)gridDim.x * blockDim.x) {
    mask[k] = 1;
    x[k] = -1;
  }
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) {
    bstart[b] = 0;
    bend[b] = blk < G ? blk : G;
  }
  if (b == 0) {
    st->t = 0;
    st->active = G > 0 ? B : 0;
    st->active_next = 0;
    st->pad = 0;
  }
}

size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

bool desc_ok(const fdllm_generation_desc* d) {
  return d && d->B > 0 && d->G > 0 && d->blk > 0 && d->blk <= FDLLM_MAX_BLOCK && d->V > 0 &&
         d->max_steps > 0 && d->chunk > 0 && d->logits && d->mask && d->x && d->block_start &&
         d->block_end && d->sel >= FDLLM_SEL_THRESHOLD && d->sel <= FDLLM_SEL_ROBUST &&
         d->eta_uniform == d->eta_uniform && (long long)d->B * d->blk <= 0x7fffffffLL;
}

}  // namespace fdllm_loop

using namespace fdllm_loop;

struct fdllm_generation_s {
  fdllm_generation_desc d;
  GenState* st;
  int32_t* n_commit;
  void* step_ws;
  size_t step_ws_bytes;
  hipStream_t cap;
  hipGraph_t graph;
  hipGraphExec_t exec;
  hipEvent_t ev[2];
  int32_t* host_active;    // pinned host copy of st->active
};

static fdllm_status enqueue_steps(fdllm_generation g, int steps, hipStream_t s) {
  const fdllm_generation_desc& d = g->d;
  const uint32_t k0 = (uint32_t)(d.seed & 0xFFFFFFFFull), k1 = (uint32_t)(d.seed >> 32);
  const int nq = (d.V + 3) / 4;
  const dim3 sgrid((unsigned)(d.B * d.blk), (unsigned)((nq + 255) / 256));
  for (int k = 0; k < steps; ++k) {
    hipLaunchKernelGGL(k_synth, sgrid, dim3(256), 0, s, (uint16_t*)d.logits, d.B, d.G, d.V, d.blk,
                       d.block_start, d.block_end, k0, k1, &g->st->t, 0, &g->st->active);
    if (hipGetLastError() != hipSuccess) return FDLLM_ERR_HIP;
    const fdllm_status st = fdllm_decode_step(
        d.logits, FDLLM_BF16, d.B, d.G, d.V, d.mask, d.block_start, d.block_end, d.x, d.sel,
        d.param, d.eta, d.eta_uniform, nullptr, nullptr, nullptr, nullptr, nullptr, g->n_commit,
        g->step_ws, g->step_ws_bytes, (fdllm_stream)s);
    if (st != FDLLM_OK) return st;
    hipLaunchKernelGGL(k_advance, dim3((unsigned)((d.B + 3) / 4)), dim3(256), 0, s, d.mask,
                       d.block_start, d.block_end, d.B, d.G, d.blk, g->st, g->n_commit,
                       d.n_commit_hist, d.max_steps, (int32_t*)nullptr);
    hipLaunchKernelGGL(k_step_end, dim3(1), dim3(64), 0, s, g->st);
    if (hipGetLastError() != hipSuccess) return FDLLM_ERR_HIP;
  }
  return FDLLM_OK;
}

extern "C" {

fdllm_status fdllm_synth_logits(void* logits, int B, int L, int V, int blk,
                                const int32_t* block_start, const int32_t* block_end,
                                uint64_t seed, int step, fdllm_stream stream) {
  if (B < 0 || L < 1 || V < 1 || blk < 1 || blk > FDLLM_MAX_BLOCK || step < 0)
    return FDLLM_ERR_INVALID_ARG;
  if (B == 0) return FDLLM_OK;
  if (!logits || !block_start || !block_end) return FDLLM_ERR_INVALID_ARG;
  if ((long long)B * blk > 0x7fffffffLL) return FDLLM_ERR_SIZE;
  const int nq = (V + 3) / 4;
  hipLaunchKernelGGL(k_synth, dim3((unsigned)(B * blk), (unsigned)((nq + 255) / 256)), dim3(256), 0,
                     (hipStream_t)stream, (uint16_t*)logits, B, L, V, blk, block_start, block_end,
                     (uint32_t)(seed & 0xFFFFFFFFull), (uint32_t)(seed >> 32),
                     (const int32_t*)nullptr, step, (const int32_t*)nullptr);
  return hipGetLastError() == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

fdllm_status fdllm_advance_blocks(const uint8_t* mask, int32_t* block_start, int32_t* block_end,
                                  int B, int G, int blk, int32_t* n_active, fdllm_stream stream) {
  if (B < 0 || G < 1 || blk < 1) return FDLLM_ERR_INVALID_ARG;
  if (B == 0) return FDLLM_OK;
  if (!mask || !block_start || !block_end) return FDLLM_ERR_INVALID_ARG;
  hipStream_t s = (hipStream_t)stream;
  if (n_active) hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, s, n_active, 1);
  hipLaunchKernelGGL(k_advance, dim3((unsigned)((B + 3) / 4)), dim3(256), 0, s, mask, block_start,
                     block_end, B, G, blk, (GenState*)nullptr, (const int32_t*)nullptr,
                     (int32_t*)nullptr, 0, n_active);
  return hipGetLastError() == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

fdllm_status fdllm_generation_workspace_size(const fdllm_generation_desc* d, size_t* bytes) {
  if (!d || !bytes || !desc_ok(d)) return FDLLM_ERR_INVALID_ARG;
  size_t ws = 0;
  const fdllm_status st = fdllm_workspace_size(d->B, d->G, d->V, FDLLM_BF16, &ws);
  if (st != FDLLM_OK) return st;
  *bytes = align256(sizeof(GenState)) + align256((size_t)d->B * 4) + align256(ws);
  return FDLLM_OK;
}

fdllm_status fdllm_generation_create(const fdllm_generation_desc* d, fdllm_generation* out) {
  if (!out) return FDLLM_ERR_INVALID_ARG;
  *out = nullptr;
  size_t need = 0;
  const fdllm_status st = fdllm_generation_workspace_size(d, &need);
  if (st != FDLLM_OK) return st;
  if (!d->workspace || d->workspace_bytes < need) return FDLLM_ERR_WORKSPACE;
  fdllm_generation g = (fdllm_generation)calloc(1, sizeof(fdllm_generation_s));
  if (!g) return FDLLM_ERR_HIP;
  g->d = *d;
  char* w = (char*)d->workspace;
  g->st = (GenState*)w;
  g->n_commit = (int32_t*)(w + align256(sizeof(GenState)));
  g->step_ws = w + align256(sizeof(GenState)) + align256((size_t)d->B * 4);
  g->step_ws_bytes = need - align256(sizeof(GenState)) - align256((size_t)d->B * 4);
  bool ok = hipEventCreateWithFlags(&g->ev[0], hipEventDisableTiming) == hipSuccess &&
            hipEventCreateWithFlags(&g->ev[1], hipEventDisableTiming) == hipSuccess &&
            hipHostMalloc((void**)&g->host_active, 64, hipHostMallocDefault) == hipSuccess;
  if (ok && d->use_graph) {
    ok = hipStreamCreateWithFlags(&g->cap, hipStreamNonBlocking) == hipSuccess &&
         hipStreamBeginCapture(g->cap, hipStreamCaptureModeThreadLocal) == hipSuccess;
    if (ok) {
      const fdllm_status es = enqueue_steps(g, d->chunk, g->cap);
      const bool ended = hipStreamEndCapture(g->cap, &g->graph) == hipSuccess;
      ok = es == FDLLM_OK && ended &&
           hipGraphInstantiate(&g->exec, g->graph, nullptr, nullptr, 0) == hipSuccess;
    }
  }
  if (!ok) {
    fdllm_generation_destroy(g);
    return FDLLM_ERR_HIP;
  }
  *out = g;
  return FDLLM_OK;
}

fdllm_status fdllm_generation_run(fdllm_generation g, fdllm_stream stream, int32_t* steps) {
  if (!g) return FDLLM_ERR_INVALID_ARG;
  const fdllm_generation_desc& d = g->d;
  hipStream_t s = (hipStream_t)stream;
  const int ig = (int)(((long long)d.B * d.G + 255) / 256);
  hipLaunchKernelGGL(k_init, dim3((unsigned)(ig < 65536 ? (ig > 0 ? ig : 1) : 65536)), dim3(256), 0,
                     s, d.mask, d.x, d.block_start, d.block_end, d.B, d.G, d.blk, g->st);
  if (hipGetLastError() != hipSuccess) return FDLLM_ERR_HIP;
  const int chunks = (d.max_steps + d.chunk - 1) / d.chunk;
  for (int c = 0; c < chunks; ++c) {
    if (d.use_graph) {
      if (hipGraphLaunch(g->exec, s) != hipSuccess) return FDLLM_ERR_HIP;
    } else {
      const fdllm_status st = enqueue_steps(g, d.chunk, s);
      if (st != FDLLM_OK) return st;
    }
    if (hipMemcpyAsync(g->host_active + (c & 1), &g->st->active, sizeof(int32_t),
                       hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipEventRecord(g->ev[c & 1], s) != hipSuccess)
      return FDLLM_ERR_HIP;
    // one chunk behind the device: the previous chunk's count decides
    if (c >= 1) {
      if (hipEventSynchronize(g->ev[(c - 1) & 1]) != hipSuccess) return FDLLM_ERR_HIP;
      if (g->host_active[(c - 1) & 1] == 0) break;
    }
  }
  if (hipStreamSynchronize(s) != hipSuccess) return FDLLM_ERR_HIP;
  if (steps) {
    GenState h{};
    if (hipMemcpy(&h, g->st, sizeof(GenState), hipMemcpyDeviceToHost) != hipSuccess)
      return FDLLM_ERR_HIP;
    *steps = h.t;
  }
  return FDLLM_OK;
}

fdllm_status fdllm_generation_destroy(fdllm_generation g) {
  if (!g) return FDLLM_OK;
  // every resource is released; the first failure is reported
  hipError_t first = hipSuccess;
  auto note = [&first](hipError_t e) {
    if (first == hipSuccess) first = e;
  };
  if (g->exec) note(hipGraphExecDestroy(g->exec));
  if (g->graph) note(hipGraphDestroy(g->graph));
  if (g->cap) note(hipStreamDestroy(g->cap));
  if (g->ev[0]) note(hipEventDestroy(g->ev[0]));
  if (g->ev[1]) note(hipEventDestroy(g->ev[1]));
  if (g->host_active) note(hipHostFree(g->host_active));
  free(g);
  return first == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

}  // extern "C"
