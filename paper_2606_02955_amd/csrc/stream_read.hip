// stream_read.hip -- read-only HBM stream on gfx950, the bandwidth reference
// for the vocabulary pass (see include/fdllm_bench.h for the contract).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "fdllm_bench.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kWavesPerGroup = 4;
constexpr int kU = 8;                        // 16-byte loads per lane per batch
constexpr int kChunkLoads = 256;             // wave-wide 1 KiB loads per chunk (256 KiB)
constexpr long long kChunkVecs = (long long)kChunkLoads * kWave;
// At most 192 persistent workgroups (768 wavefronts, 16 KiB in flight each):
// the fastest of 64 to 8192 workgroups on an 8.29 GB buffer; more concurrent
// streams lower the rate (7.25 TB/s at 192, 7.04 at 256, 6.6 at 1024).
constexpr long long kMaxGroups = 192;

__device__ __forceinline__ uint32_t fold(const u32x4& r) { return r.x ^ r.y ^ r.z ^ r.w; }

// Persistent wavefronts take chunks round-robin; inside a full chunk two
// batches of kU loads are in flight (the next batch is issued before the
// current one is consumed).
__global__ void __launch_bounds__(kWave * kWavesPerGroup)
k_stream_read(const u32x4* __restrict__ src, long long nvec, uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x % kWave;
  const long long wave = (long long)blockIdx.x * kWavesPerGroup + threadIdx.x / kWave;
  const long long nwaves = (long long)gridDim.x * kWavesPerGroup;
  const long long nchunks = (nvec + kChunkVecs - 1) / kChunkVecs;
  uint32_t acc = 0;
  for (long long c = wave; c < nchunks; c += nwaves) {
    const long long v0 = c * kChunkVecs;
    const u32x4* q = src + v0 + lane;
    if (v0 + kChunkVecs <= nvec) {
      u32x4 a[kU], b[kU];
#pragma unroll
      for (int u = 0; u < kU; ++u) a[u] = __builtin_nontemporal_load(q + u * kWave);
#pragma unroll 1
      for (int j = 0; j < kChunkLoads; j += 2 * kU) {
#pragma unroll
        for (int u = 0; u < kU; ++u) b[u] = __builtin_nontemporal_load(q + (j + kU + u) * kWave);
#pragma unroll
        for (int u = 0; u < kU; ++u) acc ^= fold(a[u]);
        if (j + 2 * kU < kChunkLoads) {
#pragma unroll
          for (int u = 0; u < kU; ++u) a[u] = __builtin_nontemporal_load(q + (j + 2 * kU + u) * kWave);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) acc ^= fold(b[u]);
      }
    } else {
      for (long long v = v0 + lane; v < nvec; v += kWave) acc ^= fold(__builtin_nontemporal_load(src + v));
    }
  }
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) acc ^= (uint32_t)__shfl_xor((int)acc, d);
  if (lane == 0) atomicXor(sink, acc);
}

}  // namespace

extern "C" int fdllm_stream_read(const void* src, size_t bytes, uint32_t* sink,
                                 fdllm_bench_stream stream) {
  if (bytes == 0) return 0;
  if (!src || !sink || bytes % 16 != 0 || ((uintptr_t)src % 16) != 0) return -1;
  const long long nvec = (long long)(bytes / 16);
  const long long nchunks = (nvec + kChunkVecs - 1) / kChunkVecs;
  // every wavefront takes the same number of chunks (no partial last round)
  const long long per_wave = (nchunks + kMaxGroups * kWavesPerGroup - 1) / (kMaxGroups * kWavesPerGroup);
  const long long waves = (nchunks + per_wave - 1) / per_wave;
  const long long groups = (waves + kWavesPerGroup - 1) / kWavesPerGroup;
  hipLaunchKernelGGL(k_stream_read, dim3((unsigned)groups), dim3(kWave * kWavesPerGroup), 0,
                     (hipStream_t)stream, (const u32x4*)src, nvec, sink);
  return hipGetLastError() == hipSuccess ? 0 : -5;
}
