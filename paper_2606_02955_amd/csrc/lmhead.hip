// lmhead.hip -- the LM head fused with the vocabulary pass on gfx950.
//
// Alg. 1's model call ends in the output projection: a candidate position's
// logits are l_v = sum_k h_k W_vk.  Here they are formed tile by tile on the
// matrix cores (v_mfma_f32_32x32x16_bf16, bf16 operands, float32
// accumulation) and folded straight into the vocabulary pass's online
// (maximum, exponent reference, sum, argmax) state, so no logit reaches HBM;
// the per-position outputs and the selection are then those of
// fdllm_confidence / fdllm_decode_step (Sec. 3 "Notation"; Alg. 1).
#include <hip/hip_runtime.h>

#include <stdint.h>

#include "fdllm.h"
#include "pass_common.h"

namespace fdllm {

// ---------------------------------------------------------------------------
// LM head fused with the vocabulary pass: logits = hidden . W^T are formed
// tile by tile in MFMA accumulators and folded into the per-row online
// (max, exponent reference, sum, argmax) state; no logit is written to HBM.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kLmWaves = 8;                    // waves per workgroup
constexpr int kLmVt = 256;                     // vocabulary rows per tile (MFMA A operand)
constexpr int kLmPt = 256;                     // positions per workgroup (MFMA B operand)
constexpr int kLmBK = 64;                      // hidden-dimension elements per LDS stage
constexpr int kLmRowVec = kLmBK / 8 + 1;       // 16-byte vectors per LDS row (one of padding)
constexpr int kLmThreads = kLmWaves * kWave;
constexpr int kLmWChunks = kLmVt * (kLmBK / 8) / kLmThreads;   // 16-byte loads per thread
constexpr int kLmHChunks = kLmPt * (kLmBK / 8) / kLmThreads;
constexpr int kLmRows = kLmPt;                 // candidate rows per workgroup
constexpr int kLmCols = kLmVt;                 // vocabulary columns per tile

// Candidate rows of every sequence, compacted (any order: a row's result
// does not depend on the rows it shares a tile with); default outputs for
// every other position.  One wavefront per sequence.
__global__ void __launch_bounds__(256)
k_lm_compact(const uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
             const int32_t* __restrict__ bend, int B, int L, int32_t* __restrict__ rows,
             int32_t* __restrict__ count, RowOut out) {
  const int lane = threadIdx.x % kWave;
  const int b = blockIdx.x * 4 + threadIdx.x / kWave;
  if (b >= B) return;
  const int s = bstart[b], e = bend[b];
  const bool ok = window_ok(s, e, L);
  const size_t row0 = (size_t)b * L;
  for (int q0 = 0; q0 < L; q0 += kWave) {
    const int q = q0 + lane;
    const bool cand = q < L && ok && q >= s && q < e && mask[row0 + q] != 0;
    if (q < L && !cand) store_default(out, row0 + q);
    const unsigned long long bal = __ballot(cand);
    if (bal == 0ull) continue;
    int base = 0;
    if (lane == 0) base = atomicAdd(count, __popcll(bal));
    base = __shfl(base, 0);
    if (cand) rows[base + __popcll(bal & ((1ull << lane) - 1ull))] = (int32_t)(row0 + q);
  }
}

__global__ void k_lm_zero(int32_t* __restrict__ p) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *p = 0;
}

// Per-lane online state of one position over the vocabulary entries this
// lane sees.
struct LmState {
  float M, K;
  double S;
  int first;
};

// Folds the lane's 64 accumulators of one position (vocabulary entries
// base + 32 mi + 8 (i/4) + 4 h + i%4, increasing in (mi, i)) into its state.
__device__ __forceinline__ void lm_fold(LmState& st, const f32x16 (&acc)[4][2], int ni, int base,
                                        int V) {
  float tm = kNegInf;
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int v = base + 32 * mi + 8 * (i / 4) + i % 4;
      if (v < V) tm = fmaxf(tm, acc[mi][ni][i]);
    }
  if (tm > st.M) {
    const float Kn = exp_ref(tm);
    st.S = rescale(st.S, st.K, Kn);
    st.K = Kn;
    st.M = tm;
    int f = 0x7fffffff;
#pragma unroll
    for (int mi = 3; mi >= 0; --mi)
#pragma unroll
      for (int i = 15; i >= 0; --i) {
        const int v = base + 32 * mi + 8 * (i / 4) + i % 4;
        if (v < V && acc[mi][ni][i] == tm) f = v;
      }
    st.first = f;
  }
  // every term enters a double sum on its own, so the greedy element's term
  // stays exact and s' = (S - e_M) / e_M keeps its relative accuracy
  double sum[2] = {0.0, 0.0};
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int v = base + 32 * mi + 8 * (i / 4) + i % 4;
      sum[i & 1] += v < V ? (double)term(acc[mi][ni][i], st.K) : 0.0;
    }
  st.S += sum[0] + sum[1];
}

__device__ __forceinline__ void lm_combine(LmState& st, float M2, float K2, double S2, int f2) {
  const float Mn = fmaxf(st.M, M2);
  const int fa = st.M == Mn ? st.first : 0x7fffffff;
  const int fb = M2 == Mn ? f2 : 0x7fffffff;
  ks_combine(st.K, st.S, K2, S2);
  st.M = Mn;
  st.first = min(fa, fb);
}

// grid (position tiles, vocabulary splits).  A workgroup takes kLmPt
// candidate positions and the split's vocabulary tiles of kLmVt rows; wave w
// computes vocabulary rows 128 (w % 2) .. +127 of a tile against positions
// 64 (w / 2) .. +63 (4 x 2 MFMA 32x32x16 accumulators, vocabulary along the
// MFMA rows so each lane's accumulators belong to two positions only).
// Hidden-dimension stages of kLmBK are double-buffered in LDS.
__global__ void __launch_bounds__(kLmThreads)
k_lm_partial(const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ weight,
             const int32_t* __restrict__ rows, const int32_t* __restrict__ count, int d, int V,
             int tiles_per_split, WavePartial* __restrict__ partials, int n_split) {
  extern __shared__ u32x4 lm_lds[];
  constexpr int kWBuf = kLmVt * kLmRowVec, kHBuf = kLmPt * kLmRowVec;   // u32x4 per buffer
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  const int vw = wave % 2, pw = wave / 2;
  const int nrows = *count;
  const int p0 = blockIdx.x * kLmPt;
  if (p0 >= nrows) return;
  const int n_tiles = (V + kLmVt - 1) / kLmVt;
  const int t_begin = blockIdx.y * tiles_per_split;
  const int t_end = min(t_begin + tiles_per_split, n_tiles);
  const int dv = d / 8;                                   // 16-byte vectors per row of hidden / weight

  // chunk j of this thread: LDS row tid/8 + 64 j, vector tid % 8 (kLmBK / 8 == 8)
  const int c_row = tid / (kLmBK / 8), c_kc = tid % (kLmBK / 8);
  const int c_dst = c_row * kLmRowVec + c_kc;
  constexpr int kRowStep = kLmThreads / (kLmBK / 8);      // LDS rows between a thread's chunks
  const u32x4* hv = reinterpret_cast<const u32x4*>(hidden);
  const u32x4* wv = reinterpret_cast<const u32x4*>(weight);
  int h_off[kLmHChunks];                                  // u32x4 offsets (positions past the end repeat p0)
#pragma unroll
  for (int j = 0; j < kLmHChunks; ++j) {
    const int r = p0 + c_row + j * kRowStep;
    h_off[j] = rows[r < nrows ? r : p0] * dv + c_kc;
  }

  LmState st[2];
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) st[ni] = LmState{kNegInf, kRefFloor, 0.0, 0x7fffffff};

  const int nks = d / kLmBK;
  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * kLmVt;
    int w_off[kLmWChunks];
#pragma unroll
    for (int j = 0; j < kLmWChunks; ++j) {
      const int v = n0 + c_row + j * kRowStep;
      w_off[j] = (v < V ? v : V - 1) * dv + c_kc;
    }
    f32x16 acc[4][2];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mi][ni][i] = 0.0f;
    u32x4 rw[kLmWChunks], rh[kLmHChunks];
    // stage 0 into buffer 0, stage 1 into registers
#pragma unroll
    for (int j = 0; j < kLmWChunks; ++j) rw[j] = wv[w_off[j]];
#pragma unroll
    for (int j = 0; j < kLmHChunks; ++j) rh[j] = hv[h_off[j]];
    __syncthreads();                                      // the previous tile's reads are done
#pragma unroll
    for (int j = 0; j < kLmWChunks; ++j) lm_lds[c_dst + j * kRowStep * kLmRowVec] = rw[j];
#pragma unroll
    for (int j = 0; j < kLmHChunks; ++j) lm_lds[2 * kWBuf + c_dst + j * kRowStep * kLmRowVec] = rh[j];
    if (nks > 1) {
#pragma unroll
      for (int j = 0; j < kLmWChunks; ++j) rw[j] = wv[w_off[j] + kLmBK / 8];
#pragma unroll
      for (int j = 0; j < kLmHChunks; ++j) rh[j] = hv[h_off[j] + kLmBK / 8];
    }
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
      const u32x4* cw = lm_lds + (ks & 1) * kWBuf;
      const u32x4* ch = lm_lds + 2 * kWBuf + (ks & 1) * kHBuf;
#pragma unroll
      for (int kk = 0; kk < kLmBK / 16; ++kk) {
        const int kv = kk * 2 + lane / 32;                // 16-byte vector index along k
        bf16x8 b[2];
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          b[ni] = __builtin_bit_cast(bf16x8, ch[(64 * pw + 32 * ni + lane % 32) * kLmRowVec + kv]);
#pragma unroll
        for (int mi = 0; mi < 4; ++mi) {
          const bf16x8 a = __builtin_bit_cast(bf16x8, cw[(128 * vw + 32 * mi + lane % 32) * kLmRowVec + kv]);
#pragma unroll
          for (int ni = 0; ni < 2; ++ni)
            acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[ni], acc[mi][ni], 0, 0, 0);
        }
      }
      if (ks + 1 < nks) {                                 // stage ks+1: registers -> other buffer
        u32x4* nw = lm_lds + ((ks + 1) & 1) * kWBuf;
        u32x4* nh = lm_lds + 2 * kWBuf + ((ks + 1) & 1) * kHBuf;
#pragma unroll
        for (int j = 0; j < kLmWChunks; ++j) nw[c_dst + j * kRowStep * kLmRowVec] = rw[j];
#pragma unroll
        for (int j = 0; j < kLmHChunks; ++j) nh[c_dst + j * kRowStep * kLmRowVec] = rh[j];
      }
      if (ks + 2 < nks) {                                 // stage ks+2 in flight during the MFMAs
        const int off = (ks + 2) * (kLmBK / 8);
#pragma unroll
        for (int j = 0; j < kLmWChunks; ++j) rw[j] = wv[w_off[j] + off];
#pragma unroll
        for (int j = 0; j < kLmHChunks; ++j) rh[j] = hv[h_off[j] + off];
      }
      __syncthreads();
    }
    const int base = n0 + 128 * vw + 4 * (lane / 32);
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) lm_fold(st[ni], acc, ni, base, V);
  }
  // lanes l and l + 32 hold the same positions (interleaved vocabulary rows)
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    const float M2 = __shfl_xor(st[ni].M, 32);
    const float K2 = __shfl_xor(st[ni].K, 32);
    const double S2 = __shfl_xor(st[ni].S, 32);
    const int f2 = __shfl_xor(st[ni].first, 32);
    lm_combine(st[ni], M2, K2, S2, f2);
  }
  // the two vocabulary halves of a position meet in LDS (buffers are free now)
  WavePartial* xch = reinterpret_cast<WavePartial*>(lm_lds);
  __syncthreads();
  if (vw == 1 && lane < 32) {
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
      xch[64 * pw + 32 * ni + lane] = WavePartial{st[ni].M, st[ni].K, st[ni].S, st[ni].first};
  }
  __syncthreads();
  if (vw != 0 || lane >= 32) return;
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    const WavePartial o = xch[64 * pw + 32 * ni + lane];
    lm_combine(st[ni], o.m, o.K, o.S, o.first);
    const int r = p0 + 64 * pw + 32 * ni + lane;
    if (r < nrows)
      partials[(size_t)r * n_split + blockIdx.y] = WavePartial{st[ni].M, st[ni].K, st[ni].S, st[ni].first};
  }
}

constexpr size_t kLmLdsBytes = (size_t)(2 * kLmVt + 2 * kLmPt) * kLmRowVec * sizeof(u32x4);

// Per candidate row, one wavefront: lane l combines the splits l, l+64, ...
// of the row's contiguous partials, then a fixed butterfly over the lanes
// (both partners of every step form the same sum) and the finish.
__global__ void __launch_bounds__(256)
k_lm_finish(const int32_t* __restrict__ rows, const int32_t* __restrict__ count,
            const WavePartial* __restrict__ partials, int n_split, RowOut out) {
  const int lane = threadIdx.x % kWave;
  const int k = blockIdx.x * 4 + threadIdx.x / kWave;
  if (k >= *count) return;
  const WavePartial* p = partials + (size_t)k * n_split;
  float M = kNegInf;
  for (int j = lane; j < n_split; j += kWave) M = fmaxf(M, p[j].m);
  M = wave_max(M);
  const float K = exp_ref(M);
  double S = 0.0;
  int first = 0x7fffffff;
  for (int j = lane; j < n_split; j += kWave) {
    const WavePartial q = p[j];
    S += rescale(q.S, q.K, K);
    if (q.m == M) first = min(first, q.first);
  }
#pragma unroll
  for (int d = kWave / 2; d >= 1; d >>= 1) S += __shfl_xor(S, d);
  first = wave_min(first);
  if (lane == 0) store_row(out, (size_t)rows[k], finish_row(M, K, S, first));
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
constexpr int kLmCUs = 256;   // compute units of the target

struct LmPlan {
  int m_tiles, n_tiles, n_split, tiles_per_split;
  size_t off_rows, off_partials, off_out, bytes;
};

// Row tiles cover the upper bound B*L (tiles past the device-side count exit
// at once); the vocabulary is split so that about 512 workgroups run.
static LmPlan lm_plan(int B, int L, int V, bool need_out) {
  LmPlan p{};
  const long long n = (long long)B * L;
  p.m_tiles = (int)((n + kLmRows - 1) / kLmRows);
  p.n_tiles = (V + kLmCols - 1) / kLmCols;
  // one workgroup per CU at a time: pick the split with the shortest makespan
  // (rounds of 256 workgroups x tiles per workgroup), fewer splits on ties
  long long best = -1;
  p.tiles_per_split = p.n_tiles;
  for (int tps = 1; tps <= p.n_tiles; ++tps) {
    const long long split = (p.n_tiles + tps - 1) / tps;
    if (split > 65535) continue;
    const long long rounds = ((long long)p.m_tiles * split + kLmCUs - 1) / kLmCUs;
    const long long cost = rounds * tps;
    if (best < 0 || cost < best) {
      best = cost;
      p.tiles_per_split = tps;
    }
  }
  p.n_split = (p.n_tiles + p.tiles_per_split - 1) / p.tiles_per_split;
  p.off_rows = 256;
  p.off_partials = p.off_rows + align256((size_t)n * 4);
  p.off_out = p.off_partials + align256((size_t)n * p.n_split * sizeof(WavePartial));
  p.bytes = p.off_out + (need_out ? 3 * align256((size_t)n * 4) : 0);
  return p;
}

static bool lm_sizes_ok(int B, int L, int d, int V) {
  if (B < 0 || L < 1 || V < 1 || d < kLmBK || d % kLmBK != 0) return false;
  // 16-byte vector offsets into hidden and weight fit in 31 bits
  return (long long)B * L * (d / 8) < 0x7fffffffLL && (long long)V * (d / 8) < 0x7fffffffLL;
}

static hipError_t lm_launch(const void* hidden, const void* weight, int B, int L, int d, int V,
                            const uint8_t* mask, const int32_t* bs, const int32_t* be, RowOut out,
                            char* ws, const LmPlan& p, hipStream_t st) {
  int32_t* count = (int32_t*)ws;
  int32_t* rows = (int32_t*)(ws + p.off_rows);
  WavePartial* part = (WavePartial*)(ws + p.off_partials);
  // the partial kernel's LDS (147 KB) exceeds the default limit; set it on the
  // current device before anything is enqueued
  const hipError_t attr = hipFuncSetAttribute((const void*)k_lm_partial,
                                              hipFuncAttributeMaxDynamicSharedMemorySize,
                                              (int)kLmLdsBytes);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k_lm_zero, dim3(1), dim3(64), 0, st, count);
  hipLaunchKernelGGL(k_lm_compact, dim3((unsigned)((B + 3) / 4)), dim3(256), 0, st, mask, bs, be, B,
                     L, rows, count, out);
  hipLaunchKernelGGL(k_lm_partial, dim3((unsigned)p.m_tiles, (unsigned)p.n_split), dim3(kLmThreads),
                     kLmLdsBytes, st, (const uint16_t*)hidden, (const uint16_t*)weight, rows, count,
                     d, V, p.tiles_per_split, part, p.n_split);
  const long long n = (long long)B * L;
  hipLaunchKernelGGL(k_lm_finish, dim3((unsigned)((n + 3) / 4)), dim3(256), 0, st, rows, count,
                     part, p.n_split, out);
  return hipGetLastError();
}

}  // namespace fdllm

using namespace fdllm;

extern "C" {

fdllm_status fdllm_lmhead_workspace_size(int B, int L, int d, int V, size_t* bytes) {
  if (!bytes) return FDLLM_ERR_INVALID_ARG;
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!lm_sizes_ok(B, L, d, V)) return FDLLM_ERR_SIZE;
  *bytes = lm_plan(B, L, V, true).bytes;
  return FDLLM_OK;
}

static fdllm_status lm_common(const void* hidden, const void* weight, int B, int L, int d, int V,
                              const uint8_t* mask, const int32_t* bs, const int32_t* be,
                              RowOut& out, void* workspace, size_t workspace_bytes, hipStream_t st) {
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!lm_sizes_ok(B, L, d, V)) return FDLLM_ERR_SIZE;
  if (!hidden || !weight || !mask || !bs || !be) return FDLLM_ERR_INVALID_ARG;
  if (((uintptr_t)hidden % 16) != 0 || ((uintptr_t)weight % 16) != 0) return FDLLM_ERR_INVALID_ARG;
  const bool need_out = !out.tokens || !out.conf || !out.eps;
  const LmPlan p = lm_plan(B, L, V, need_out);
  if (!workspace || workspace_bytes < p.bytes) return FDLLM_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  const size_t n = (size_t)B * L;
  if (!out.tokens) out.tokens = (int32_t*)(ws + p.off_out);
  if (!out.conf) out.conf = (float*)(ws + p.off_out + align256(n * 4));
  if (!out.eps) out.eps = (float*)(ws + p.off_out + 2 * align256(n * 4));
  return lm_launch(hidden, weight, B, L, d, V, mask, bs, be, out, ws, p, st) == hipSuccess
             ? FDLLM_OK
             : FDLLM_ERR_HIP;
}

fdllm_status fdllm_lmhead_confidence(const void* hidden, const void* weight, int B, int L, int d,
                                     int V, const uint8_t* mask, const int32_t* block_start,
                                     const int32_t* block_end, int32_t* tokens, float* conf,
                                     float* eps, float* lse, void* workspace,
                                     size_t workspace_bytes, fdllm_stream stream) {
  if (B == 0 && L >= 1) return FDLLM_OK;
  if (!tokens || !conf) return FDLLM_ERR_INVALID_ARG;
  RowOut out{tokens, conf, eps, lse};
  return lm_common(hidden, weight, B, L, d, V, mask, block_start, block_end, out, workspace,
                   workspace_bytes, (hipStream_t)stream);
}

fdllm_status fdllm_lmhead_decode_step(const void* hidden, const void* weight, int B, int L, int d,
                                      int V, uint8_t* mask, const int32_t* block_start,
                                      const int32_t* block_end, int32_t* x, fdllm_selector sel,
                                      float param, const float* eta, float eta_uniform,
                                      int32_t* tokens, float* conf, float* eps, float* lse,
                                      uint8_t* commit, int32_t* n_commit, void* workspace,
                                      size_t workspace_bytes, fdllm_stream stream) {
  if (sel != FDLLM_SEL_THRESHOLD && sel != FDLLM_SEL_FACTOR && sel != FDLLM_SEL_PROFILE &&
      sel != FDLLM_SEL_ROBUST)
    return FDLLM_ERR_INVALID_ARG;
  if (!(eta_uniform == eta_uniform)) return FDLLM_ERR_INVALID_ARG;
  if (B == 0 && L >= 1) return FDLLM_OK;
  if (!x) return FDLLM_ERR_INVALID_ARG;
  RowOut out{tokens, conf, eps, lse};
  hipStream_t st = (hipStream_t)stream;
  const fdllm_status s1 = lm_common(hidden, weight, B, L, d, V, mask, block_start, block_end, out,
                                    workspace, workspace_bytes, st);
  if (s1 != FDLLM_OK) return s1;
  SelectIO io{out.conf, out.eps, mask, block_start, block_end, commit, n_commit, out.tokens, x,
              EtaIn{eta, eta_uniform}};
  return launch_select(sel, io, B, L, param, st) == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

}  // extern "C"
