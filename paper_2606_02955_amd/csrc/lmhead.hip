// lmhead.hip -- the LM head fused with the vocabulary pass on gfx950.
//
// Alg. 1's model call ends in the output projection: a candidate position's
// logits are l_v = sum_k h_k W_vk.  Here they are formed tile by tile on the
// matrix cores (v_mfma_f32_16x16x32_bf16, bf16 operands, float32
// accumulation) and folded straight into the vocabulary pass's online
// (maximum, exponent reference, sum, argmax) state, so no logit reaches HBM;
// the per-position outputs and the selection are then those of
// fdllm_confidence / fdllm_decode_step (Sec. 3 "Notation"; Alg. 1).
//
// Main loop of the partial kernel: a workgroup of 8 waves owns 256 candidate
// positions x 256 vocabulary rows per tile; the hidden dimension streams in
// stages of 64 elements (128 bytes of every weight and hidden row, so each
// load uses whole cache lines; 64 KiB per stage) that buffer_load ... lds
// writes straight into LDS, two stages resident.  One barrier per stage;
// each wave's 64 MFMAs of a stage are interleaved with the reads of the next
// half stage's operands, and the second half with the loads of the stage
// after next.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <atomic>

#include "fdllm.h"
#include "pass_common.h"

namespace fdllm {

// ---------------------------------------------------------------------------
// LM head fused with the vocabulary pass: logits = hidden . W^T are formed
// tile by tile in MFMA accumulators and folded into the per-row online
// (max, exponent reference, sum, argmax) state; no logit is written to HBM.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kLmWaves = 8;                    // waves per workgroup
constexpr int kLmVt = 256;                     // vocabulary rows per tile (MFMA A operand)
constexpr int kLmPt = 256;                     // positions per workgroup (MFMA B operand)
constexpr int kLmBK = 64;                      // hidden-dimension elements per LDS stage
constexpr int kLmNBuf = 2;                     // stages resident in LDS
constexpr int kLmThreads = kLmWaves * kWave;
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

// Folds the lane's 32 accumulators of one position (vocabulary entries
// base + 16 mi + i, increasing in (mi, i)) into its state.
__device__ __forceinline__ void lm_fold(LmState& st, const f32x4 (&acc)[8][4], int ni, int base,
                                          int V) {
  float tm = kNegInf;
#pragma unroll
  for (int mi = 0; mi < 8; ++mi)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = base + 16 * mi + i;
      if (v < V) tm = fmaxf(tm, acc[mi][ni][i]);
    }
  if (tm > st.M) {
    const float Kn = exp_ref(tm);
    st.S = rescale(st.S, st.K, Kn);
    st.K = Kn;
    st.M = tm;
    int f = 0x7fffffff;
#pragma unroll
    for (int mi = 7; mi >= 0; --mi)
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        const int v = base + 16 * mi + i;
        if (v < V && acc[mi][ni][i] == tm) f = v;
      }
    st.first = f;
  }
  // every term enters a double sum on its own, so the greedy element's term
  // stays exact and s' = (S - e_M) / e_M keeps its relative accuracy
  double sum[2] = {0.0, 0.0};
#pragma unroll
  for (int mi = 0; mi < 8; ++mi)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = base + 16 * mi + i;
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

// ---- LDS-DMA main loop -----------------------------------------------------
// Stages of kLmBK hidden elements: 256 weight rows and 256 hidden rows of
// kLmBK * 2 bytes each, written by buffer_load ... lds (each lane of a wave
// instruction fills the next 16 bytes of LDS).  The stage after next is
// loaded into the buffer of the stage just read, in the second half of the
// current stage.  Rows are stored unpadded; the 16-byte vector s of row r
// sits in slot s ^ lm_swz(r).  lm_swz was chosen from LDS bank-conflict
// counter measurements of ds_read_b128 patterns on gfx950: with it the
// operand reads (lane l: row l % 16, vector 4 h + l / 16) are conflict-free.
constexpr int kLmSlots = kLmBK / 8;                       // 16-byte vectors per row and stage
constexpr int kLmRowBytes = kLmBK * 2;
constexpr int kLmWBytes = kLmVt * kLmRowBytes;            // weight part of a stage
constexpr int kLmStageBytes = (kLmVt + kLmPt) * kLmRowBytes;
constexpr int kLmDmaRows = kWave / kLmSlots;              // rows per wave-wide load
constexpr int kLmWDma = kLmVt / kLmDmaRows / kLmWaves;    // weight loads per wave and stage
constexpr int kLmHDma = kLmPt / kLmDmaRows / kLmWaves;
constexpr int kLmDmaPerStage = kLmWDma + kLmHDma;
constexpr size_t kLmLdsBytes = (size_t)kLmNBuf * kLmStageBytes;
static_assert(kLmWDma == 4 && kLmHDma == 4, "the interleaved schedule issues four loads of each");

__device__ __forceinline__ int lm_swz(int r) { return (r & 1) | ((r >> 1) & 2) | ((r << 1) & 4); }

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef int i32x4 __attribute__((ext_vector_type(4)));

// buffer resource of a raw byte range (stride 0, bounds check on the byte
// offset), all four words wave-uniform
__device__ __forceinline__ i32x4 lm_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// one wave-wide 16-byte-per-lane load into LDS: lane i's vector lands at
// byte lds + 16 i.  Issued as inline assembly: the compiler cannot tell which
// buffer such a load writes and would drain every load in flight before the
// next LDS read; the explicit vmcnt waits of lm_sync are the ones needed.
__device__ __forceinline__ void lm_dma(i32x4 rsrc, uint32_t lds, uint32_t voff, int soff) {
  int keep;   // m0 is the compiler's register: saved and restored around the load
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %2, %3, %4 offen lds\n\t"
               "s_mov_b32 m0, %0"
               : "=&s"(keep) : "s"(lds), "v"(voff), "s"(rsrc), "s"(soff) : "memory");
}

// waits until at most N of this wave's loads are outstanding and its LDS
// reads are done, then meets the other waves; the memory clobber keeps LDS
// accesses on their side
template <int N>
__device__ __forceinline__ void lm_sync() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

#define LM_FENCE() __builtin_amdgcn_sched_barrier(0)

// the producer: the next stage this wave loads (tile relative to the
// workgroup's first, stage within the tile), the buffer it goes to, and the
// lane's load offsets.  Past the last stage the last one is loaded again
// (into a buffer nobody reads any more), so every stage issues the same
// number of loads.
struct LmProducer {
  int tile, ks, left, buf;
  i32x4 wr, hr;
  uint32_t w_voff[kLmWDma], h_voff[kLmHDma];
  uint32_t lds_w[kLmWDma], lds_h[kLmHDma];   // wave's LDS offsets within a stage
};

__device__ __forceinline__ void lm_tile_setup(LmProducer& p, const uint16_t* weight, int t, int V,
                                              int d, int lane, int wave) {
  const int n0 = t * kLmVt;
  const uint32_t row_bytes = (uint32_t)d * 2u;
  p.wr = lm_rsrc(weight + (size_t)n0 * d, kLmVt * row_bytes);
  const int lr = lane / kLmSlots, ls = lane % kLmSlots;
#pragma unroll
  for (int j = 0; j < kLmWDma; ++j) {
    const int r = (wave * kLmWDma + j) * kLmDmaRows + lr;
    const int v = min(n0 + r, V - 1) - n0;              // rows past the vocabulary repeat the last
    p.w_voff[j] = (uint32_t)v * row_bytes + (uint32_t)((ls ^ lm_swz(r)) * 16);
  }
}

// grid (position tiles, vocabulary splits).  A workgroup takes kLmPt
// candidate positions and the split's vocabulary tiles of kLmVt rows; wave w
// computes vocabulary rows 128 (w % 2) .. +127 of a tile against positions
// 64 (w / 2) .. +63 as 8 x 4 MFMA 16x16x32 blocks, vocabulary along the MFMA
// rows: lane l holds positions 16 ni + l % 16 and, for each, vocabulary rows
// 16 mi + 4 (l / 16) + i of the wave's 128.
__global__ void __launch_bounds__(kLmThreads)
k_lm_partial(const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ weight,
             const int32_t* __restrict__ rows, const int32_t* __restrict__ count, int d, int V,
             int tiles_per_split, uint32_t hid_bytes, WavePartial* __restrict__ partials, int n_split) {
  extern __shared__ __attribute__((aligned(1024))) char lm_lds[];
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int vw = wave % 2, pw = wave / 2;
  const int nrows = *count;
  const int p0 = blockIdx.x * kLmPt;
  if (p0 >= nrows) return;
  const int n_tiles = (V + kLmVt - 1) / kLmVt;
  const int t_begin = blockIdx.y * tiles_per_split;
  const int t_end = min(t_begin + tiles_per_split, n_tiles);
  const int nks = d / kLmBK;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)lm_lds;

  LmProducer pr;
  pr.tile = 0;
  pr.ks = 0;
  pr.left = (t_end - t_begin) * nks;
  pr.buf = 0;
  pr.hr = lm_rsrc(hidden, hid_bytes);
  {
    const int lr = lane / kLmSlots, ls = lane % kLmSlots;
#pragma unroll
    for (int j = 0; j < kLmHDma; ++j) {
      const int r = (wave * kLmHDma + j) * kLmDmaRows + lr;
      const int q = p0 + r < nrows ? p0 + r : p0;       // past the end: repeat the first row
      pr.h_voff[j] = (uint32_t)rows[q] * (uint32_t)d * 2u + (uint32_t)((ls ^ lm_swz(r)) * 16);
      pr.lds_h[j] = (uint32_t)(kLmWBytes + (wave * kLmHDma + j) * kLmDmaRows * kLmRowBytes);
    }
#pragma unroll
    for (int j = 0; j < kLmWDma; ++j)
      pr.lds_w[j] = (uint32_t)((wave * kLmWDma + j) * kLmDmaRows * kLmRowBytes);
  }
  lm_tile_setup(pr, weight, t_begin, V, d, lane, wave);

  // the loads of the producer's stage: W j (j < 4) or H j - 4
  auto dma = [&](int j) {
    const uint32_t sb = lds0 + (uint32_t)pr.buf * kLmStageBytes;
    const int soff = pr.ks * kLmRowBytes;
    if (j < kLmWDma)
      lm_dma(pr.wr, sb + pr.lds_w[j], pr.w_voff[j], soff);
    else
      lm_dma(pr.hr, sb + pr.lds_h[j - kLmWDma], pr.h_voff[j - kLmWDma], soff);
  };
  auto advance = [&]() {
    if (pr.left > 1) {
      --pr.left;
      if (++pr.ks == nks) {
        pr.ks = 0;
        ++pr.tile;
        lm_tile_setup(pr, weight, t_begin + pr.tile, V, d, lane, wave);
      }
    }
    pr.buf = pr.buf + 1 == kLmNBuf ? 0 : pr.buf + 1;
  };

  // operand addresses of this lane: row l % 16 of a 16-row block, 16-byte
  // vector 4 h + l / 16 of the stage's 64 hidden elements in half h
  uint32_t a_addr[2], b_addr[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t slot = (uint32_t)(((4 * h + lane / 16) ^ lm_swz(lane % 16)) * 16);
    a_addr[h] = (uint32_t)((128 * vw + lane % 16) * kLmRowBytes) + slot;
    b_addr[h] = (uint32_t)(kLmWBytes + (64 * pw + lane % 16) * kLmRowBytes) + slot;
  }
  auto lds_at = [&](uint32_t a) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(lm_lds + (a - lds0));
  };

  LmState st[4];
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) st[ni] = LmState{kNegInf, kRefFloor, 0.0, 0x7fffffff};

  f32x4 acc[8][4];
  bf16x8 fa[8], fb[4], nb4[4], na7;
#define LM_M(mi, ni) acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[mi], fb[ni], acc[mi][ni], 0, 0, 0)
  // the 32 MFMAs of one half stage on (fa, fb); the operands of the next half
  // stage (weight operands at sa, hidden operands at sb) are read as the
  // registers they replace fall dead; with_loads also issues the stage loads
  auto half = [&](uint32_t sa, uint32_t sb, bool with_loads) {
    LM_M(0, 0); LM_FENCE(); nb4[0] = lds_at(sb); LM_FENCE();
    LM_M(0, 1); LM_FENCE(); nb4[1] = lds_at(sb + 16 * kLmRowBytes); LM_FENCE();
    LM_M(0, 2); LM_FENCE(); nb4[2] = lds_at(sb + 32 * kLmRowBytes); LM_FENCE();
    LM_M(0, 3); LM_FENCE(); nb4[3] = lds_at(sb + 48 * kLmRowBytes); LM_FENCE();
#pragma unroll
    for (int mi = 1; mi < 8; ++mi) {
      LM_M(mi, 0); LM_FENCE();
      fa[mi - 1] = lds_at(sa + (mi - 1) * 16 * kLmRowBytes); LM_FENCE();
      LM_M(mi, 1); LM_FENCE();
      if (with_loads) { dma(mi - 1); LM_FENCE(); }
      if (mi == 7) { na7 = lds_at(sa + 7 * 16 * kLmRowBytes); LM_FENCE(); }
      LM_M(mi, 2); LM_FENCE();
      if (with_loads && mi == 7) { dma(7); LM_FENCE(); }
      LM_M(mi, 3); LM_FENCE();
    }
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) fb[ni] = nb4[ni];
    fa[7] = na7;
  };

  // prologue: both buffers' stages in flight, then wait for the first
  for (int s = 0; s < kLmNBuf; ++s) {
#pragma unroll
    for (int j = 0; j < kLmDmaPerStage; ++j) dma(j);
    advance();
  }
  lm_sync<kLmDmaPerStage>();
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) fb[ni] = lds_at(lds0 + b_addr[0] + ni * 16 * kLmRowBytes);
#pragma unroll
  for (int mi = 0; mi < 8; ++mi) fa[mi] = lds_at(lds0 + a_addr[0] + mi * 16 * kLmRowBytes);

  int cbuf = 0;
  for (int t = t_begin; t < t_end; ++t) {
#pragma unroll
    for (int mi = 0; mi < 8; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mi][ni][i] = 0.0f;
    for (int ks = 0; ks < nks; ++ks) {
      const uint32_t cb = lds0 + (uint32_t)cbuf * kLmStageBytes;
      const int nbuf = cbuf ^ 1;
      const uint32_t nb = lds0 + (uint32_t)nbuf * kLmStageBytes;
      // first half: MFMAs on the stage's half 0, its half 1 read in between
      LM_FENCE();
      half(cb + a_addr[1], cb + b_addr[1], false);
      // every wave has read all of this stage's buffer, and the next stage
      // (the only loads outstanding) has landed
      LM_FENCE();
      lm_sync<0>();
      // second half: MFMAs on half 1; the next stage's half 0 read and the
      // stage after it loaded into this stage's buffer in between
      half(nb + a_addr[0], nb + b_addr[0], true);
      LM_FENCE();
      advance();
      cbuf = nbuf;
    }
    const int base = t * kLmVt + 128 * vw + 4 * (lane / 16);
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) lm_fold(st[ni], acc, ni, base, V);
  }
#undef LM_M
  // lanes l, l^16, l^32, l^48 hold the same positions
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
#pragma unroll
    for (int x = 16; x <= 32; x *= 2) {
      const float M2 = __shfl_xor(st[ni].M, x);
      const float K2 = __shfl_xor(st[ni].K, x);
      const double S2 = __shfl_xor(st[ni].S, x);
      const int f2 = __shfl_xor(st[ni].first, x);
      lm_combine(st[ni], M2, K2, S2, f2);
    }
  }
  // the two vocabulary halves of a position meet in LDS, once no load is
  // still writing into it
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  WavePartial* xch = reinterpret_cast<WavePartial*>(lm_lds);
  __syncthreads();
  if (vw == 1 && lane < 16) {
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
      xch[64 * pw + 16 * ni + lane] = WavePartial{st[ni].M, st[ni].K, st[ni].S, st[ni].first};
  }
  __syncthreads();
  if (vw != 0 || lane >= 16) return;
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const WavePartial o = xch[64 * pw + 16 * ni + lane];
    lm_combine(st[ni], o.m, o.K, o.S, o.first);
    const int r = p0 + 64 * pw + 16 * ni + lane;
    if (r < nrows)
      partials[(size_t)r * n_split + blockIdx.y] = WavePartial{st[ni].M, st[ni].K, st[ni].S, st[ni].first};
  }
}

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
  if (B < 0 || L < 1 || V < 1 || d < 64 || d % 64 != 0) return false;
  // hidden is addressed by 32-bit byte offsets (buffer loads)
  return (long long)B * L * d * 2 <= 0xffffffffLL && (long long)V * (d / 8) < 0x7fffffffLL;
}

// The partial kernel's dynamic LDS (128 KiB) is above the default limit; the
// limit is raised once per device, before the first launch there.
constexpr int kLmMaxDevices = 64;
static std::atomic<bool> lm_lds_allowed[kLmMaxDevices];

static hipError_t lm_allow_lds() {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kLmMaxDevices && lm_lds_allowed[dev].load(std::memory_order_acquire))
    return hipSuccess;
  const hipError_t a = hipFuncSetAttribute((const void*)k_lm_partial,
                                           hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)kLmLdsBytes);
  if (a == hipSuccess && dev >= 0 && dev < kLmMaxDevices)
    lm_lds_allowed[dev].store(true, std::memory_order_release);
  return a;
}

static hipError_t lm_launch(const void* hidden, const void* weight, int B, int L, int d, int V,
                            const uint8_t* mask, const int32_t* bs, const int32_t* be, RowOut out,
                            char* ws, const LmPlan& p, hipStream_t st) {
  int32_t* count = (int32_t*)ws;
  int32_t* rows = (int32_t*)(ws + p.off_rows);
  WavePartial* part = (WavePartial*)(ws + p.off_partials);
  const hipError_t attr = lm_allow_lds();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(k_lm_zero, dim3(1), dim3(64), 0, st, count);
  hipLaunchKernelGGL(k_lm_compact, dim3((unsigned)((B + 3) / 4)), dim3(256), 0, st, mask, bs, be, B,
                     L, rows, count, out);
  hipLaunchKernelGGL(k_lm_partial, dim3((unsigned)p.m_tiles, (unsigned)p.n_split), dim3(kLmThreads),
                     kLmLdsBytes, st, (const uint16_t*)hidden, (const uint16_t*)weight, rows, count,
                     d, V, p.tiles_per_split, (uint32_t)((size_t)B * L * d * 2), part, p.n_split);
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
