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
// Three plans, by the number of positions N = B L:
//   N <= 32     k_lm_stream: W streamed once, hidden operands in registers,
//               logits folded in the kernel (HBM-bound);
//   N <= 64     k_lm_kstream + k_lm_ksum: the same with the hidden dimension
//               split over two workgroups, partial logits in the workspace;
//   otherwise   k_lm_partial: MFMA tiles of 256 positions x 256 rows
//               (bound by the matrix cores at large N);
// each followed by k_lm_finish, which combines the per-split states.
//
// Main loop of the partial kernel: a workgroup of 8 waves owns 256 candidate
// positions x 256 vocabulary rows per tile; the hidden dimension streams in
// stages of 64 elements (128 bytes of every weight and hidden row, so each
// load uses whole cache lines; 32 KiB of weights and 32 KiB of hidden states
// per stage) that buffer_load ... lds writes straight into LDS, three weight
// and two hidden stages resident (160 KiB).  One barrier per stage; each
// wave's 64 MFMAs of a stage are interleaved with the reads of the next half
// stage's operands, and the second half with the loads of the hidden part of
// the stage after next and the weight part of the one after that.
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

// Folds the lane's accumulators of one position (vocabulary entries
// base + 16 mi + i, increasing in (mi, i)) into its state.
template <int MI, int NI>
__device__ __forceinline__ void lm_fold(LmState& st, const f32x4 (&acc)[MI][NI], int ni, int base,
                                        int V) {
  float tm = kNegInf;
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
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
    for (int mi = MI - 1; mi >= 0; --mi)
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
  for (int mi = 0; mi < MI; ++mi)
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
// instruction fills the next 16 bytes of LDS).  The weight part runs one
// stage further ahead (three buffers; it comes from HBM or the Infinity
// Cache) than the hidden part (two buffers; mostly L2 hits); both are loaded
// into the buffers of the stage just read, in the second half of the current
// stage.  Rows are stored unpadded; the 16-byte vector s of row r
// sits in slot s ^ lm_swz(r).  lm_swz was chosen from LDS bank-conflict
// counter measurements of ds_read_b128 patterns on gfx950: with it the
// operand reads (lane l: row l % 16, vector 4 h + l / 16) are conflict-free.
constexpr int kLmSlots = kLmBK / 8;                       // 16-byte vectors per row and stage
constexpr int kLmRowBytes = kLmBK * 2;
constexpr int kLmWBytes = kLmVt * kLmRowBytes;            // weight part of a stage
constexpr int kLmDmaRows = kWave / kLmSlots;              // rows per wave-wide load
constexpr int kLmWDma = kLmVt / kLmDmaRows / kLmWaves;    // weight loads per wave and stage
constexpr int kLmHDma = kLmPt / kLmDmaRows / kLmWaves;
constexpr int kLmDmaPerStage = kLmWDma + kLmHDma;
constexpr int kLmWBuf = 3, kLmHBuf = 2;                  // weight and hidden stages resident
constexpr int kLmHBytes = kLmPt * kLmRowBytes;            // hidden part of a stage
constexpr int kLmHOff = kLmWBuf * kLmWBytes;              // hidden buffers after the weight ones
constexpr size_t kLmLdsBytes = (size_t)kLmWBuf * kLmWBytes + (size_t)kLmHBuf * kLmHBytes;
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
  int tile, ks, left, buf;        // weight stages
  int hks, hleft, hbuf;           // hidden stages (one behind)
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
  pr.hks = 0;
  pr.hleft = pr.left;
  pr.hbuf = 0;
  pr.hr = lm_rsrc(hidden, hid_bytes);
  {
    const int lr = lane / kLmSlots, ls = lane % kLmSlots;
#pragma unroll
    for (int j = 0; j < kLmHDma; ++j) {
      const int r = (wave * kLmHDma + j) * kLmDmaRows + lr;
      const int q = p0 + r < nrows ? p0 + r : p0;       // past the end: repeat the first row
      pr.h_voff[j] = (uint32_t)rows[q] * (uint32_t)d * 2u + (uint32_t)((ls ^ lm_swz(r)) * 16);
      pr.lds_h[j] = (uint32_t)(kLmHOff + (wave * kLmHDma + j) * kLmDmaRows * kLmRowBytes);
    }
#pragma unroll
    for (int j = 0; j < kLmWDma; ++j)
      pr.lds_w[j] = (uint32_t)((wave * kLmWDma + j) * kLmDmaRows * kLmRowBytes);
  }
  lm_tile_setup(pr, weight, t_begin, V, d, lane, wave);

  // the loads of the producers' stages: H j (j < 4) of the hidden producer,
  // then W j - 4 of the weight producer (one stage ahead)
  auto dma = [&](int j) {
    if (j < kLmHDma)
      lm_dma(pr.hr, lds0 + (uint32_t)pr.hbuf * kLmHBytes + pr.lds_h[j], pr.h_voff[j],
             pr.hks * kLmRowBytes);
    else
      lm_dma(pr.wr, lds0 + (uint32_t)pr.buf * kLmWBytes + pr.lds_w[j - kLmHDma],
             pr.w_voff[j - kLmHDma], pr.ks * kLmRowBytes);
  };
  auto advance_w = [&]() {
    if (pr.left > 1) {
      --pr.left;
      if (++pr.ks == nks) {
        pr.ks = 0;
        ++pr.tile;
        lm_tile_setup(pr, weight, t_begin + pr.tile, V, d, lane, wave);
      }
    }
    pr.buf = pr.buf + 1 == kLmWBuf ? 0 : pr.buf + 1;
  };
  auto advance_h = [&]() {
    if (pr.hleft > 1) {
      --pr.hleft;
      if (++pr.hks == nks) pr.hks = 0;
    }
    pr.hbuf ^= 1;
  };

  // operand addresses of this lane: row l % 16 of a 16-row block, 16-byte
  // vector 4 h + l / 16 of the stage's 64 hidden elements in half h
  uint32_t a_addr[2], b_addr[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t slot = (uint32_t)(((4 * h + lane / 16) ^ lm_swz(lane % 16)) * 16);
    a_addr[h] = (uint32_t)((128 * vw + lane % 16) * kLmRowBytes) + slot;
    b_addr[h] = (uint32_t)(kLmHOff + (64 * pw + lane % 16) * kLmRowBytes) + slot;
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

  // prologue: stages 0 and 1 of both, and the weight part of stage 2, in
  // flight (in this order), then wait for stage 0
  for (int s = 0; s < 2; ++s) {
#pragma unroll
    for (int j = 0; j < kLmDmaPerStage; ++j) dma(j);
    advance_h();
    advance_w();
  }
#pragma unroll
  for (int j = kLmHDma; j < kLmDmaPerStage; ++j) dma(j);
  advance_w();
  lm_sync<kLmDmaPerStage + kLmWDma>();
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) fb[ni] = lds_at(lds0 + b_addr[0] + ni * 16 * kLmRowBytes);
#pragma unroll
  for (int mi = 0; mi < 8; ++mi) fa[mi] = lds_at(lds0 + a_addr[0] + mi * 16 * kLmRowBytes);

  int wbuf = 0, hbuf = 0;     // buffers of the stage being consumed
  for (int t = t_begin; t < t_end; ++t) {
#pragma unroll
    for (int mi = 0; mi < 8; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[mi][ni][i] = 0.0f;
    for (int ks = 0; ks < nks; ++ks) {
      const uint32_t cw = lds0 + (uint32_t)wbuf * kLmWBytes, ch = lds0 + (uint32_t)hbuf * kLmHBytes;
      const int nwbuf = wbuf + 1 == kLmWBuf ? 0 : wbuf + 1, nhbuf = hbuf ^ 1;
      const uint32_t nw = lds0 + (uint32_t)nwbuf * kLmWBytes, nh = lds0 + (uint32_t)nhbuf * kLmHBytes;
      // first half: MFMAs on the stage's half 0, its half 1 read in between
      LM_FENCE();
      half(cw + a_addr[1], ch + b_addr[1], false);
      // every wave has read all of this stage's buffers, and the next stage
      // has landed (only the weight part of the one after is outstanding)
      LM_FENCE();
      lm_sync<kLmWDma>();
      // second half: MFMAs on half 1; the next stage's half 0 read, and the
      // hidden part of the stage after next and the weight part of the one
      // after that loaded into this stage's buffers, in between
      half(nw + a_addr[0], nh + b_addr[0], true);
      LM_FENCE();
      advance_h();
      advance_w();
      wbuf = nwbuf;
      hbuf = nhbuf;
    }
    const int base = t * kLmVt + 128 * vw + 4 * (lane / 16);
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) lm_fold<8, 4>(st[ni], acc, ni, base, V);
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

// ---------------------------------------------------------------------------
// at most kLsRows positions in all (one sequence's block)
// ---------------------------------------------------------------------------
// With few positions the LM head is bound by reading W once (2 V d bytes;
// the 2 N V d flop are a few percent of the matrix cores' time), and the rate
// of that read depends on how it is issued: streams that each read a few rows
// 8 KiB apart reach ~5 TB/s, a contiguous range per workgroup read by global
// loads ~7 TB/s, the same range by buffer_load ... lds ~6.2 TB/s.  Here every
// workgroup streams a contiguous range of W, kLsBlk whole rows (16 d bytes)
// per block: each wave load instruction reads 1 KiB in address order into
// registers, which are stored to LDS while the next block's loads are in
// flight.
// The 8 waves split the hidden dimension and keep their share of the
// positions' hidden operands in registers for the whole kernel; per block each
// wave runs its MFMAs over its share (A = the block's rows from LDS, B = the
// hidden operands), and 256 threads each sum one (row, position) logit over
// the 8 partial products and fold it into their own running state; the 8 row
// states of a position are combined at the end.  Every workgroup finds the
// candidate positions itself (there are at most 32); workgroup 0 also writes
// them out, with their count, for the finish, and the default outputs of the
// other positions.
constexpr int kLsRows = 32;        // positions served (two 16-column MFMA blocks)
constexpr int kLsWaves = 8;
constexpr int kLsBlk = 8;          // vocabulary rows per block
constexpr int kLsMaxD = 4096;      // hidden operands held in registers: d / 8 per wave
constexpr size_t kLsRedBytes = (size_t)kLsWaves * 2 * kWave * sizeof(f32x4);  // 16 KiB
// two row blocks and two sets of the waves' partial products (160 KiB at
// d = 4096, all of a CU's LDS)
constexpr size_t kLsLdsBytes(int d) { return 2 * (size_t)kLsBlk * d * 2 + 2 * kLsRedBytes; }

__device__ __forceinline__ int ls_swz(int r) { return r & 7; }

// DM = d / 512: 16-byte loads per thread and block; 2 DM 32-element chunks
// of the hidden dimension per wave
template <int DM>
__global__ void __launch_bounds__(kLsWaves * kWave)
k_lm_stream(const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ weight,
            const uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
            const int32_t* __restrict__ bend, int B, int L, int V, int32_t* __restrict__ rows,
            int32_t* __restrict__ count, RowOut out, WavePartial* __restrict__ partials,
            int n_split) {
  constexpr int d = DM * 512;
  constexpr int NC = 2 * DM;                                 // 32-element chunks per wave
  constexpr int vec_row = d / 8;                             // 16-byte vectors per row
  constexpr uint32_t blk_bytes = (uint32_t)kLsBlk * d * 2;
  extern __shared__ __attribute__((aligned(1024))) char ls_lds[];
  // the candidate list sits in the second set of partial products, first
  // written after the loop's second barrier
  int32_t* cand_rows = reinterpret_cast<int32_t*>(ls_lds + 2 * blk_bytes + kLsRedBytes);
  int* cand_n = reinterpret_cast<int*>(cand_rows + kLsRows);
  const int t = threadIdx.x;
  const int lane = t % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
  const int g = blockIdx.x;
  const int G = gridDim.x;

  // the candidate positions, in position order (B L <= kLsRows)
  if (wave == 0) {
    const int n = B * L;
    bool cand = false;
    if (lane < n) {
      const int b = lane / L, q = lane % L;
      const int s = bstart[b], e = bend[b];
      cand = window_ok(s, e, L) && q >= s && q < e && mask[lane] != 0;
    }
    const unsigned long long bal = __ballot(cand);
    const int idx = __popcll(bal & ((1ull << lane) - 1ull));
    if (cand) cand_rows[idx] = lane;
    if (lane == 0) *cand_n = __popcll(bal);
    if (g == 0) {
      if (cand) rows[idx] = lane;
      else if (lane < n) store_default(out, lane);
      if (lane == 0) *count = __popcll(bal);
    }
  }
  __syncthreads();
  const int nrows = *cand_n;
  if (nrows == 0) return;

  const int nblk = (V + kLsBlk - 1) / kLsBlk;
  const int b_beg = (int)((long long)g * nblk / G), b_end = (int)((long long)(g + 1) * nblk / G);
  const int cnt = b_end - b_beg;
  // partial products of block i in set i % 2: f32x4 [wave][ni][lane]
  float* red = reinterpret_cast<float*>(ls_lds + 2 * blk_bytes);
  const int k0 = wave * (d / kLsWaves);

  // the hidden operands of this wave's share, for positions 16 ni + l % 16
  // (past the count: the first row; their results are not stored)
  u32x4 hb[NC][2];
  {
    const int q0 = lane % 16, q1 = 16 + lane % 16;
    const uint16_t* h0 = hidden + (size_t)cand_rows[q0 < nrows ? q0 : 0] * d + k0 + 8 * (lane / 16);
    const uint16_t* h1 = hidden + (size_t)cand_rows[q1 < nrows ? q1 : 0] * d + k0 + 8 * (lane / 16);
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      hb[c][0] = *reinterpret_cast<const u32x4*>(h0 + 32 * c);
      hb[c][1] = *reinterpret_cast<const u32x4*>(h1 + 32 * c);
    }
  }
  // block loads: thread t loads the block's 16-byte vectors j * 512 + t into
  // registers (each wave instruction reads 1 KiB of W in address order) and
  // stores them to LDS slot (row r, vector s ^ ls_swz(r)): the rows are 2 d
  // bytes apart, a multiple of the bank period, and the swizzle puts the
  // operand reads of the 8 rows in distinct banks.
  const u32x4* wv = reinterpret_cast<const u32x4*>(weight);
  u32x4 stg[DM];
  auto load_regs = [&](int i) {
    const int vb = (b_beg + i) * kLsBlk;
#pragma unroll
    for (int j = 0; j < DM; ++j) {
      const int slot = j * kLsWaves * kWave + t;
      const int v = min(vb + slot / vec_row, V - 1);         // rows past V repeat the last
      stg[j] = __builtin_nontemporal_load(wv + (size_t)v * vec_row + slot % vec_row);
    }
  };
  auto store_lds = [&](int buf) {
    u32x4* bl = reinterpret_cast<u32x4*>(ls_lds + buf * blk_bytes);
#pragma unroll
    for (int j = 0; j < DM; ++j) {
      const int slot = j * kLsWaves * kWave + t;
      const int r = slot / vec_row, sv = slot % vec_row;
      bl[r * vec_row + (sv ^ ls_swz(r))] = stg[j];
    }
  };
  // the (row, position) of this thread's running state: threads 0..255 take
  // row fr = t / 32 of every block and position fp = t % 32
  const int fr = t / kLsRows, fp = t % kLsRows;
  const bool folds = t < kLsBlk * kLsRows;
  // where the logit of (fr, fp) sits among the waves' accumulators:
  // ni = fp / 16, lane 16 (fr / 4) + fp % 16, element fr % 4
  const int red_idx = ((fp / 16) * kWave + 16 * (fr / 4) + fp % 16) * 4 + fr % 4;
  LmState st{kNegInf, kRefFloor, 0.0, 0x7fffffff};
  // sums block i's 8 partial products of (fr, fp) and folds the logit
  auto fold = [&](int i) {
    const float* rs = red + (i & 1) * (kLsRedBytes / sizeof(float));
    const int v = (b_beg + i) * kLsBlk + fr;
    if (folds && v < V) {
      float x = rs[red_idx];
#pragma unroll
      for (int w = 1; w < kLsWaves; ++w) x += rs[w * 2 * kWave * 4 + red_idx];
      if (x > st.M) {
        const float Kn = exp_ref(x);
        st.S = rescale(st.S, st.K, Kn);
        st.K = Kn;
        st.M = x;
        st.first = v;
      }
      st.S += (double)term(x, st.K);
    }
  };
  // operand address of this lane in a buffer: row l % 8 (rows 8..15 of the
  // MFMA block repeat rows 0..7), vector k0 / 8 + 4 c + l / 16
  const int ar = lane % kLsBlk;
  const int a_row = ar * vec_row;

  load_regs(0);
  store_lds(0);
  // vmcnt(0): the hidden operands have arrived before the loop, so inside it
  // the only loads in flight are the next block's, waited for at its store
  // (without this the loop would wait for every load at its first MFMAs)
  __builtin_amdgcn_s_waitcnt(0x0f70);
  if (cnt > 1) load_regs(1);
  for (int it = 0; it < cnt; ++it) {
    const int buf = it & 1;
    // one barrier per block: block it is in LDS (stored during the previous
    // iteration), the previous block's partial products are complete, and
    // the fold that read this iteration's set (two blocks back) is done
    __syncthreads();
    const u32x4* bl = reinterpret_cast<const u32x4*>(ls_lds + buf * blk_bytes);
    // two accumulators per column block halve the dependent MFMA chain
    f32x4 acc[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[h][ni][i] = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int sv = k0 / 8 + 4 * c + lane / 16;
      const bf16x8 a = __builtin_bit_cast(bf16x8, bl[a_row + (sv ^ ls_swz(ar))]);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        acc[c & 1][ni] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            a, __builtin_bit_cast(bf16x8, hb[c][ni]), acc[c & 1][ni], 0, 0, 0);
    }
    f32x4* redv = reinterpret_cast<f32x4*>(red + buf * (kLsRedBytes / sizeof(float)));
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) redv[(wave * 2 + ni) * kWave + lane] = acc[0][ni] + acc[1][ni];
    // the previous block's logits, while other waves still multiply
    if (it > 0) fold(it - 1);
    // the next block into the buffer every wave finished reading before the
    // barrier above, then the block after it into the registers
    if (it + 1 < cnt) store_lds(buf ^ 1);
    if (it + 2 < cnt) load_regs(it + 2);
  }
  __syncthreads();
  fold(cnt - 1);
  // the row states of a position meet in LDS (the row buffers are free)
  __syncthreads();
  WavePartial* xs = reinterpret_cast<WavePartial*>(ls_lds);
  if (folds) xs[fr * kLsRows + fp] = WavePartial{st.M, st.K, st.S, st.first};
  __syncthreads();
  if (t < kLsRows && t < nrows) {
    LmState c = {xs[t].m, xs[t].K, xs[t].S, xs[t].first};
#pragma unroll
    for (int r = 1; r < kLsBlk; ++r) {
      const WavePartial o = xs[r * kLsRows + t];
      lm_combine(c, o.m, o.K, o.S, o.first);
    }
    partials[(size_t)t * n_split + g] = WavePartial{c.M, c.K, c.S, c.first};
  }
}

// ---------------------------------------------------------------------------
// 33..64 positions: the hidden dimension split over workgroups
// ---------------------------------------------------------------------------
// A CU's registers hold the hidden operands of about 32 positions at d = 4096,
// so for up to 32 S positions the hidden dimension is cut into S parts of
// d / S elements and workgroup g takes part g % S of the contiguous row range
// of group g / S: W is still read once, in blocks of 8 S rows x d / S
// elements (16 d bytes, 64 KiB at d = 4096; each row piece contiguous).  Wave
// w owns the 16 positions of column block w % 2S and the (w / 2S)-th of the
// part's elements (4 / S waves per column block), with those hidden operands
// in registers (128 VGPRs at d = 4096).  The waves' products of a block meet
// in LDS, where the next iteration adds the halves and writes the block's
// logits over the part (float32, MFMA accumulation) as one contiguous run of
// 16-byte vectors: plogits[part][v][position].  k_lm_ksum adds the S parts in
// order and folds them.  The plan uses S = 2: with S = 4 (128 positions) the
// partial logits' extra traffic (2 x 259 MB at V = 126464) and the 8-fold
// LDS operand reads left it no faster than the tiled kernel.
constexpr int kKsWaves = 8;

// two sets of the waves' products: 8 waves x S / 2 row blocks x 1 KiB each
template <int S>
constexpr size_t ks_red_bytes() {
  return 2 * (size_t)kKsWaves * (S / 2) * kWave * sizeof(f32x4);
}
// two row blocks and the products (144 KiB for S = 2 at d = 4096)
template <int S>
constexpr size_t ks_lds_bytes(int d) {
  return 2 * (size_t)16 * d + ks_red_bytes<S>();
}

template <int DM, int S>
__global__ void __launch_bounds__(kKsWaves * kWave)
k_lm_kstream(const uint16_t* __restrict__ hidden, const uint16_t* __restrict__ weight,
             const uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
             const int32_t* __restrict__ bend, int B, int L, int V, int32_t* __restrict__ rows,
             int32_t* __restrict__ count, RowOut out, float* __restrict__ plogits) {
  constexpr int d = DM * 512;
  constexpr int dk = d / S;                                 // elements per part
  constexpr int NP = kLsRows * S;                           // positions served
  constexpr int NB = NP / 16;                               // 16-column MFMA blocks
  constexpr int KW = kKsWaves / NB;                         // waves per column block
  constexpr int dw = dk / KW;                               // elements per wave (d / 4)
  constexpr int NC = dw / 32;                               // 32-element chunks per wave
  constexpr int R = 8 * S;                                  // rows per block
  constexpr int MB = R / 16;                                // 16-row MFMA blocks per block
  constexpr int vec_part = dk / 8;                          // 16-byte vectors per row piece
  constexpr int vec_row = d / 8;
  constexpr uint32_t blk_bytes = (uint32_t)R * dk * 2;
  constexpr int NL = (int)(blk_bytes / (kKsWaves * kWave * 16));  // loads per thread and block
  static_assert(KW * NB == kKsWaves && MB >= 1 && NL == DM && NC >= 1, "k-split shape");
  extern __shared__ __attribute__((aligned(1024))) char ks_lds[];
  // products: float [set][wave][row block][element][lane]
  float* red = reinterpret_cast<float*>(ks_lds + 2 * blk_bytes);
  constexpr int red_set = kKsWaves * MB * 4 * kWave;              // floats per set
  // the candidate list sits in the second set, first written after the
  // loop's second barrier
  int32_t* cand_rows = reinterpret_cast<int32_t*>(red + red_set);
  int* cand_n = cand_rows + NP;
  const int t = threadIdx.x;
  const int lane = t % kWave;
  const int wave = __builtin_amdgcn_readfirstlane(t / kWave);
  const int g = blockIdx.x;
  const int kp = g % S;                                     // part of the hidden dimension
  const int gr = g / S, GR = gridDim.x / S;                 // row-range group

  // the candidate positions, in position order (B L <= NP)
  if (wave == 0) {
    const int n = B * L;
    int base = 0;
    for (int q0 = 0; q0 < NP; q0 += kWave) {
      const int q = q0 + lane;
      bool cand = false;
      if (q < n) {
        const int b = q / L, i = q % L;
        const int s = bstart[b], e = bend[b];
        cand = window_ok(s, e, L) && i >= s && i < e && mask[q] != 0;
      }
      const unsigned long long bal = __ballot(cand);
      const int idx = base + __popcll(bal & ((1ull << lane) - 1ull));
      if (cand) cand_rows[idx] = q;
      if (g == 0) {
        if (cand) rows[idx] = q;
        else if (q < n) store_default(out, q);
      }
      base += __popcll(bal);
    }
    if (lane == 0) {
      *cand_n = base;
      if (g == 0) *count = base;
    }
  }
  __syncthreads();
  const int nrows = *cand_n;
  if (nrows == 0) return;

  const int nblk = (V + R - 1) / R;
  const int b_beg = (int)((long long)gr * nblk / GR), b_end = (int)((long long)(gr + 1) * nblk / GR);
  const int cnt = b_end - b_beg;
  const int cb = wave % NB, kw = wave / NB;
  const int k0 = kp * dk + kw * dw;                         // this wave's first element

  // hidden operands of positions 16 cb + l % 16 (past the count: the first
  // row; their logits are written but never folded)
  u32x4 hb[NC];
  {
    const int q = 16 * cb + lane % 16;
    const uint16_t* h = hidden + (size_t)cand_rows[q < nrows ? q : 0] * d + k0 + 8 * (lane / 16);
#pragma unroll
    for (int c = 0; c < NC; ++c) hb[c] = *reinterpret_cast<const u32x4*>(h + 32 * c);
  }
  // block loads as in k_lm_stream, over the part's row pieces; LDS slot
  // (row r, vector s) holds the piece's vector s ^ (r % 16), so the 16 rows
  // an operand read touches sit in distinct banks
  const u32x4* wv = reinterpret_cast<const u32x4*>(weight);
  u32x4 stg[NL];
  auto load_regs = [&](int i) {
    const int vb = (b_beg + i) * R;
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int slot = j * kKsWaves * kWave + t;
      const int v = min(vb + slot / vec_part, V - 1);       // rows past V repeat the last
      stg[j] = __builtin_nontemporal_load(wv + (size_t)v * vec_row + kp * vec_part + slot % vec_part);
    }
  };
  auto store_lds = [&](int buf) {
    u32x4* bl = reinterpret_cast<u32x4*>(ks_lds + buf * blk_bytes);
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int slot = j * kKsWaves * kWave + t;
      const int r = slot / vec_part, sv = slot % vec_part;
      bl[r * vec_part + (sv ^ (r & 15))] = stg[j];
    }
  };
  // logits of block i from the products in set i % 2: the block's R x NP
  // floats are contiguous in plogits, one 16-byte vector (4 positions of a
  // row) per thread and step; in the products, row r, position p of column
  // block cb sits at element r % 4 of lanes 16 ((r % 16) / 4) + p % 16 of the
  // waves kw NB + cb, row block r / 16
  auto store_logits = [&](int i) {
    constexpr int NV = R * NP / 4;                          // vectors per block
    const float* rs = red + (i & 1) * red_set;
    const int v0 = (b_beg + i) * R;
#pragma unroll
    for (int j = 0; j < (NV + kKsWaves * kWave - 1) / (kKsWaves * kWave); ++j) {
      const int x = j * kKsWaves * kWave + t;
      const int r = x / (NP / 4), p = 4 * (x % (NP / 4));
      if (x < NV && v0 + r < V) {
        const int cbx = p / 16;
        const int off = ((r / 16) * 4 + r % 4) * kWave + 16 * ((r % 16) / 4) + p % 16;
        f32x4 sum = *reinterpret_cast<const f32x4*>(rs + cbx * MB * 4 * kWave + off);
#pragma unroll
        for (int k = 1; k < KW; ++k)
          sum += *reinterpret_cast<const f32x4*>(rs + (k * NB + cbx) * MB * 4 * kWave + off);
        *reinterpret_cast<f32x4*>(plogits + ((size_t)kp * V + v0 + r) * NP + p) = sum;
      }
    }
  };
  const int ar = lane % 16;                                 // operand row within an MFMA block

  load_regs(0);
  store_lds(0);
  __builtin_amdgcn_s_waitcnt(0x0f70);                       // vmcnt(0), as in k_lm_stream
  if (cnt > 1) load_regs(1);
  for (int it = 0; it < cnt; ++it) {
    const int buf = it & 1;
    // block it is in LDS; the products of block it - 1 are complete, and
    // those of block it - 2 (this iteration's set) have been written out
    __syncthreads();
    if (it > 0) store_logits(it - 1);
    const u32x4* bl = reinterpret_cast<const u32x4*>(ks_lds + buf * blk_bytes);
    f32x4 acc[2][MB];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[h][mb][e] = 0.0f;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int sv = kw * (dw / 8) + 4 * c + lane / 16;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, bl[(16 * mb + ar) * vec_part + (sv ^ ar)]);
        acc[c & 1][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, hb[c]),
                                                                 acc[c & 1][mb], 0, 0, 0);
      }
    }
    float* ws_ = red + (it & 1) * red_set + wave * MB * 4 * kWave + lane;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int e = 0; e < 4; ++e) ws_[(mb * 4 + e) * kWave] = acc[0][mb][e] + acc[1][mb][e];
    if (it + 1 < cnt) store_lds(buf ^ 1);
    if (it + 2 < cnt) load_regs(it + 2);
  }
  __syncthreads();
  store_logits(cnt - 1);
}

// Adds the S parts' logits of every candidate position, in part order, and
// folds them: workgroup j takes the vocabulary entries [j chunk, (j+1) chunk);
// thread t takes the 4 positions 4 (t % Q) .. +3 (Q = NP / 4) at every
// (256 / Q)-th entry; the threads of a position are combined in order at the
// end, one partial per (position, workgroup) for k_lm_finish.
template <int S>
__global__ void __launch_bounds__(256)
k_lm_ksum(const float* __restrict__ plogits, const int32_t* __restrict__ count, int V, int chunk,
          WavePartial* __restrict__ partials, int n_split) {
  constexpr int NP = kLsRows * S, Q = NP / 4, VS = 256 / Q;
  __shared__ WavePartial xs[VS][NP];
  const int t = threadIdx.x, q = t % Q, vs = t / Q;
  const int n = *count;
  if (n == 0) return;
  const int v0 = blockIdx.x * chunk, v1 = min(V, v0 + chunk);
  LmState st[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) st[e] = LmState{kNegInf, kRefFloor, 0.0, 0x7fffffff};
  for (int v = v0 + vs; v < v1; v += VS) {
    f32x4 x = *reinterpret_cast<const f32x4*>(plogits + (size_t)v * NP + 4 * q);
#pragma unroll
    for (int k = 1; k < S; ++k) x += *reinterpret_cast<const f32x4*>(plogits + ((size_t)k * V + v) * NP + 4 * q);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (x[e] > st[e].M) {
        const float Kn = exp_ref(x[e]);
        st[e].S = rescale(st[e].S, st[e].K, Kn);
        st[e].K = Kn;
        st[e].M = x[e];
        st[e].first = v;
      }
      st[e].S += (double)term(x[e], st[e].K);
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) xs[vs][4 * q + e] = WavePartial{st[e].M, st[e].K, st[e].S, st[e].first};
  __syncthreads();
  if (t < n) {
    LmState c = {xs[0][t].m, xs[0][t].K, xs[0][t].S, xs[0][t].first};
#pragma unroll
    for (int r = 1; r < VS; ++r) lm_combine(c, xs[r][t].m, xs[r][t].K, xs[r][t].S, xs[r][t].first);
    partials[(size_t)t * n_split + blockIdx.x] = WavePartial{c.M, c.K, c.S, c.first};
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

// Parts of the hidden dimension for the streaming kernels: 1 (k_lm_stream)
// up to kLsRows positions, 2 (k_lm_kstream) up to 2 kLsRows, when
// a block is a whole number of 16-byte loads per thread and each wave's share
// of the hidden operands fits its registers; 0: the tiled kernel.
static int lm_kparts(long long n, int d) {
  if (d > kLsMaxD) return 0;
  if (n <= kLsRows) return d % 512 == 0 ? 1 : 0;
  if (n <= 2 * kLsRows) return d % 1024 == 0 ? 2 : 0;
  return 0;
}

// the streaming kernel for d = 512 DM
typedef void (*LmStreamFn)(const uint16_t*, const uint16_t*, const uint8_t*, const int32_t*,
                           const int32_t*, int, int, int, int32_t*, int32_t*, RowOut, WavePartial*,
                           int);
static const LmStreamFn kLmStream[kLsMaxD / 512] = {
    k_lm_stream<1>, k_lm_stream<2>, k_lm_stream<3>, k_lm_stream<4>,
    k_lm_stream<5>, k_lm_stream<6>, k_lm_stream<7>, k_lm_stream<8>};

// the k-split kernel (S = 2) for d = 1024 i
typedef void (*LmKStreamFn)(const uint16_t*, const uint16_t*, const uint8_t*, const int32_t*,
                            const int32_t*, int, int, int, int32_t*, int32_t*, RowOut, float*);
static const LmKStreamFn kLmKStream2[kLsMaxD / 1024] = {
    k_lm_kstream<2, 2>, k_lm_kstream<4, 2>, k_lm_kstream<6, 2>, k_lm_kstream<8, 2>};
constexpr int kKsSplits = 512;     // k_lm_ksum workgroups (vocabulary chunks)

struct LmPlan {
  int small;     // parts of the hidden dimension: 1 k_lm_stream, 2 k_lm_kstream; 0 tiled
  int groups;    // k_lm_kstream: row-range groups (S groups workgroups)
  int chunk;     // k_lm_ksum: vocabulary entries per workgroup
  size_t off_plogits;
  int m_tiles, n_tiles, n_split, tiles_per_split;
  size_t off_rows, off_partials, off_out, bytes;
};

// Row tiles cover the upper bound B*L (tiles past the device-side count exit
// at once); the vocabulary is split so that about 512 workgroups run.
static LmPlan lm_plan(int B, int L, int d, int V, bool need_out) {
  LmPlan p{};
  const long long n = (long long)B * L;
  const int S = lm_kparts(n, d);
  if (S == 1) {
    // one workgroup per compute unit, each a contiguous range of row blocks
    p.small = 1;
    const int nblk = (V + kLsBlk - 1) / kLsBlk;
    p.n_split = nblk < kLmCUs ? nblk : kLmCUs;
    p.off_rows = 256;
    p.off_partials = p.off_rows + align256((size_t)n * 4);
    p.off_out = p.off_partials + align256((size_t)n * p.n_split * sizeof(WavePartial));
    p.bytes = p.off_out + (need_out ? 3 * align256((size_t)n * 4) : 0);
    return p;
  }
  if (S > 1) {
    // S workgroups (one per part) per row range, one workgroup per compute
    // unit; the parts' logits of all 32 S positions in the workspace
    p.small = S;
    const int nblk = (V + 8 * S - 1) / (8 * S);
    p.groups = nblk < kLmCUs / S ? nblk : kLmCUs / S;
    p.chunk = (V + kKsSplits - 1) / kKsSplits;
    p.n_split = (V + p.chunk - 1) / p.chunk;
    p.off_rows = 256;
    p.off_partials = p.off_rows + align256((size_t)n * 4);
    p.off_plogits = p.off_partials + align256((size_t)n * p.n_split * sizeof(WavePartial));
    p.off_out = p.off_plogits + align256((size_t)S * V * kLsRows * S * sizeof(float));
    p.bytes = p.off_out + (need_out ? 3 * align256((size_t)n * 4) : 0);
    return p;
  }
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

// The streaming and tiled kernels' dynamic LDS (up to 160 KiB) is above the
// default limit; the limit is raised once per device, before the first launch
// there.
constexpr int kLmMaxDevices = 64;
static std::atomic<bool> lm_lds_allowed[kLmMaxDevices];

static hipError_t lm_allow_lds() {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < kLmMaxDevices && lm_lds_allowed[dev].load(std::memory_order_acquire))
    return hipSuccess;
  hipError_t a = hipFuncSetAttribute((const void*)k_lm_partial,
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLmLdsBytes);
  for (int i = 0; i < kLsMaxD / 512 && a == hipSuccess; ++i)
    a = hipFuncSetAttribute((const void*)kLmStream[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)kLsLdsBytes(512 * (i + 1)));
  for (int i = 0; i < kLsMaxD / 1024 && a == hipSuccess; ++i)
    a = hipFuncSetAttribute((const void*)kLmKStream2[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)ks_lds_bytes<2>(1024 * (i + 1)));
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
  if (p.small > 1) {
    // the k-split kernel compacts the candidates itself
    const uint16_t* h = (const uint16_t*)hidden;
    const uint16_t* w = (const uint16_t*)weight;
    float* plog = (float*)(ws + p.off_plogits);
    const dim3 grid((unsigned)(p.groups * 2)), block(kKsWaves * kWave);
    hipLaunchKernelGGL(kLmKStream2[d / 1024 - 1], grid, block, ks_lds_bytes<2>(d), st, h, w, mask, bs,
                       be, B, L, V, rows, count, out, plog);
    hipLaunchKernelGGL(k_lm_ksum<2>, dim3((unsigned)p.n_split), dim3(256), 0, st, plog, count, V,
                       p.chunk, part, p.n_split);
  } else if (p.small) {
    // the streaming kernel compacts the candidates itself
    hipLaunchKernelGGL(kLmStream[d / 512 - 1], dim3((unsigned)p.n_split), dim3(kLsWaves * kWave),
                       kLsLdsBytes(d), st, (const uint16_t*)hidden, (const uint16_t*)weight, mask,
                       bs, be, B, L, V, rows, count, out, part, p.n_split);
  } else {
    hipLaunchKernelGGL(k_lm_zero, dim3(1), dim3(64), 0, st, count);
    hipLaunchKernelGGL(k_lm_compact, dim3((unsigned)((B + 3) / 4)), dim3(256), 0, st, mask, bs, be,
                       B, L, rows, count, out);
    hipLaunchKernelGGL(k_lm_partial, dim3((unsigned)p.m_tiles, (unsigned)p.n_split),
                       dim3(kLmThreads), kLmLdsBytes, st, (const uint16_t*)hidden,
                       (const uint16_t*)weight, rows, count, d, V, p.tiles_per_split,
                       (uint32_t)((size_t)B * L * d * 2), part, p.n_split);
  }
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
  *bytes = lm_plan(B, L, d, V, true).bytes;
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
  const LmPlan p = lm_plan(B, L, d, V, need_out);
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
