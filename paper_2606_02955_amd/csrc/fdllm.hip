// fdllm.hip -- gfx950 kernels and C ABI of the Fast-dLLM++ commit selector.
//
// One decoding step of Frechet profile decoding (arXiv 2606.02955, Alg. 1):
//   (1) vocabulary pass: per candidate position, the greedy token, its softmax
//       confidence c, the complement eps = 1 - c and the log-sum-exp
//       (Sec. 3 "Notation"); every logit of a candidate row is read once;
//   (2) selection: per block, sort the candidates by confidence and
//       apply the Frechet profile / factor / threshold rule (Sec. 3
//       "Frechet profile quantities", Sec. 2, Sec. 5 "Baselines");
//   (3) reveal: write the chosen tokens into the sequence and clear their mask.
//
// The vocabulary pass is bound by HBM bandwidth: per logit it does one
// exp2, a few VALU ops and no reuse, so there is no dense contraction and
// no MFMA.  Design:
//   * a row is streamed by one wavefront (or split over S wavefronts for
//     small batches) with 16-byte loads; lane l of the wave reads vectors
//     l, l+64, ... so every wave-wide load is 1 KiB contiguous;
//   * loads are grouped in batches of U vectors per lane; for each batch the
//     lane first takes the batch maximum (v_max3), then adds
//     2^(x*log2e - K) for every element into a double accumulator.  K is an
//     integer-valued float, K = ceil(m * log2e) for the running maximum m,
//     so rescaling the accumulator when m grows is an exact ldexp.  No sum
//     ever holds the greedy element: the batch in which a lane's maximum
//     appeared is summed apart and, at the row end, again without one
//     element equal to that maximum, and stretches of a row are merged by
//     letting all but one holder of the row maximum put their own maximum's
//     term back; so s' = sum_{v != t} exp(l_v - M) is formed with no
//     subtraction and eps keeps its relative accuracy when c -> 1;
//   * the argmax is tracked per batch: each lane keeps, in LDS, the batch
//     in which its maximum first appeared; at the end, lanes holding
//     the row maximum scan that batch for the lowest index, then a wave
//     minimum gives the lowest index of the whole row;
//   * wavefront reductions use DPP row operations, ds_swizzle and
//     v_readlane; partials of a split row meet in LDS in fixed order, so
//     results do not depend on scheduling.
// A block of up to 64 positions is selected in one wavefront: a 64-lane
// bitonic sort of (eps, slot) keys, a double-precision prefix scan of the
// heterogeneity bonus, a ballot for n*, and ds_permute to route each decision
// back to its position.  Longer blocks (up to 1024 positions) sort the same
// keys in LDS across a workgroup with a fixed-order scan.  The
// calibration-robust rule (the appendix on calibration-robust certificates)
// is the profile rule on eps_low = min(1, eps + eta).
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include <mutex>

#include "fdllm.h"
#include "pass_common.h"

// Tile parameters (compile-time): vectors per lane per batch, and waves per
// workgroup of the fused kernel.
#ifndef FDLLM_FUSED_WAVES
#define FDLLM_FUSED_WAVES 8
#endif
#ifndef FDLLM_U_BF16
#define FDLLM_U_BF16 4
#endif
#ifndef FDLLM_U_F32
#define FDLLM_U_F32 4
#endif
#ifndef FDLLM_U_SPLIT_BF16
#define FDLLM_U_SPLIT_BF16 2   // bf16 rows split over several waves: shorter parts, fewer registers
#endif
#ifndef FDLLM_TARGET_WAVES
#define FDLLM_TARGET_WAVES 16384  // small batches: split rows until about this many waves stream
#endif
#ifndef FDLLM_FUSED_MIN_B
#define FDLLM_FUSED_MIN_B 256     // batches from this size run one workgroup per sequence
#endif
#ifndef FDLLM_GROUPS32_MIN_B
#define FDLLM_GROUPS32_MIN_B 8    // small batches from this size: 32 row groups per sequence, not 64
#endif
#ifndef FDLLM_HYBRID_MAX_REM
#define FDLLM_HYBRID_MAX_REM 64   // sequences beyond a multiple of the CU count run on a side stream
#endif
#ifndef FDLLM_WAVES_PER_EU
#define FDLLM_WAVES_PER_EU 0   // minimum waves per SIMD the fused kernel is compiled for (0: no hint)
#endif

namespace fdllm {
// Row groups per sequence of the split pass (window positions q, q + W, ...
// of a row group): 64, one wavefront's block, for the fewest sequences,
// where a wider window's rows should all stream at once; 32, the paper's
// block, from FDLLM_GROUPS32_MIN_B sequences, where the grid is half as
// large and a 64-wide window's second row per group still finds the chip
// busy; never more than the span.
constexpr int kGroups32MinB = FDLLM_GROUPS32_MIN_B;
__host__ __device__ inline int row_groups(int B, int L) {
  const int g = B >= kGroups32MinB ? 32 : 64;
  return L < g ? L : g;
}

// ---------------------------------------------------------------------------
// vector formats: one lane loads 16 bytes (or one element on the scalar path)
// ---------------------------------------------------------------------------
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// bit pattern of FDLLM_MAX_ABS_LOGIT as a float; for finite and non-finite
// values alike, |x| > bound  <=>  (bits(x) & 0x7FFFFFFF) > kBoundBits
constexpr unsigned kBoundBits = 0x4B189680u;   // 1.0e7f
static_assert(__builtin_bit_cast(unsigned, FDLLM_MAX_ABS_LOGIT) == kBoundBits, "logit bound bits");
__device__ __forceinline__ bool bad_bits(unsigned f32bits) { return (f32bits & 0x7FFFFFFFu) > kBoundBits; }

struct VecBf16x8 {
  static constexpr int kElems = 8;
  static constexpr int kU = FDLLM_U_BF16;   // vectors per lane per batch
  static constexpr int kUSplit = FDLLM_U_SPLIT_BF16;   // the same, rows split over waves
  using Raw = u32x4;
  __device__ static Raw pad() { return Raw{0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u, 0xFF80FF80u}; }
  __device__ static void unpack(const Raw& r, float (&x)[kElems]) {
    x[0] = __uint_as_float(r.x << 16); x[1] = __uint_as_float(r.x & 0xFFFF0000u);
    x[2] = __uint_as_float(r.y << 16); x[3] = __uint_as_float(r.y & 0xFFFF0000u);
    x[4] = __uint_as_float(r.z << 16); x[5] = __uint_as_float(r.z & 0xFFFF0000u);
    x[6] = __uint_as_float(r.w << 16); x[7] = __uint_as_float(r.w & 0xFFFF0000u);
  }
  __device__ static bool bad(const Raw& r) {
    return bad_bits(r.x << 16) | bad_bits(r.x & 0xFFFF0000u) | bad_bits(r.y << 16) |
           bad_bits(r.y & 0xFFFF0000u) | bad_bits(r.z << 16) | bad_bits(r.z & 0xFFFF0000u) |
           bad_bits(r.w << 16) | bad_bits(r.w & 0xFFFF0000u);
  }
};
struct VecF32x4 {
  static constexpr int kElems = 4;
  static constexpr int kU = FDLLM_U_F32;
  static constexpr int kUSplit = FDLLM_U_F32;
  using Raw = u32x4;
  __device__ static Raw pad() { return Raw{0xFF800000u, 0xFF800000u, 0xFF800000u, 0xFF800000u}; }
  __device__ static void unpack(const Raw& r, float (&x)[kElems]) {
    x[0] = __uint_as_float(r.x); x[1] = __uint_as_float(r.y);
    x[2] = __uint_as_float(r.z); x[3] = __uint_as_float(r.w);
  }
  __device__ static bool bad(const Raw& r) {
    return bad_bits(r.x) | bad_bits(r.y) | bad_bits(r.z) | bad_bits(r.w);
  }
};
struct VecBf16x1 {
  static constexpr int kElems = 1;
  static constexpr int kU = 8;
  static constexpr int kUSplit = 8;
  using Raw = unsigned short;
  __device__ static Raw pad() { return (unsigned short)0xFF80u; }
  __device__ static void unpack(const Raw& r, float (&x)[kElems]) { x[0] = __uint_as_float((unsigned)r << 16); }
  __device__ static bool bad(const Raw& r) { return bad_bits((unsigned)r << 16); }
};
struct VecF32x1 {
  static constexpr int kElems = 1;
  static constexpr int kU = 8;
  static constexpr int kUSplit = 8;
  using Raw = unsigned int;
  __device__ static Raw pad() { return 0xFF800000u; }
  __device__ static void unpack(const Raw& r, float (&x)[kElems]) { x[0] = __uint_as_float(r); }
  __device__ static bool bad(const Raw& r) { return bad_bits(r); }
};

template <class Raw>
__device__ __forceinline__ Raw load_stream(const Raw* p) {
  return __builtin_nontemporal_load(p);
}

// ---------------------------------------------------------------------------
// vocabulary pass over one wave's share of a row
// ---------------------------------------------------------------------------

constexpr int kAcc = 4;   // independent double accumulators per lane

// The wave handles wave-loads k = w, w+S, w+2S, ... of the row (a wave-load
// is 64 consecutive vectors); lane l reads vector k*64 + l.
template <class Vec, int U, int S>
__device__ __forceinline__ WavePartial row_pass(const typename Vec::Raw* __restrict__ row, int nvec, int w,
                                                typename Vec::Raw* __restrict__ kept) {
  using Raw = typename Vec::Raw;
  constexpr int E = Vec::kElems;
  const int lane = lane_id();
  const int nwl = (nvec + kWave - 1) / kWave;          // wave-loads in the row
  const int nfull = nvec / kWave;                       // wave-loads with no padding
  const int nj = nwl > w ? (nwl - w + S - 1) / S : 0;   // this wave's wave-loads
  const int njf = nfull > w ? (nfull - w + S - 1) / S : 0;
  const Raw* p = row + w * kWave + lane;
  constexpr int kStride = S * kWave;

  float m = kNegInf;
  float K = kRefFloor;
  // acc: the terms of every batch but the kept one (below); pend: the kept
  // batch's terms, dropped at the end, where the kept batch is summed again
  // without one element equal to m (so no sum ever holds the lane maximum)
  double acc = 0.0, pend = 0.0;
  // the batch in which this lane's maximum first appeared, and its vectors,
  // kept in this wave's LDS area `kept` (2 U kWave vectors): every batch is
  // written there, a lane whose maximum grows into slot 0 (u kWave + lane),
  // the others into slot 1, so no per-lane select is needed; the lowest index
  // of the row maximum is found there at the end (a re-read from memory
  // would cost a dependent HBM latency per row)
  int rec = -1;

  // sum of a batch's terms: kAcc accumulators, each started from its first
  // term (as 0 + t would give, without the add), then a fixed pairing
  static_assert(U * E >= kAcc, "a batch fills every accumulator");
  auto batch_sum = [&](const float (&x)[U][E]) {
    double t[kAcc];
#pragma unroll
    for (int a = 0; a < kAcc; ++a) t[a] = (double)term(x[a / E][a % E], K);
#pragma unroll
    for (int i = kAcc; i < U * E; ++i) t[i % kAcc] += (double)term(x[i / E][i % E], K);
    return (t[0] + t[1]) + (t[2] + t[3]);
  };

  auto consume = [&](const Raw (&r)[U], int batch) {
    float x[U][E];
#pragma unroll
    for (int u = 0; u < U; ++u) Vec::unpack(r[u], x[u]);
    float bm = kNegInf;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int e = 0; e < E; ++e) bm = fmaxf(bm, x[u][e]);
    const bool grows = bm > m;
    rec = grows ? batch : rec;
    Raw* const dst = kept + (grows ? 0 : U * kWave) + lane;
#pragma unroll
    for (int u = 0; u < U; ++u) dst[u * kWave] = r[u];
    const float mn = fmaxf(m, bm);
    // a lane that has only seen padding keeps a finite reference, so that
    // padding terms are exp2(-inf) = 0 rather than exp2(-inf + inf)
    const float Kn = fmaxf(exp_ref(mn), kRefFloor);
    acc = rescale(acc, K, Kn);
    pend = rescale(pend, K, Kn);
    m = mn;
    K = Kn;
    const double bs = batch_sum(x);
    // a new kept batch sends the previous one's terms to acc
    acc += grows ? pend : bs;
    pend = grows ? bs : pend;
  };

  // Batches of U wave-loads; the first nbf are whole (no lane past the row
  // end).  In the steady state the loads of batch jb+1 are issued before
  // batch jb is consumed, unconditionally, so each wave keeps a batch of
  // 16-byte loads in flight while it computes.  The last, partial batch is
  // loaded with per-lane predicates after the pipeline drains.
  const int nb = (nj + U - 1) / U;
  const int nbf = njf / U;
  auto load_full = [&](Raw (&r)[U], int jb) {
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = load_stream(p + (jb * U + u) * kStride);
  };
  auto load_part = [&](Raw (&r)[U], int jb) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = jb * U + u;
      const int v = (w + j * S) * kWave + lane;
      r[u] = (j < nj && v < nvec) ? load_stream(p + j * kStride) : Vec::pad();
    }
  };
  Raw ra[U], rb[U];
  int jb = 0;
  if (nbf > 0) {
    load_full(ra, 0);
    for (; jb + 2 < nbf; jb += 2) {
      load_full(rb, jb + 1);
      consume(ra, jb);
      load_full(ra, jb + 2);
      consume(rb, jb + 1);
    }
    if (jb + 1 < nbf) {
      load_full(rb, jb + 1);
      consume(ra, jb);
      consume(rb, jb + 1);
      jb += 2;
    } else {
      consume(ra, jb);
      jb += 1;
    }
  }
  for (; jb < nb; ++jb) {
    load_part(ra, jb);
    consume(ra, jb);
  }

  // the kept batch again, without one element equal to the lane maximum
  // (padding is -inf: its terms are 0)
  Raw keep[U];
#pragma unroll
  for (int u = 0; u < U; ++u) keep[u] = rec >= 0 ? kept[u * kWave + lane] : Vec::pad();
  double s = acc;
  if (rec >= 0) {
    bool left_out = false;
    double t[kAcc];
#pragma unroll
    for (int a = 0; a < kAcc; ++a) t[a] = 0.0;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float x[E];
      Vec::unpack(keep[u], x);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const bool skip = !left_out && x[e] == m;
        left_out = left_out || skip;
        t[(u * E + e) % kAcc] += skip ? 0.0 : (double)term(x[e], K);
      }
    }
    s += (t[0] + t[1]) + (t[2] + t[3]);
  }

  WavePartial out;
  // across lanes: the wave maximum M and its reference, then every lane but
  // the lowest one holding M puts its own maximum's term back, and a fixed
  // butterfly sums (bitwise equal in every lane)
  out.m = wave_max(m);
  out.K = fmaxf(exp_ref(out.m), kRefFloor);
  const unsigned long long holders = __ballot(m == out.m);
  const bool owner = lane == (int)__builtin_ctzll(holders);
  double v = rescale(s, K, out.K);
  if (!owner) v += rescale((double)term(m, K), K, out.K);
  out.S = wave_sum_f64(v);
  // lowest index of the maximum: lanes holding it scan their kept batch
  int first = 0x7fffffff;
  if (m == out.m && rec >= 0) {
#pragma unroll
    for (int u = U - 1; u >= 0; --u) {
      const int j = rec * U + u;
      const int v = (w + j * S) * kWave + lane;
      if (j < nj && v < nvec) {
        float x[E];
        Vec::unpack(keep[u], x);
#pragma unroll
        for (int e = E - 1; e >= 0; --e)
          if (x[e] == out.m) first = v * E + e;
      }
    }
  }
  out.first = wave_min(first);
  return out;
}

// ---------------------------------------------------------------------------
// kernel: vocabulary pass, S wavefronts per row, rows of all B*L slots
// ---------------------------------------------------------------------------
template <int S>
struct SplitShape {
  static constexpr int kWaves = S < 4 ? 4 : S;      // waves per workgroup
  static constexpr int kRows = kWaves / S;          // rows per workgroup
  static constexpr int kThreads = kWaves * kWave;
};

// A row's S wave partials combined: the row maximum M and its reference,
// every part but the lowest-index one holding M puts its own maximum's term
// back, and the parts' sums add up by a fixed binary tree -- pairs (0,1),
// (2,3), ..., then pairs of pairs -- in one of two forms that give the same
// bits: a wavefront whose lanes q < S hold part q (a butterfly over the
// lanes, used where a row's parts meet in one workgroup) and one thread
// holding all S parts (the selection kernels reading parts from the
// workspace; every part's load is issued at once).
template <int S>
__device__ __forceinline__ RowResult combine_parts_lanes(const WavePartial& mine) {
  const int lane = lane_id();
  float M = mine.m;
  if constexpr (S >= 2) M = fmaxf(M, partner_f32<0>(M));
  if constexpr (S >= 4) M = fmaxf(M, partner_f32<1>(M));
  if constexpr (S >= 8) M = fmaxf(M, partner_f32<2>(M));
  if constexpr (S >= 16) M = fmaxf(M, partner_f32<3>(M));
  const float K = fmaxf(exp_ref(M), kRefFloor);
  const unsigned long long group = (S >= 64 ? ~0ull : ((1ull << S) - 1ull)) << (lane / S * S);
  const unsigned long long holders = __ballot(mine.m == M) & group;
  const bool owner = lane == (int)__builtin_ctzll(holders);
  double v = rescale(mine.S, mine.K, K);
  if (!owner) v += rescale((double)term(mine.m, mine.K), mine.K, K);
  if constexpr (S >= 2) v += partner_f64<0>(v);
  if constexpr (S >= 4) v += partner_f64<1>(v);
  if constexpr (S >= 8) v += partner_f64<2>(v);
  if constexpr (S >= 16) v += partner_f64<3>(v);
  int f = mine.m == M ? mine.first : 0x7fffffff;   // lowest index among the parts holding M
  if constexpr (S >= 2) f = min(f, partner_i32<0>(f));
  if constexpr (S >= 4) f = min(f, partner_i32<1>(f));
  if constexpr (S >= 8) f = min(f, partner_i32<2>(f));
  if constexpr (S >= 16) f = min(f, partner_i32<3>(f));
  return finish_row_x(M, K, v, f);
}

template <int S>
__device__ __forceinline__ RowResult combine_parts_regs(const WavePartial (&p)[S]) {
  float M = p[0].m;
#pragma unroll
  for (int q = 1; q < S; ++q) M = fmaxf(M, p[q].m);
  const float K = fmaxf(exp_ref(M), kRefFloor);
  int owner = S;
#pragma unroll
  for (int q = S - 1; q >= 0; --q)
    if (p[q].m == M) owner = q;
  double v[S];
#pragma unroll
  for (int q = 0; q < S; ++q) {
    v[q] = rescale(p[q].S, p[q].K, K);
    if (q != owner) v[q] += rescale((double)term(p[q].m, p[q].K), p[q].K, K);
  }
#pragma unroll
  for (int width = 1; width < S; width <<= 1)
#pragma unroll
    for (int q = 0; q < S; q += 2 * width) v[q] += v[q + width];
  int first = 0x7fffffff;
#pragma unroll
  for (int q = 0; q < S; ++q)
    if (p[q].m == M) first = min(first, p[q].first);
  return finish_row_x(M, K, v[0], first);
}

template <int S>
__device__ __forceinline__ RowResult combine_parts(const WavePartial* part) {
  WavePartial p[S];
#pragma unroll
  for (int q = 0; q < S; ++q) p[q] = part[q];
  return combine_parts_regs<S>(p);
}

// Row group r of the grid handles the window-relative slot (b, q), q < W =
// row_groups(B, L): the window positions q, q + W, ... of sequence b (one for a
// window of at most W positions), and the defaults of the positions j = q,
// q + W, ... of the whole row of L slots that lie outside the window.  So
// only B W row groups are launched, however long the span L.
template <class Vec, int U, int S>
__global__ void __launch_bounds__(SplitShape<S>::kThreads)
k_confidence(const typename Vec::Raw* __restrict__ logits, int B, int L, int nvec,
             const uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
             const int32_t* __restrict__ bend, RowOut out) {
  using Shape = SplitShape<S>;
  __shared__ WavePartial part[Shape::kWaves];
  __shared__ typename Vec::Raw s_kept[2 * U * Shape::kThreads];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const int rloc = wave / S;
  const int w = wave % S;
  const int W = row_groups(B, L);
  // row group index: a launch holds fewer than 2^32 work-items, so fewer
  // than 2^26 workgroups of at least 64 threads and two row groups at most
  // each: 32-bit division
  const unsigned vs = blockIdx.x * (unsigned)Shape::kRows + (unsigned)rloc;
  const bool live = (unsigned long long)vs < (unsigned long long)B * (unsigned long long)W;
  int b = 0, q = 0, s = 0, len = 0;
  if (live) {
    b = (int)(vs / (unsigned)W);
    q = (int)(vs % (unsigned)W);
    const int s0 = bstart[b], e0 = bend[b];
    if (window_ok(s0, e0, L)) {
      s = s0;
      len = e0 - s0;
    }
  }
  const size_t row0 = (size_t)b * L;
  // defaults of this row group's positions outside the window, one per lane
  if (live && w == 0)
    for (int j = q + lane * W; j < L; j += W * kWave)
      if (j < s || j >= s + len) store_default(out, row0 + j);
  // trips over the window; where row groups of one workgroup meet barriers
  // (S = 2: two row groups), a count that depends on L only
  const int trips = (S == 1 || Shape::kRows == 1) ? (len - q + W - 1) / W : (L + W - 1) / W;
  for (int it = 0; it < trips; ++it) {
    const int rel = q + it * W;
    const bool inwin = live && rel < len;
    const size_t slot = row0 + (size_t)(s + rel);
    const bool cand = inwin && mask[slot] != 0;
    WavePartial wp{};
    if (cand) wp = row_pass<Vec, U, S>(logits + (long long)slot * nvec, nvec, w, s_kept + wave * 2 * U * kWave);
    if constexpr (S > 1) {
      if (lane == 0) part[wave] = wp;
      __syncthreads();
      if (w == 0 && cand) {
        // the row group's first wave merges the S parts across its lanes
        const WavePartial mine = lane < S ? part[rloc * S + lane]
                                          : WavePartial{kNegInf, kRefFloor, 0.0, 0x7fffffff};
        const RowResult rr = combine_parts_lanes<S>(mine);
        if (lane == 0) store_row(out, slot, rr);
      }
      if (w == 0 && lane == 0 && inwin && !cand) store_default(out, slot);
      __syncthreads();   // part[] is written again by the next trip
    } else if (lane == 0 && inwin) {
      if (!cand)
        store_default(out, slot);
      else
        store_row(out, slot, finish_row_x(wp.m, wp.K, wp.S, wp.first));
    }
  }
}

// The same pass with a row's S parts spread over S / 4 workgroups of 4 waves
// (more CUs stream the few rows of a small batch); each wave's partial goes
// to parts[slot][w], combined by the select kernel.  Non-candidates get their
// defaults here.
template <class Vec, int U, int S>
__global__ void __launch_bounds__(256)
k_confidence_parts(const typename Vec::Raw* __restrict__ logits, int B, int L, int nvec,
                   const uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
                   const int32_t* __restrict__ bend, RowOut out, WavePartial* __restrict__ parts) {
  constexpr int P = S / 4;                                  // workgroups per slot
  __shared__ typename Vec::Raw s_kept[2 * U * 256];
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const long long slot = blockIdx.x / P;
  const int w = (int)(blockIdx.x % P) * 4 + wave;           // part of the row
  const int b = (int)(slot / L), i = (int)(slot % L);
  // the mask byte and the bounds are read together (one round trip)
  const bool masked = mask[slot] != 0;
  const int s = bstart[b], e = bend[b];
  const bool cand = masked & window_ok(s, e, L) & (i >= s) & (i < e);
  if (!cand) {
    if (w == 0 && lane == 0) store_default(out, (size_t)slot);
    return;
  }
  const WavePartial wp = row_pass<Vec, U, S>(logits + slot * (long long)nvec, nvec, w, s_kept + wave * 2 * U * kWave);
  if (lane == 0) parts[slot * S + w] = wp;
}

// ---------------------------------------------------------------------------
// selection in one wavefront
// ---------------------------------------------------------------------------

__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int mask) {
  int lo = __shfl_xor((int)(v & 0xffffffffull), mask);
  int hi = __shfl_xor((int)(v >> 32), mask);
  return ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo;
}

// Ascending bitonic sort of one 64-bit key per lane.
__device__ __forceinline__ unsigned long long wave_sort(unsigned long long key, int lane) {
#pragma unroll
  for (int k = 2; k <= kWave; k <<= 1) {
#pragma unroll
    for (int j = k >> 1; j > 0; j >>= 1) {
      const unsigned long long o = shfl_xor_u64(key, j);
      const bool up = (lane & k) == 0;
      const bool low = (lane & j) == 0;
      const unsigned long long lo = key < o ? key : o;
      const unsigned long long hi = key < o ? o : key;
      key = (low == up) ? lo : hi;
    }
  }
  return key;
}

__device__ __forceinline__ double shfl_up_f64(double v, int d) {
  long long b = __double_as_longlong(v);
  int lo = __shfl_up((int)(b & 0xffffffffll), d);
  int hi = __shfl_up((int)(b >> 32), d);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double shfl_f64(double v, int src) {
  long long b = __double_as_longlong(v);
  int lo = __shfl((int)(b & 0xffffffffll), src);
  int hi = __shfl((int)(b >> 32), src);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// Inclusive prefix sum across the wave, fixed order.
__device__ __forceinline__ double wave_scan_f64(double v, int lane) {
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const double o = shfl_up_f64(v, d);
    if (lane >= d) v += o;
  }
  return v;
}

// Sort key of a candidate: [invalid:1][bits(e) >> 9 : 53][slot:10].  e is in
// [0, 1], so bits(e) < 2^62; dropping 9 of the 52 mantissa bits keeps every
// float32-derived value exact (ties below 2^-43 relative fall to the slot).
constexpr unsigned long long kSlotMask = 1023ull;
__device__ __forceinline__ unsigned long long sort_key(bool valid, double e, int slot) {
  const unsigned long long eb = (unsigned long long)__double_as_longlong(e);
  return ((unsigned long long)(valid ? 0u : 1u) << 63) | ((eb >> 9) << 10) | (unsigned)slot;
}

// Decides the commit set of one block.  Lane j describes slot j of the block
// (position start + j): `valid` marks a candidate, `e` is its complement
// eps = 1 - c in double (the order is by e ascending, i.e. confidence
// descending, ties to the lower position) and `conf` its confidence (used by
// the threshold rule only).  Returns n* (the number of commits) and sets
// `commit_slot` for lane j's own slot.
template <int R>
__device__ int select_wave(bool valid, double e, float conf, float param, bool& commit_slot) {
  const int lane = lane_id();
  const unsigned long long vmask = __ballot(valid);
  const int m = __popcll(vmask);
  const unsigned long long sk = wave_sort(sort_key(valid, e, lane), lane);
  const int rank_slot = (int)(sk & kSlotMask);   // slot held by sorted rank `lane`
  const bool rvalid = lane < m;
  bool take;
  int nstar;
  if constexpr (R == kThreshold) {
    const float c = __shfl(conf, rank_slot);
    const bool pass = rvalid && c >= param;
    const unsigned long long pm = __ballot(pass);
    if (pm != 0ull) {
      take = pass;
      nstar = __popcll(pm);
    } else {
      take = rvalid && lane == 0;
      nstar = m > 0 ? 1 : 0;
    }
  } else {
    const double es = shfl_f64(e, rank_slot);               // eps_(n), n = lane + 1
    const double ep = shfl_up_f64(es, 1);
    double lhs = (double)(lane + 2) * es;                   // (n+1) eps_(n)
    if constexpr (R == kProfile) {
      const double t = (rvalid && lane >= 1) ? (double)lane * (es - ep) : 0.0;
      lhs -= wave_scan_f64(t, lane);                        // minus B_n
    }
    const bool acc = rvalid && lhs < (double)param;
    const unsigned long long am = __ballot(acc);
    nstar = am ? 64 - __clzll((long long)am) : (m > 0 ? 1 : 0);
    take = lane < nstar;
  }
  // route rank decisions back to slots (rank_slot is a permutation of 0..63)
  const int routed = __builtin_amdgcn_ds_permute(rank_slot * 4, take ? 1 : 0);
  commit_slot = routed != 0;
  return nstar;
}


// ---------------------------------------------------------------------------
// selection of one block of up to kMaxBlock candidates by a workgroup
// ---------------------------------------------------------------------------
// Block-size ablations go beyond one wavefront; the same rules are evaluated
// with the keys sorted in LDS (bitonic network over N = 2^k >= len entries)
// and a fixed-order double-precision scan of the heterogeneity bonus.
constexpr int kMaxWaves = 16;          // waves of the largest selecting workgroup
struct WideLds {
  unsigned long long key[kMaxBlock];   // sort keys by slot; after the sort, by rank
  double e[kMaxBlock];                 // eps by slot
  float conf[kMaxBlock];               // confidence by slot
  int tok[kMaxBlock];                  // greedy token by slot (fused kernel)
  int flag[kMaxBlock];                 // commit decision by slot
  double wsum[kMaxWaves];              // per-wave totals of the scan
  int m;                               // number of candidates
  int nstar;
  int count;
};

__device__ __forceinline__ int next_pow2(int v) {
  int n = 1;
  while (n < v) n <<= 1;
  return n;
}

// Requires (then a barrier): key[0, N) for every slot, padding slots invalid;
// e and conf of every candidate slot; m.  Every thread of the NT-thread
// workgroup calls it.  Leaves flag[slot] for every slot in [0, N), returns n*.
// The first kOwners threads own the ranks, so the rounding order of the scan
// depends on N only, not on the workgroup size of the calling kernel.
constexpr int kOwners = 256;

template <int R, int NT>
__device__ int select_wg(WideLds& sh, int N, float param) {
  static_assert(NT % kWave == 0 && NT >= kOwners && NT / kWave <= kMaxWaves, "workgroup shape");
  const int tid = threadIdx.x;
  const int lane = tid % kWave;
  const int wave = tid / kWave;
  for (int k = 2; k <= N; k <<= 1) {            // bitonic sort, ascending
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < (N >> 1); i += NT) {
        const int a = ((i & ~(j - 1)) << 1) | (i & (j - 1));
        const int c = a | j;
        const unsigned long long ka = sh.key[a], kc = sh.key[c];
        if ((ka > kc) == ((a & k) == 0)) {
          sh.key[a] = kc;
          sh.key[c] = ka;
        }
      }
      __syncthreads();
    }
  }
  const int m = sh.m;
  if (tid == 0) {
    sh.nstar = 0;
    sh.count = 0;
  }
  // thread tid < kOwners owns the contiguous ranks [r0, r0 + kpt), the others none
  const int kpt = tid < kOwners ? (N + kOwners - 1) / kOwners : 0;
  const int r0 = tid * kpt;
  int nstar;
  if constexpr (R == kThreshold) {
    int cnt = 0;
    for (int q = 0; q < kpt; ++q) {
      const int r = r0 + q;
      if (r < m && sh.conf[(int)(sh.key[r] & kSlotMask)] >= param) ++cnt;
    }
    __syncthreads();
    if (cnt) atomicAdd(&sh.count, cnt);
    __syncthreads();
    const int total = sh.count;
    for (int q = 0; q < kpt && r0 + q < N; ++q) {
      const int r = r0 + q;
      const int slot = (int)(sh.key[r] & kSlotMask);
      const bool take = total > 0 ? (r < m && sh.conf[slot] >= param) : (r == 0 && m > 0);
      sh.flag[slot] = take ? 1 : 0;
    }
    nstar = total > 0 ? total : (m > 0 ? 1 : 0);
  } else {
    // t_r = r (e_(r) - e_(r-1)) for 0-based rank r >= 1; B at rank r = sum_{r' <= r} t_r'
    double local = 0.0;
    if constexpr (R == kProfile) {
      for (int q = 0; q < kpt; ++q) {
        const int r = r0 + q;
        if (r >= 1 && r < m)
          local += (double)r * (sh.e[(int)(sh.key[r] & kSlotMask)] -
                                sh.e[(int)(sh.key[r - 1] & kSlotMask)]);
      }
    }
    const double incl = wave_scan_f64(local, lane);
    if (lane == kWave - 1) sh.wsum[wave] = incl;
    __syncthreads();
    double b = shfl_up_f64(incl, 1);
    if (lane == 0) b = 0.0;
    for (int w = 0; w < wave; ++w) b += sh.wsum[w];   // terms of all lower ranks
    int best = 0;
    for (int q = 0; q < kpt; ++q) {
      const int r = r0 + q;
      if (r >= m) break;
      const double er = sh.e[(int)(sh.key[r] & kSlotMask)];
      if constexpr (R == kProfile) {
        if (r >= 1) b += (double)r * (er - sh.e[(int)(sh.key[r - 1] & kSlotMask)]);
      }
      const double lhs = (double)(r + 2) * er - (R == kProfile ? b : 0.0);
      if (lhs < (double)param) best = r + 1;
    }
    if (best) atomicMax(&sh.nstar, best);
    __syncthreads();
    nstar = sh.nstar > 0 ? sh.nstar : (m > 0 ? 1 : 0);
    for (int q = 0; q < kpt && r0 + q < N; ++q)
      sh.flag[(int)(sh.key[r0 + q] & kSlotMask)] = r0 + q < nstar ? 1 : 0;
  }
  __syncthreads();
  return nstar;
}


// One wavefront decides a block of len <= 64 slots (lane j = slot j) and
// writes its in-window commit flags, reveal and n_commit.
template <int R, bool Robust>
__device__ __forceinline__ void select_block_wave(const SelectIO& io, size_t row, int b, int s,
                                                  int len, bool ok, float param) {
  const int lane = lane_id();
  const bool inwin = lane < len;
  // every lane issues all of its loads at once (lanes past the window read
  // the row's first slot, in bounds, and discard it; absent arrays are stood
  // in for by conf); the fences keep the loads ahead of the arithmetic
  const size_t i = row + (inwin ? (size_t)(s + lane) : 0);
  const uint8_t mb = io.mask[i];
  const float cv = io.conf[i];
  const float ev = (io.eps ? io.eps : io.conf)[i];
  const int32_t tv = (io.x ? io.tokens : reinterpret_cast<const int32_t*>(io.conf))[i];
  float hv = 0.0f;
  if constexpr (Robust) hv = (io.eta.eta ? io.eta.eta : io.conf)[i];
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  const bool valid = inwin && mb != 0;
  const float c = valid ? cv : 0.0f;
  double e = 1.0;
  if (valid) {
    e = io.eps ? (double)ev : 1.0 - (double)c;   // 1 - c is exact in double
    if constexpr (Robust) e = fmin(1.0, e + fmax((double)(io.eta.eta ? hv : io.eta.uniform), 0.0));
  }
  bool take = false;
  const int nstar = select_wave<R>(valid, e, c, param, take);
  if (io.commit && inwin) io.commit[i] = take ? 1 : 0;
  if (take && io.x) {
    io.x[i] = tv;
    io.mask[i] = 0;
  }
  if (io.n_commit && lane == 0) io.n_commit[b] = ok ? nstar : -1;
}

// Rows of at most 64 positions: one wavefront per block, four blocks per
// workgroup, lane j for position j of the row.  Every load a lane needs
// (bounds, mask, conf / eps / token or the wave partials, eta) is addressed
// by its position alone and issued at once, and the values stay in
// registers from the pass's outputs to the reveal, so the kernel waits on
// memory once.  Candidates are ordered by position exactly as in the
// window-relative form (the slot in the sort key only breaks ties).
// PS > 0: the candidates' per-position outputs are first formed from their
// PS wave partials (k_confidence_parts), each by the lane that selects it.
template <int R, bool Robust, int PS>
__global__ void __launch_bounds__(256) k_select(SelectIO io, int B, int L, float param,
                                                const WavePartial* __restrict__ parts, RowOut out) {
  const int lane = threadIdx.x % kWave;
  const int b = blockIdx.x * 4 + threadIdx.x / kWave;
  if (b >= B) return;
  const size_t row = (size_t)b * L;
  const size_t i = row + (size_t)lane;
  const bool slot = lane < L;
  // every load of the kernel is issued before any of them returns: each lane
  // reads its slot's mask byte, outputs (or wave partials) and eta whether or
  // not the slot turns out to be a candidate, lanes past the row reading the
  // row's first slot (all in bounds; their values are not used)
  const size_t ic = slot ? i : row;
  const int s = io.bstart[b], e_end = io.bend[b];
  const uint8_t mb = io.mask[ic];
  WavePartial p[PS > 0 ? PS : 1];
  float c = 0.0f, ef = 1.0f, h = 0.0f;
  int tok = -1;
  if constexpr (PS > 0) {
#pragma unroll
    for (int q = 0; q < PS; ++q) p[q] = parts[ic * PS + q];
  } else {
    // absent arrays are stood in for by conf (same extent), read and unused
    c = io.conf[ic];
    const float ev = (io.eps ? io.eps : io.conf)[ic];
    const int32_t tv = (io.x ? io.tokens : reinterpret_cast<const int32_t*>(io.conf))[ic];
    ef = io.eps ? ev : 1.0f;
    tok = io.x ? tv : -1;
  }
  if constexpr (Robust) {
    // without per-position eta, a float of conf or of the partials stands in
    const float* stand_in;
    if constexpr (PS > 0)
      stand_in = reinterpret_cast<const float*>(parts);
    else
      stand_in = io.conf;
    const float hv = (io.eta.eta ? io.eta.eta : stand_in)[ic];
    h = io.eta.eta ? hv : io.eta.uniform;
  }
  // all of them issue before anything waits for one: a compiler memory fence
  // keeps the loads above it, a scheduling fence keeps the arithmetic below
  // (neither emits an instruction; each load's wait comes at its first use)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
  const bool m = slot && mb != 0;
  const bool ok = window_ok(s, e_end, L);
  const bool inwin = ok && lane >= s && lane < e_end;
  const bool valid = inwin && m;
  double e = 1.0;
  if constexpr (PS > 0) {
    const RowResult rr = combine_parts_regs<PS>(p);
    if (valid) store_row(out, i, rr);
    c = valid ? rr.conf : 0.0f;
    e = valid ? (double)rr.eps : 1.0;
    tok = rr.token;
  } else {
    const double ev = io.eps ? (double)ef : 1.0 - (double)c;   // 1 - c is exact in double
    e = valid ? ev : 1.0;
    c = valid ? c : 0.0f;
  }
  if constexpr (Robust) e = valid ? fmin(1.0, e + fmax((double)h, 0.0)) : e;
  bool take = false;
  const int nstar = select_wave<R>(valid, e, c, param, take);
  take = take && valid;
  if (io.commit && slot) io.commit[i] = take ? 1 : 0;
  if (take && io.x) {
    io.x[i] = tok;
    io.mask[i] = 0;
  }
  if (io.n_commit && lane == 0) io.n_commit[b] = ok ? nstar : -1;
}

// Rows of more than 64 positions: one workgroup per block; blocks of at most
// 64 candidates still select in one wavefront, larger ones in the workgroup.
template <int R, bool Robust, int NT>
__global__ void __launch_bounds__(NT) k_select_wide(SelectIO io, int B, int L, float param) {
  __shared__ WideLds sh;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  const size_t row = (size_t)b * L;
  const int s = io.bstart[b], e_end = io.bend[b];
  const bool ok = window_ok(s, e_end, L);
  const int len = ok ? e_end - s : 0;
  if (io.commit) {
    for (int q = tid; q < L; q += NT)
      if (q < s || q >= s + len) io.commit[row + q] = 0;
  }
  if (len <= kWave) {
    if (tid < kWave) select_block_wave<R, Robust>(io, row, b, s, len, ok, param);
    return;
  }
  const int N = next_pow2(len);
  if (tid == 0) sh.m = 0;
  __syncthreads();
  int cnt = 0;
  for (int slot = tid; slot < N; slot += NT) {
    const size_t i = row + (size_t)(s + slot);
    const bool valid = slot < len && io.mask[i] != 0;
    double e = 1.0;
    if (valid) {
      const float c = io.conf[i];
      e = cand_eps(io.eps, c, i);
      if constexpr (Robust) e = robust_eps(e, io.eta, i);
      sh.conf[slot] = c;
      sh.e[slot] = e;
      ++cnt;
    }
    sh.key[slot] = sort_key(valid, e, slot);
  }
  if (cnt) atomicAdd(&sh.m, cnt);
  __syncthreads();
  const int nstar = select_wg<R, NT>(sh, N, param);
  for (int slot = tid; slot < len; slot += NT) {
    const size_t i = row + (size_t)(s + slot);
    const bool take = sh.flag[slot] != 0;
    if (io.commit) io.commit[i] = take ? 1 : 0;
    if (take && io.x) {
      io.x[i] = io.tokens[i];
      io.mask[i] = 0;
    }
  }
  if (io.n_commit && tid == 0) io.n_commit[b] = nstar;
}

// ---------------------------------------------------------------------------
// kernel: fused decode step, one workgroup of W waves per sequence
// ---------------------------------------------------------------------------
template <class Vec, int U, int W, int R, bool Robust>
__global__ void __launch_bounds__(W * kWave)
#if FDLLM_WAVES_PER_EU > 0
__attribute__((amdgpu_waves_per_eu(FDLLM_WAVES_PER_EU)))
#endif
k_fused(const typename Vec::Raw* __restrict__ logits, int B, int L, int nvec,
        uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
        const int32_t* __restrict__ bend, int32_t* __restrict__ x, float param, EtaIn eta,
        RowOut out, uint8_t* __restrict__ commit, int32_t* __restrict__ n_commit) {
  __shared__ int s_cand[kWaveBlock];      // candidate slots, compacted
  __shared__ typename Vec::Raw s_kept[2 * U * W * kWave];
  __shared__ int s_tok[kWaveBlock];
  __shared__ float s_conf[kWaveBlock];
  __shared__ float s_eps[kWaveBlock];
  __shared__ int s_m;
  const int b = blockIdx.x;
  const int wave = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  const size_t row0 = (size_t)b * L;
  const int s = bstart[b], e = bend[b];
  const bool ok = window_ok(s, e, L);
  const int len = ok ? e - s : 0;
  if (wave == 0) {
    const bool valid = lane < len && mask[row0 + s + lane] != 0;
    const unsigned long long vm = __ballot(valid);
    const int before = __popcll(vm & ((1ull << lane) - 1ull));
    if (valid) s_cand[before] = lane;
    if (lane == 0) s_m = __popcll(vm);
  }
  // default outputs for every non-candidate row of this sequence
  for (int q = threadIdx.x; q < L; q += W * kWave) {
    const bool inwin = q >= s && q < s + len;
    if (!inwin || mask[row0 + q] == 0) {
      store_default(out, row0 + q);
      if (commit) commit[row0 + q] = 0;
    }
  }
  __syncthreads();
  const int m = s_m;
  for (int c = wave; c < m; c += W) {
    const int slot = s_cand[c];
    const size_t r = row0 + s + slot;
    const WavePartial wp = row_pass<Vec, U, 1>(logits + r * (size_t)nvec, nvec, 0, s_kept + wave * 2 * U * kWave);
    const RowResult rr = finish_row_x(wp.m, wp.K, wp.S, wp.first);
    if (lane == 0) {
      store_row(out, r, rr);
      s_tok[slot] = rr.token;
      s_conf[slot] = rr.conf;
      s_eps[slot] = rr.eps;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  const bool valid = lane < len && mask[row0 + s + lane] != 0;
  double ev = valid ? (double)s_eps[lane] : 1.0;
  if constexpr (Robust) {
    if (valid) ev = robust_eps(ev, eta, row0 + s + lane);
  }
  bool take = false;
  const int nstar = select_wave<R>(valid, ev, valid ? s_conf[lane] : 0.0f, param, take);
  if (valid) {
    if (commit) commit[row0 + s + lane] = take ? 1 : 0;
    if (take) {
      x[row0 + s + lane] = s_tok[lane];
      mask[row0 + s + lane] = 0;
    }
  }
  if (n_commit && lane == 0) n_commit[b] = ok ? nstar : -1;
}

// Fused decode step for rows of more than 64 positions (blocks up to
// kMaxBlock); the vocabulary pass is the same, the selection as in
// k_select_wide.
template <class Vec, int U, int W, int R, bool Robust>
__global__ void __launch_bounds__(W * kWave)
k_fused_wide(const typename Vec::Raw* __restrict__ logits, int B, int L, int nvec,
             uint8_t* __restrict__ mask, const int32_t* __restrict__ bstart,
             const int32_t* __restrict__ bend, int32_t* __restrict__ x, float param, EtaIn eta,
             RowOut out, uint8_t* __restrict__ commit, int32_t* __restrict__ n_commit) {
  constexpr int NT = W * kWave;
  __shared__ WideLds sh;
  __shared__ int s_cand[kMaxBlock];       // candidate slots, compacted
  __shared__ typename Vec::Raw s_kept[2 * U * W * kWave];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int wave = tid / kWave;
  const int lane = tid % kWave;
  const size_t row0 = (size_t)b * L;
  const int s = bstart[b], e = bend[b];
  const bool ok = window_ok(s, e, L);
  const int len = ok ? e - s : 0;
  if (wave == 0) {
    int base = 0;
    for (int c0 = 0; c0 < len; c0 += kWave) {
      const int slot = c0 + lane;
      const bool valid = slot < len && mask[row0 + s + slot] != 0;
      const unsigned long long vm = __ballot(valid);
      if (valid) s_cand[base + __popcll(vm & ((1ull << lane) - 1ull))] = slot;
      base += __popcll(vm);
    }
    if (lane == 0) sh.m = base;
  }
  for (int q = tid; q < L; q += NT) {
    const bool inwin = q >= s && q < s + len;
    if (!inwin || mask[row0 + q] == 0) {
      store_default(out, row0 + q);
      if (commit) commit[row0 + q] = 0;
    }
  }
  __syncthreads();
  const int m = sh.m;
  for (int c = wave; c < m; c += W) {
    const int slot = s_cand[c];
    const size_t r = row0 + s + slot;
    const WavePartial wp = row_pass<Vec, U, 1>(logits + r * (size_t)nvec, nvec, 0, s_kept + wave * 2 * U * kWave);
    const RowResult rr = finish_row_x(wp.m, wp.K, wp.S, wp.first);
    if (lane == 0) {
      store_row(out, r, rr);
      sh.tok[slot] = rr.token;
      sh.conf[slot] = rr.conf;
      sh.e[slot] = (double)rr.eps;
    }
  }
  __syncthreads();
  if (len <= kWave) {
    if (wave != 0) return;
    const size_t i = row0 + (size_t)(s + lane);
    const bool valid = lane < len && mask[i] != 0;
    double ev = valid ? sh.e[lane] : 1.0;
    if constexpr (Robust) {
      if (valid) ev = robust_eps(ev, eta, i);
    }
    bool take = false;
    const int nstar = select_wave<R>(valid, ev, valid ? sh.conf[lane] : 0.0f, param, take);
    if (valid) {
      if (commit) commit[i] = take ? 1 : 0;
      if (take) {
        x[i] = sh.tok[lane];
        mask[i] = 0;
      }
    }
    if (n_commit && lane == 0) n_commit[b] = ok ? nstar : -1;
    return;
  }
  const int N = next_pow2(len);
  for (int slot = tid; slot < N; slot += NT) {
    const size_t i = row0 + (size_t)(s + slot);
    const bool valid = slot < len && mask[i] != 0;
    double ev = 1.0;
    if (valid) {
      ev = sh.e[slot];
      if constexpr (Robust) {
        ev = robust_eps(ev, eta, i);
        sh.e[slot] = ev;
      }
    }
    sh.key[slot] = sort_key(valid, ev, slot);
  }
  __syncthreads();
  const int nstar = select_wg<R, NT>(sh, N, param);
  for (int slot = tid; slot < len; slot += NT) {
    const size_t i = row0 + (size_t)(s + slot);
    if (mask[i] != 0) {
      const bool take = sh.flag[slot] != 0;
      if (commit) commit[i] = take ? 1 : 0;
      if (take) {
        x[i] = sh.tok[slot];
        mask[i] = 0;
      }
    }
  }
  if (n_commit && tid == 0) n_commit[b] = nstar;
}

__global__ void __launch_bounds__(256) k_reveal(const uint8_t* __restrict__ commit,
                                                 const int32_t* __restrict__ tokens,
                                                 int32_t* __restrict__ x, uint8_t* __restrict__ mask,
                                                 long long n) {
  for (long long k = (long long)blockIdx.x * blockDim.x + threadIdx.x; k < n;
       k += (long long)gridDim.x * blockDim.x) {
    if (commit[k]) {
      x[k] = tokens[k];
      mask[k] = 0;
    }
  }
}

// ---------------------------------------------------------------------------
// opt-in input check: windows, and candidate rows holding a logit that is
// NaN, inf or beyond FDLLM_MAX_ABS_LOGIT.  counts: [out of span, too long,
// bad rows]; one wave per slot of the span, four per workgroup.
// ---------------------------------------------------------------------------
__global__ void k_check_clear(int32_t* __restrict__ counts) {
  if (threadIdx.x < 3) counts[threadIdx.x] = 0;
}

template <class Vec>
__global__ void __launch_bounds__(256) k_check(const typename Vec::Raw* __restrict__ logits, int B,
                                               int L, int nvec, const uint8_t* __restrict__ mask,
                                               const int32_t* __restrict__ bstart,
                                               const int32_t* __restrict__ bend,
                                               int32_t* __restrict__ counts) {
  const int lane = threadIdx.x % kWave;
  const long long slot = (long long)blockIdx.x * 4 + threadIdx.x / kWave;
  if (slot >= (long long)B * L) return;
  const int b = (int)(slot / L), i = (int)(slot % L);
  const int s = bstart[b], e = bend[b];
  if (!(s >= 0 && s <= e && e <= L)) {
    if (i == 0 && lane == 0) atomicAdd(&counts[0], 1);
    return;
  }
  if (e - s > kMaxBlock) {
    if (i == 0 && lane == 0) atomicAdd(&counts[1], 1);
    return;
  }
  if (i < s || i >= e || mask[slot] == 0) return;
  const typename Vec::Raw* row = logits + slot * (long long)nvec;
  bool bad = false;
  for (int v = lane; v < nvec; v += kWave) bad |= Vec::bad(load_stream(row + v));
  if (__ballot(bad) != 0ull && lane == 0) atomicAdd(&counts[2], 1);
}

// ---------------------------------------------------------------------------
// host side: planning and launches
// ---------------------------------------------------------------------------
struct Plan {
  bool fused;   // one workgroup per sequence, selection in the same kernel
  int split;    // wavefronts per row in the confidence kernel
  int parts;    // decode step with a workspace: split over split / 4 workgroups (0: no)
  int rem;      // fused: the last rem sequences take the small-batch plan, beside (0: none)
  int rsplit, rparts;   // that plan's split and parts
};

// Compute units of the current device (0 when there is none), cached.
static int device_cus() {
  static std::mutex mu;
  static int cus[64];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lock(mu);
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
      return 0;
    cus[dev] = n;
  }
  return cus[dev];
}

constexpr int kFusedMinB = FDLLM_FUSED_MIN_B;
constexpr int kHybridMaxRem = FDLLM_HYBRID_MAX_REM;   // largest remainder run beside the main kernel
constexpr int kFusedWaves = FDLLM_FUSED_WAVES;   // waves per workgroup in the fused kernel
constexpr int kTargetWaves = FDLLM_TARGET_WAVES;   // row-streaming waves the split aims for

static Plan make_plan(int B, int L, int V, fdllm_dtype dt) {
  Plan p{};
  // slots per sequence the split aims to fill: spans of at most one
  // wavefront count every position (the parts kernel has a slot for each),
  // longer spans their window-relative row groups
  const long long win = L <= kWaveBlock ? L : row_groups(B, L);
  p.fused = B >= kFusedMinB;
  p.split = 1;
  if (p.fused) {
    // one 8-wave workgroup per sequence fills a CU, so a few sequences beyond
    // a multiple of the CU count would make a second round that leaves most
    // CUs idle; they take the small-batch plan instead, on a side stream
    const int cus = device_cus();
    const int rem = cus > 0 ? B % cus : 0;
    if (B > cus && rem <= kHybridMaxRem && rem < kFusedMinB) {
      const Plan q = make_plan(rem, L, V, dt);
      p.rem = rem;
      p.rsplit = q.split;
      p.rparts = q.parts;
    }
  }
  if (!p.fused) {
    // split rows while each part keeps at least 8 16-byte vectors per lane
    const long long row_bytes = (long long)V * (dt == FDLLM_BF16 ? 2 : 4);
    const long long max_split = row_bytes / (16LL * kWave * 8);
    const long long slots = (long long)B * win;
    while (p.split < 16 && 2LL * p.split <= max_split && slots * p.split < kTargetWaves) p.split <<= 1;
    // a row split 8 or 16 ways fills one CU; blocks of at most one wavefront
    // can take their rows' parts from several workgroups instead
    if (L <= kWaveBlock && p.split >= 8) p.parts = p.split;
  }
  return p;
}

static bool vec_path(const void* logits, int V, fdllm_dtype dt) {
  const int per = dt == FDLLM_BF16 ? 8 : 4;
  return V % per == 0 && ((uintptr_t)logits % 16) == 0;
}

template <class Vec>
static hipError_t launch_confidence_t(const void* logits, int B, int L, int nvec, int split,
                                      const uint8_t* mask, const int32_t* bs, const int32_t* be,
                                      RowOut out, hipStream_t st) {
  const long long nvslots = (long long)B * row_groups(B, L);   // window-relative
  const auto* lg = (const typename Vec::Raw*)logits;
#define FDLLM_CONF_CASE(SPLIT)                                                                  \
  case SPLIT: {                                                                                 \
    using Sh = SplitShape<SPLIT>;                                                               \
    const long long grid = (nvslots + Sh::kRows - 1) / Sh::kRows;                               \
    hipLaunchKernelGGL((k_confidence<Vec, SPLIT == 1 ? Vec::kU : Vec::kUSplit, SPLIT>),           \
                       dim3((unsigned)grid), dim3(Sh::kThreads),                                \
                       0, st, lg, B, L, nvec, mask, bs, be, out);                               \
    break;                                                                                      \
  }
  switch (split) {
    FDLLM_CONF_CASE(1)
    FDLLM_CONF_CASE(2)
    FDLLM_CONF_CASE(4)
    FDLLM_CONF_CASE(8)
    FDLLM_CONF_CASE(16)
    default:
      return hipErrorInvalidValue;
  }
#undef FDLLM_CONF_CASE
  return hipGetLastError();
}

template <class Vec>
static hipError_t launch_confidence_parts_t(const void* logits, int B, int L, int nvec, int split,
                                            const uint8_t* mask, const int32_t* bs,
                                            const int32_t* be, RowOut out, WavePartial* parts,
                                            hipStream_t st) {
  const long long nslots = (long long)B * L;
  const auto* lg = (const typename Vec::Raw*)logits;
  const dim3 grid((unsigned)(nslots * (split / 4))), block(256);
  if (split == 8)
    hipLaunchKernelGGL((k_confidence_parts<Vec, Vec::kUSplit, 8>), grid, block, 0, st, lg, B, L, nvec,
                       mask, bs, be, out, parts);
  else if (split == 16)
    hipLaunchKernelGGL((k_confidence_parts<Vec, Vec::kUSplit, 16>), grid, block, 0, st, lg, B, L, nvec,
                       mask, bs, be, out, parts);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

static hipError_t launch_confidence_parts(const void* logits, fdllm_dtype dt, int B, int L, int V,
                                          int split, const uint8_t* mask, const int32_t* bs,
                                          const int32_t* be, RowOut out, WavePartial* parts,
                                          hipStream_t st) {
  if (vec_path(logits, V, dt)) {
    if (dt == FDLLM_BF16)
      return launch_confidence_parts_t<VecBf16x8>(logits, B, L, V / 8, split, mask, bs, be, out,
                                                  parts, st);
    return launch_confidence_parts_t<VecF32x4>(logits, B, L, V / 4, split, mask, bs, be, out, parts,
                                               st);
  }
  if (dt == FDLLM_BF16)
    return launch_confidence_parts_t<VecBf16x1>(logits, B, L, V, split, mask, bs, be, out, parts, st);
  return launch_confidence_parts_t<VecF32x1>(logits, B, L, V, split, mask, bs, be, out, parts, st);
}

static hipError_t launch_confidence(const void* logits, fdllm_dtype dt, int B, int L, int V,
                                    int split, const uint8_t* mask, const int32_t* bs,
                                    const int32_t* be, RowOut out, hipStream_t st) {
  if (vec_path(logits, V, dt)) {
    if (dt == FDLLM_BF16)
      return launch_confidence_t<VecBf16x8>(logits, B, L, V / 8, split, mask, bs, be, out, st);
    return launch_confidence_t<VecF32x4>(logits, B, L, V / 4, split, mask, bs, be, out, st);
  }
  if (dt == FDLLM_BF16)
    return launch_confidence_t<VecBf16x1>(logits, B, L, V, split, mask, bs, be, out, st);
  return launch_confidence_t<VecF32x1>(logits, B, L, V, split, mask, bs, be, out, st);
}

template <int R, bool Robust>
static void launch_select_t(const SelectIO& io, int B, int L, float param, hipStream_t st,
                            int ps, const WavePartial* parts, RowOut out) {
  constexpr int kWideThreads = 256;
  const dim3 g((unsigned)((B + 3) / 4)), t(256);
  if (ps == 8)
    hipLaunchKernelGGL((k_select<R, Robust, 8>), g, t, 0, st, io, B, L, param, parts, out);
  else if (ps == 16)
    hipLaunchKernelGGL((k_select<R, Robust, 16>), g, t, 0, st, io, B, L, param, parts, out);
  else if (L <= kWaveBlock)
    hipLaunchKernelGGL((k_select<R, Robust, 0>), g, t, 0, st, io, B, L, param, parts, out);
  else
    hipLaunchKernelGGL((k_select_wide<R, Robust, kWideThreads>), dim3((unsigned)B),
                       dim3(kWideThreads), 0, st, io, B, L, param);
}

// ps: 0, or the parts per row (8 or 16, L <= 64) left by k_confidence_parts
hipError_t launch_select(fdllm_selector sel, const SelectIO& io, int B, int L, float param,
                         hipStream_t st, int ps, const WavePartial* parts, RowOut out) {
  switch (sel) {
    case FDLLM_SEL_THRESHOLD: launch_select_t<kThreshold, false>(io, B, L, param, st, ps, parts, out); break;
    case FDLLM_SEL_FACTOR: launch_select_t<kFactor, false>(io, B, L, param, st, ps, parts, out); break;
    case FDLLM_SEL_ROBUST: launch_select_t<kProfile, true>(io, B, L, param, st, ps, parts, out); break;
    default: launch_select_t<kProfile, false>(io, B, L, param, st, ps, parts, out); break;
  }
  return hipGetLastError();
}

hipError_t launch_select(fdllm_selector sel, const SelectIO& io, int B, int L, float param,
                         hipStream_t st) {
  return launch_select(sel, io, B, L, param, st, 0, nullptr, RowOut{});
}

template <class Vec, int R, bool Robust>
static void launch_fused_t(const void* logits, int B, int L, int nvec, uint8_t* mask,
                           const int32_t* bs, const int32_t* be, int32_t* x, float param,
                           EtaIn eta, RowOut out, uint8_t* commit, int32_t* n_commit,
                           hipStream_t st) {
  if (L <= kWaveBlock)
    hipLaunchKernelGGL((k_fused<Vec, Vec::kU, kFusedWaves, R, Robust>), dim3((unsigned)B),
                       dim3(kFusedWaves * kWave), 0, st, (const typename Vec::Raw*)logits, B, L,
                       nvec, mask, bs, be, x, param, eta, out, commit, n_commit);
  else
    hipLaunchKernelGGL((k_fused_wide<Vec, Vec::kU, kFusedWaves, R, Robust>), dim3((unsigned)B),
                       dim3(kFusedWaves * kWave), 0, st, (const typename Vec::Raw*)logits, B, L,
                       nvec, mask, bs, be, x, param, eta, out, commit, n_commit);
}

template <class Vec>
static hipError_t launch_fused_v(fdllm_selector sel, const void* logits, int B, int L, int nvec,
                                 uint8_t* mask, const int32_t* bs, const int32_t* be, int32_t* x,
                                 float param, EtaIn eta, RowOut out, uint8_t* commit,
                                 int32_t* n_commit, hipStream_t st) {
  switch (sel) {
    case FDLLM_SEL_THRESHOLD:
      launch_fused_t<Vec, kThreshold, false>(logits, B, L, nvec, mask, bs, be, x, param, eta, out,
                                             commit, n_commit, st);
      break;
    case FDLLM_SEL_FACTOR:
      launch_fused_t<Vec, kFactor, false>(logits, B, L, nvec, mask, bs, be, x, param, eta, out,
                                          commit, n_commit, st);
      break;
    case FDLLM_SEL_ROBUST:
      launch_fused_t<Vec, kProfile, true>(logits, B, L, nvec, mask, bs, be, x, param, eta, out,
                                          commit, n_commit, st);
      break;
    default:
      launch_fused_t<Vec, kProfile, false>(logits, B, L, nvec, mask, bs, be, x, param, eta, out,
                                           commit, n_commit, st);
      break;
  }
  return hipGetLastError();
}

static hipError_t launch_fused(fdllm_selector sel, const void* logits, fdllm_dtype dt, int B, int L,
                               int V, uint8_t* mask, const int32_t* bs, const int32_t* be,
                               int32_t* x, float param, EtaIn eta, RowOut out, uint8_t* commit,
                               int32_t* n_commit, hipStream_t st) {
  if (vec_path(logits, V, dt)) {
    if (dt == FDLLM_BF16)
      return launch_fused_v<VecBf16x8>(sel, logits, B, L, V / 8, mask, bs, be, x, param, eta, out,
                                       commit, n_commit, st);
    return launch_fused_v<VecF32x4>(sel, logits, B, L, V / 4, mask, bs, be, x, param, eta, out,
                                    commit, n_commit, st);
  }
  if (dt == FDLLM_BF16)
    return launch_fused_v<VecBf16x1>(sel, logits, B, L, V, mask, bs, be, x, param, eta, out, commit,
                                     n_commit, st);
  return launch_fused_v<VecF32x1>(sel, logits, B, L, V, mask, bs, be, x, param, eta, out, commit,
                                  n_commit, st);
}

// A stream of the library's own per device, on which the small-batch
// remainder of a fused step runs beside the fused kernel (default priority).
static std::mutex g_side_mu;
constexpr int kSideDevices = 64;
static hipStream_t g_side[kSideDevices];

static hipError_t side_stream(hipStream_t* out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kSideDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_side_mu);
  if (!g_side[dev]) {
    e = hipStreamCreateWithFlags(&g_side[dev], hipStreamNonBlocking);
    if (e != hipSuccess) {
      g_side[dev] = nullptr;
      return e;
    }
  }
  *out = g_side[dev];
  return hipSuccess;
}

static bool sizes_ok(int B, int L, int V) {
  if (B < 0 || L < 1 || V < 1) return false;
  const long double total = (long double)B * (long double)L * (long double)V;
  return total < 4.0e18L;
}


// tokens, conf and eps when the caller does not take them, then the rows'
// wave partials of the parts plan
static size_t out_bytes_for(int B, int L) { return 3 * align256((size_t)B * (size_t)L * 4); }
static size_t workspace_bytes_for(int B, int L, const Plan& p) {
  if (p.fused) {
    if (!p.rem) return 0;
    const size_t n = (size_t)p.rem * (size_t)L;
    return out_bytes_for(p.rem, L) + (p.rparts ? align256(n * p.rparts * sizeof(WavePartial)) : 0);
  }
  const size_t n = (size_t)B * (size_t)L;
  return out_bytes_for(B, L) + (p.parts ? align256(n * p.parts * sizeof(WavePartial)) : 0);
}

// The plan of the small-batch remainder of a fused plan.
static Plan remainder_plan(const Plan& p) {
  Plan q{};
  q.split = p.rsplit;
  q.parts = p.rparts;
  return q;
}

// The small-batch step: the vocabulary pass into the caller's arrays (or
// the workspace), then one launch that selects and reveals.
static fdllm_status step_split(const Plan& p, fdllm_selector sel, const void* logits,
                               fdllm_dtype dtype, int B, int L, int V, uint8_t* mask,
                               const int32_t* block_start, const int32_t* block_end, int32_t* x,
                               float param, EtaIn etain, int32_t* tokens, float* conf, float* eps,
                               float* lse, uint8_t* commit, int32_t* n_commit, void* workspace,
                               size_t workspace_bytes, hipStream_t st) {
  const size_t n = (size_t)B * (size_t)L;
  const bool need_ws = !tokens || !conf || !eps;
  if (need_ws && (!workspace || workspace_bytes < out_bytes_for(B, L))) return FDLLM_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  if (!tokens) tokens = (int32_t*)ws;
  if (!conf) conf = (float*)(ws + align256(n * 4));
  if (!eps) eps = (float*)(ws + 2 * align256(n * 4));
  const RowOut out{tokens, conf, eps, lse};
  SelectIO io{conf, eps, mask, block_start, block_end, commit, n_commit, tokens, x, etain};
  hipError_t err;
  if (p.parts && workspace && workspace_bytes >= out_bytes_for(B, L) +
                                                     align256(n * p.parts * sizeof(WavePartial))) {
    // the rows' parts from several workgroups each, combined by the selection
    // (the same bits as the single-workgroup rows of fdllm_confidence)
    WavePartial* parts = (WavePartial*)(ws + out_bytes_for(B, L));
    err = launch_confidence_parts(logits, dtype, B, L, V, p.parts, mask, block_start, block_end, out,
                                  parts, st);
    if (err != hipSuccess) return FDLLM_ERR_HIP;
    err = launch_select(sel, io, B, L, param, st, p.parts, parts, out);
    return err == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
  }
  err = launch_confidence(logits, dtype, B, L, V, p.split, mask, block_start, block_end, out, st);
  if (err != hipSuccess) return FDLLM_ERR_HIP;
  err = launch_select(sel, io, B, L, param, st);
  return err == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

}  // namespace fdllm

using namespace fdllm;

extern "C" {

const char* fdllm_status_string(fdllm_status st) {
  switch (st) {
    case FDLLM_OK: return "ok";
    case FDLLM_ERR_INVALID_ARG: return "invalid argument (null pointer, negative size or bad enum)";
    case FDLLM_ERR_UNSUPPORTED_DTYPE: return "unsupported logits dtype";
    case FDLLM_ERR_SIZE: return "unsupported size (V < 1 or too many elements)";
    case FDLLM_ERR_WORKSPACE: return "workspace missing or too small";
    case FDLLM_ERR_HIP: return "HIP runtime error at launch";
    case FDLLM_ERR_BOUNDS: return "a block window lies outside [0, L] (start > end, start < 0 or end > L)";
    case FDLLM_ERR_BLOCK_TOO_LARGE: return "a block window is longer than FDLLM_MAX_BLOCK positions";
    case FDLLM_ERR_NONFINITE: return "a candidate logit is NaN, inf or beyond FDLLM_MAX_ABS_LOGIT";
    case FDLLM_ERR_SCRATCH: return "the call needs more than the library's static scratch (FDLLM_STATIC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

fdllm_status fdllm_check_inputs(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                                const uint8_t* mask, const int32_t* block_start,
                                const int32_t* block_end, int32_t* counts, fdllm_stream stream) {
  if (dtype != FDLLM_BF16 && dtype != FDLLM_F32) return FDLLM_ERR_UNSUPPORTED_DTYPE;
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!sizes_ok(B, L, V)) return FDLLM_ERR_SIZE;
  if (!counts) return FDLLM_ERR_INVALID_ARG;
  if (B > 0 && (!logits || !mask || !block_start || !block_end)) return FDLLM_ERR_INVALID_ARG;
  hipStream_t st = (hipStream_t)stream;
  hipLaunchKernelGGL(k_check_clear, dim3(1), dim3(kWave), 0, st, counts);
  if (B > 0) {
    const unsigned grid = (unsigned)(((long long)B * L + 3) / 4);
    if (vec_path(logits, V, dtype)) {
      if (dtype == FDLLM_BF16)
        hipLaunchKernelGGL(k_check<VecBf16x8>, dim3(grid), dim3(256), 0, st,
                           (const u32x4*)logits, B, L, V / 8, mask, block_start, block_end, counts);
      else
        hipLaunchKernelGGL(k_check<VecF32x4>, dim3(grid), dim3(256), 0, st,
                           (const u32x4*)logits, B, L, V / 4, mask, block_start, block_end, counts);
    } else if (dtype == FDLLM_BF16) {
      hipLaunchKernelGGL(k_check<VecBf16x1>, dim3(grid), dim3(256), 0, st,
                         (const unsigned short*)logits, B, L, V, mask, block_start, block_end, counts);
    } else {
      hipLaunchKernelGGL(k_check<VecF32x1>, dim3(grid), dim3(256), 0, st,
                         (const unsigned int*)logits, B, L, V, mask, block_start, block_end, counts);
    }
  }
  if (hipGetLastError() != hipSuccess) return FDLLM_ERR_HIP;
  int32_t host[3] = {0, 0, 0};
  if (hipMemcpyAsync(host, counts, sizeof(host), hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipStreamSynchronize(st) != hipSuccess)
    return FDLLM_ERR_HIP;
  if (host[0] > 0) return FDLLM_ERR_BOUNDS;
  if (host[1] > 0) return FDLLM_ERR_BLOCK_TOO_LARGE;
  if (host[2] > 0) return FDLLM_ERR_NONFINITE;
  return FDLLM_OK;
}

fdllm_status fdllm_workspace_size(int B, int L, int V, fdllm_dtype dtype, size_t* bytes) {
  if (!bytes) return FDLLM_ERR_INVALID_ARG;
  if (dtype != FDLLM_BF16 && dtype != FDLLM_F32) return FDLLM_ERR_UNSUPPORTED_DTYPE;
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!sizes_ok(B, L, V)) return FDLLM_ERR_SIZE;
  *bytes = workspace_bytes_for(B, L, make_plan(B, L, V, dtype));
  return FDLLM_OK;
}

fdllm_status fdllm_confidence(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                              const uint8_t* mask, const int32_t* block_start,
                              const int32_t* block_end, int32_t* tokens, float* conf, float* eps,
                              float* lse, fdllm_stream stream) {
  if (dtype != FDLLM_BF16 && dtype != FDLLM_F32) return FDLLM_ERR_UNSUPPORTED_DTYPE;
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!sizes_ok(B, L, V)) return FDLLM_ERR_SIZE;
  if (B == 0) return FDLLM_OK;
  if (!logits || !mask || !block_start || !block_end || !tokens || !conf) return FDLLM_ERR_INVALID_ARG;
  const Plan p = make_plan(B, L, V, dtype);
  RowOut out{tokens, conf, eps, lse};
  hipStream_t st = (hipStream_t)stream;
  // the rows of a fused step's small-batch remainder are split as the decode
  // step splits them, so that both give the same bits
  const int b0 = B - p.rem;
  hipError_t err = launch_confidence(logits, dtype, b0, L, V, p.split, mask, block_start, block_end,
                                     out, st);
  if (err == hipSuccess && p.rem) {
    const size_t r0 = (size_t)b0 * (size_t)L;
    const size_t esize = dtype == FDLLM_BF16 ? 2 : 4;
    auto off = [](auto* ptr, size_t k) { return ptr ? ptr + k : ptr; };
    err = launch_confidence((const char*)logits + r0 * (size_t)V * esize, dtype, p.rem, L, V,
                            p.rsplit, mask + r0, block_start + b0, block_end + b0,
                            RowOut{off(tokens, r0), off(conf, r0), off(eps, r0), off(lse, r0)}, st);
  }
  return err == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

static fdllm_status select_common(fdllm_selector sel, const float* conf, const float* eps,
                                  const uint8_t* mask, const int32_t* bs, const int32_t* be, int B,
                                  int L, float param, uint8_t* commit, int32_t* n_commit,
                                  fdllm_stream stream, EtaIn eta = EtaIn{nullptr, 0.0f}) {
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (B == 0) return FDLLM_OK;
  if (!conf || !mask || !bs || !be || !commit) return FDLLM_ERR_INVALID_ARG;
  SelectIO io{conf, eps, const_cast<uint8_t*>(mask), bs, be, commit, n_commit, nullptr, nullptr, eta};
  hipError_t err = launch_select(sel, io, B, L, param, (hipStream_t)stream);
  return err == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

fdllm_status fdllm_select_profile(const float* conf, const float* eps, const uint8_t* mask,
                                  const int32_t* block_start, const int32_t* block_end, int B,
                                  int L, float f, uint8_t* commit, int32_t* n_commit,
                                  fdllm_stream stream) {
  return select_common(FDLLM_SEL_PROFILE, conf, eps, mask, block_start, block_end, B, L, f, commit,
                       n_commit, stream);
}

fdllm_status fdllm_select_factor(const float* conf, const float* eps, const uint8_t* mask,
                                 const int32_t* block_start, const int32_t* block_end, int B,
                                 int L, float f, uint8_t* commit, int32_t* n_commit,
                                 fdllm_stream stream) {
  return select_common(FDLLM_SEL_FACTOR, conf, eps, mask, block_start, block_end, B, L, f, commit,
                       n_commit, stream);
}

fdllm_status fdllm_select_threshold(const float* conf, const float* eps, const uint8_t* mask,
                                    const int32_t* block_start, const int32_t* block_end, int B,
                                    int L, float tau, uint8_t* commit, int32_t* n_commit,
                                    fdllm_stream stream) {
  return select_common(FDLLM_SEL_THRESHOLD, conf, eps, mask, block_start, block_end, B, L, tau,
                       commit, n_commit, stream);
}

fdllm_status fdllm_select_robust(const float* conf, const float* eps, const float* eta,
                                 float eta_uniform, const uint8_t* mask, const int32_t* block_start,
                                 const int32_t* block_end, int B, int L, float f, uint8_t* commit,
                                 int32_t* n_commit, fdllm_stream stream) {
  if (!(eta_uniform == eta_uniform)) return FDLLM_ERR_INVALID_ARG;   // NaN
  return select_common(FDLLM_SEL_ROBUST, conf, eps, mask, block_start, block_end, B, L, f, commit,
                       n_commit, stream, EtaIn{eta, eta_uniform});
}

fdllm_status fdllm_reveal(const uint8_t* commit, const int32_t* tokens, int32_t* x, uint8_t* mask,
                          int B, int L, fdllm_stream stream) {
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (B == 0) return FDLLM_OK;
  if (!commit || !tokens || !x || !mask) return FDLLM_ERR_INVALID_ARG;
  const long long n = (long long)B * L;
  long long grid = (n + 255) / 256;
  if (grid > 65536) grid = 65536;
  hipLaunchKernelGGL(k_reveal, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream, commit,
                     tokens, x, mask, n);
  return hipGetLastError() == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

fdllm_status fdllm_decode_step(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                               uint8_t* mask, const int32_t* block_start, const int32_t* block_end,
                               int32_t* x, fdllm_selector sel, float param, const float* eta,
                               float eta_uniform, int32_t* tokens, float* conf, float* eps,
                               float* lse, uint8_t* commit, int32_t* n_commit, void* workspace,
                               size_t workspace_bytes, fdllm_stream stream) {
  return fdllm::decode_step(logits, dtype, B, L, V, mask, block_start, block_end, x, sel, param, eta,
                            eta_uniform, tokens, conf, eps, lse, commit, n_commit, workspace,
                            workspace_bytes, stream, true);
}

}  // extern "C"

namespace fdllm {

fdllm_status decode_step(const void* logits, fdllm_dtype dtype, int B, int L, int V, uint8_t* mask,
                         const int32_t* block_start, const int32_t* block_end, int32_t* x,
                         fdllm_selector sel, float param, const float* eta, float eta_uniform,
                         int32_t* tokens, float* conf, float* eps, float* lse, uint8_t* commit,
                         int32_t* n_commit, void* workspace, size_t workspace_bytes,
                         fdllm_stream stream, bool side_stream_ok) {
  if (dtype != FDLLM_BF16 && dtype != FDLLM_F32) return FDLLM_ERR_UNSUPPORTED_DTYPE;
  if (sel != FDLLM_SEL_THRESHOLD && sel != FDLLM_SEL_FACTOR && sel != FDLLM_SEL_PROFILE &&
      sel != FDLLM_SEL_ROBUST)
    return FDLLM_ERR_INVALID_ARG;
  if (!(eta_uniform == eta_uniform)) return FDLLM_ERR_INVALID_ARG;
  if (B < 0 || L < 1) return FDLLM_ERR_INVALID_ARG;
  if (!sizes_ok(B, L, V)) return FDLLM_ERR_SIZE;
  if (B == 0) return FDLLM_OK;
  if (!logits || !mask || !block_start || !block_end || !x) return FDLLM_ERR_INVALID_ARG;
  const Plan p = make_plan(B, L, V, dtype);
  hipStream_t st = (hipStream_t)stream;
  const EtaIn etain{eta, eta_uniform};
  if (!p.fused)
    return step_split(p, sel, logits, dtype, B, L, V, mask, block_start, block_end, x, param, etain,
                      tokens, conf, eps, lse, commit, n_commit, workspace, workspace_bytes, st);
  RowOut out{tokens, conf, eps, lse};
  const int b0 = B - p.rem;
  const Plan q = remainder_plan(p);
  const bool outs_given = tokens && conf && eps;
  const bool rem_ok = p.rem && (outs_given || (workspace && workspace_bytes >= workspace_bytes_for(B, L, p)));
  const size_t r0 = (size_t)b0 * (size_t)L;
  const size_t esize = dtype == FDLLM_BF16 ? 2 : 4;
  auto off = [](auto* ptr, size_t k) { return ptr ? ptr + k : ptr; };
  // sequences [b0, B) as a small batch (the same launches on either stream)
  auto remainder = [&](hipStream_t on) {
    return step_split(q, sel, (const char*)logits + r0 * (size_t)V * esize, dtype, p.rem, L, V,
                      mask + r0, block_start + b0, block_end + b0, x + r0, param,
                      EtaIn{off(eta, r0), eta_uniform}, off(tokens, r0), off(conf, r0),
                      off(eps, r0), off(lse, r0), off(commit, r0), off(n_commit, (size_t)b0),
                      workspace, workspace_bytes, on);
  };
  if (rem_ok && !side_stream_ok) {
    // no side stream and no events: the remainder after the fused kernel, on
    // the caller's stream (the same kernels and bits, without the overlap)
    if (launch_fused(sel, logits, dtype, b0, L, V, mask, block_start, block_end, x, param, etain, out,
                     commit, n_commit, st) != hipSuccess)
      return FDLLM_ERR_HIP;
    return remainder(st);
  }
  hipStream_t side = nullptr;
  if (rem_ok && side_stream(&side) == hipSuccess) {
    // sequences [b0, B) on the side stream, forked from and joined back to
    // the caller's stream by events, at the same time as the fused kernel
    hipEvent_t fork = nullptr, join = nullptr;
    fdllm_status res = FDLLM_ERR_HIP;
    if (hipEventCreateWithFlags(&fork, hipEventDisableTiming) == hipSuccess &&
        hipEventCreateWithFlags(&join, hipEventDisableTiming) == hipSuccess &&
        hipEventRecord(fork, st) == hipSuccess && hipStreamWaitEvent(side, fork, 0) == hipSuccess) {
      res = remainder(side);
      if (res == FDLLM_OK && hipEventRecord(join, side) != hipSuccess) res = FDLLM_ERR_HIP;
      if (res == FDLLM_OK &&
          launch_fused(sel, logits, dtype, b0, L, V, mask, block_start, block_end, x, param, etain,
                       out, commit, n_commit, st) != hipSuccess)
        res = FDLLM_ERR_HIP;
      if (res == FDLLM_OK && hipStreamWaitEvent(st, join, 0) != hipSuccess) res = FDLLM_ERR_HIP;
    }
    // a recorded event's resources are released once it completes
    if (fork) (void)hipEventDestroy(fork);
    if (join) (void)hipEventDestroy(join);
    return res;
  }
  const hipError_t err = launch_fused(sel, logits, dtype, B, L, V, mask, block_start, block_end, x,
                                      param, etain, out, commit, n_commit, st);
  return err == hipSuccess ? FDLLM_OK : FDLLM_ERR_HIP;
}

}  // namespace fdllm
