// pass_common.h -- device helpers shared by the vocabulary pass
// (fdllm.hip) and the LM head fused with it (lmhead.hip): wavefront
// primitives, the exponent-reference arithmetic of the online softmax, the
// per-row state and its final step, block bounds, outputs, and the selection
// launcher.  Internal to libfdllm.so.
#ifndef FDLLM_PASS_COMMON_H
#define FDLLM_PASS_COMMON_H

#include <hip/hip_runtime.h>

#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "fdllm.h"

namespace fdllm {

constexpr int kWave = 64;
constexpr int kMaxBlock = FDLLM_MAX_BLOCK;   // largest active block (workgroup selection)
constexpr int kWaveBlock = kWave;            // blocks up to this size select in one wavefront
constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kRefFloor = -3.0e38f;   // exponent reference before any element

// ---------------------------------------------------------------------------
// wavefront primitives (wave64)
// ---------------------------------------------------------------------------
__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// DPP controls (gfx9): quad_perm, row_half_mirror, row_mirror.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7-i within 8 (xor 4 once quads agree)
constexpr int kDppMirror = 0x140;     // lane i <-> 15-i within 16 (xor 8 once octets agree)
constexpr int kSwzXor16 = 0x401F;     // ds_swizzle bit mode: and 0x1F, xor 0x10

template <int Ctrl>
__device__ __forceinline__ int dpp(int v) {
  return __builtin_amdgcn_update_dpp(0, v, Ctrl, 0xF, 0xF, false);
}

// Butterfly all-reduce step helpers: return the partner's value for step s.
// Steps 0..3 are DPP, step 4 is ds_swizzle (within 32 lanes); the final
// 32-lane exchange is done with readlane by the callers.
template <int Step>
__device__ __forceinline__ int partner_i32(int v) {
  if constexpr (Step == 0) return dpp<kDppXor1>(v);
  else if constexpr (Step == 1) return dpp<kDppXor2>(v);
  else if constexpr (Step == 2) return dpp<kDppHalfMirror>(v);
  else if constexpr (Step == 3) return dpp<kDppMirror>(v);
  else return __builtin_amdgcn_ds_swizzle(v, kSwzXor16);
}

template <int Step>
__device__ __forceinline__ float partner_f32(float v) {
  return __int_as_float(partner_i32<Step>(__float_as_int(v)));
}

template <int Step>
__device__ __forceinline__ double partner_f64(double v) {
  long long b = __double_as_longlong(v);
  int lo = partner_i32<Step>((int)(b & 0xffffffffll));
  int hi = partner_i32<Step>((int)(b >> 32));
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ float readlane_f32(float v, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
__device__ __forceinline__ double readlane_f64(double v, int l) {
  long long b = __double_as_longlong(v);
  int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffffll), l);
  int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ float wave_max(float v) {
  v = fmaxf(v, partner_f32<0>(v));
  v = fmaxf(v, partner_f32<1>(v));
  v = fmaxf(v, partner_f32<2>(v));
  v = fmaxf(v, partner_f32<3>(v));
  v = fmaxf(v, partner_f32<4>(v));
  return fmaxf(readlane_f32(v, 0), readlane_f32(v, 32));
}

__device__ __forceinline__ int wave_min(int v) {
  v = min(v, partner_i32<0>(v));
  v = min(v, partner_i32<1>(v));
  v = min(v, partner_i32<2>(v));
  v = min(v, partner_i32<3>(v));
  v = min(v, partner_i32<4>(v));
  return min(__builtin_amdgcn_readlane(v, 0), __builtin_amdgcn_readlane(v, 32));
}

// ---------------------------------------------------------------------------
// exponent reference and per-element term.  Shared by the streaming loop
// and the final step, so the greedy element's term is recomputed bit-exactly.
// ---------------------------------------------------------------------------
//
// exp_ref(m) is the smallest integer K >= m * log2e (log2e taken as the float
// kLog2e), so for |m| <= FDLLM_MAX_ABS_LOGIT (|K| < 2^24, a float) the
// maximum's own argument m * log2e - K lies in (-1, 0] at every magnitude and
// its term in (1/2, 1].  It is formed in float arithmetic without rounding
// error: p = fl(m log2e) and e = fma(m, log2e, -p) = m log2e - p exactly (the
// error of a rounded product is a float).  While |p| < 2^24 the integers are
// on p's grid and |e| is at most half its spacing, so the exact product and p
// have the same ceiling unless p is itself an integer, and then the ceiling
// is p + 1 exactly when e > 0.  (The ceiling of p alone can leave the
// maximum's argument above 0.)  Beyond 2^24, outside the documented range, K
// is the next float above ceil(p), an integer >= the exact product, so the
// argument stays <= 0 and no term overflows.
__device__ __forceinline__ float exp_ref(float m) {
  const float p = m * kLog2e;
  const float e = __builtin_fmaf(m, kLog2e, -p);
  const float c = __builtin_ceilf(p);
  const float in_range = (c == p && e > 0.0f) ? c + 1.0f : c;
  const float next = __int_as_float(__float_as_int(c) + (c > 0.0f ? 1 : -1));
  const float beyond = __builtin_isinf(c) ? c : next;
  return __builtin_fabsf(c) < 16777216.0f ? in_range : beyond;
}
__device__ __forceinline__ float term(float x, float K) {
  return __builtin_amdgcn_exp2f(__builtin_fmaf(x, kLog2e, -K));
}
// 2^(a - b) applied to s, with a <= b integer-valued floats (exact).
__device__ __forceinline__ double rescale(double s, float a, float b) {
  float d = fmaxf(a - b, -2000.0f);
  return ldexp(s, (int)d);
}

// (K, S) pair combine: both sums brought to the larger reference.
__device__ __forceinline__ void ks_combine(float& K, double& S, float K2, double S2) {
  float Kn = fmaxf(K, K2);
  S = rescale(S, K, Kn) + rescale(S2, K2, Kn);
  K = Kn;
}

template <int Step>
__device__ __forceinline__ void ks_step(float& K, double& S) {
  float K2 = partner_f32<Step>(K);
  double S2 = partner_f64<Step>(S);
  ks_combine(K, S, K2, S2);
}

// The vocabulary pass keeps, for every stretch of a row (a lane's elements,
// a wave's, a part of a split row), the sum of the terms of all its elements
// except one occurrence of the stretch's maximum m.  Stretches are combined
// by taking the largest maximum M, having every stretch but the lowest-index
// one that holds M put its own maximum's term back, and adding in a fixed
// order: the row's sum is then every term but one occurrence of the row
// maximum, s' e_M, built without the greedy term and without any
// subtraction, so eps keeps its relative accuracy however close c is to 1.

// Sum over the wave by a fixed butterfly; every lane ends with the same bits.
__device__ __forceinline__ double wave_sum_f64(double v) {
  v += partner_f64<0>(v);
  v += partner_f64<1>(v);
  v += partner_f64<2>(v);
  v += partner_f64<3>(v);
  v += partner_f64<4>(v);
  return readlane_f64(v, 0) + readlane_f64(v, 32);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Online state of a stretch of one row: its maximum, the integer-valued
// exponent reference, the sum of scaled terms and the lowest index of the
// maximum.
struct WavePartial {
  float m;    // maximum over the wave's elements (uniform)
  float K;    // exp_ref(m) (uniform)
  double S;   // sum of 2^(x log2e - K) over the wave's elements (uniform); the
              // vocabulary pass leaves one occurrence of m out,
              // the LM-head folds keep every term (finish_row)
  int first;  // lowest element index holding m (uniform)
};

struct RowResult {
  int token;
  float conf, eps, lse;
};

// Final step of a row of the vocabulary pass from its (M, K, S, first), S
// without the greedy element's term: s' = S / e_M.
__device__ __forceinline__ RowResult finish_row_x(float M, float K, double S, int first) {
  const float Kr = exp_ref(M);
  const double eM = rescale((double)term(M, Kr), Kr, K);
  const double sp = S / eM;
  RowResult r;
  r.token = first;
  r.conf = (float)(1.0 / (1.0 + sp));
  r.eps = (float)(sp / (1.0 + sp));
  r.lse = (float)((double)M + log1p(sp));
  return r;
}

// Final step of a row of the LM-head folds from its (m, K, S, first), S with
// every term: s' = (S - e_M) / e_M with e_M the greedy element's own term,
// recomputed exactly as it was summed.
__device__ __forceinline__ RowResult finish_row(float M, float K, double S, int first) {
  const float Kr = exp_ref(M);
  const double eM = rescale((double)term(M, Kr), Kr, K);
  const double sp = fmax((S - eM) / eM, 0.0);
  RowResult r;
  r.token = first;
  r.conf = (float)(1.0 / (1.0 + sp));
  r.eps = (float)(sp / (1.0 + sp));
  r.lse = (float)((double)M + log1p(sp));
  return r;
}

// ---------------------------------------------------------------------------
// block bounds and candidates
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool window_ok(int s, int e, int L) {
  return s >= 0 && s <= e && e <= L && e - s <= kMaxBlock;
}

struct RowOut {
  int32_t* tokens;
  float* conf;
  float* eps;
  float* lse;
};

__device__ __forceinline__ void store_row(const RowOut& o, size_t idx, const RowResult& r) {
  if (o.tokens) o.tokens[idx] = r.token;
  if (o.conf) o.conf[idx] = r.conf;
  if (o.eps) o.eps[idx] = r.eps;
  if (o.lse) o.lse[idx] = r.lse;
}
__device__ __forceinline__ void store_default(const RowOut& o, size_t idx) {
  if (o.tokens) o.tokens[idx] = -1;
  if (o.conf) o.conf[idx] = 0.0f;
  if (o.eps) o.eps[idx] = 1.0f;
  if (o.lse) o.lse[idx] = 0.0f;
}

enum Rule { kThreshold = 0, kFactor = 1, kProfile = 2 };

// eps of a candidate from float eps (preferred) or conf only, then the
// calibration allowance of the robust rule: eps_low = min(1, eps + max(0, eta)).
struct EtaIn {
  const float* eta;      // [B, L] per-position allowance, or null
  float uniform;         // allowance when eta is null
};

__device__ __forceinline__ double cand_eps(const float* eps_arr, float c, size_t idx) {
  return eps_arr ? (double)eps_arr[idx] : 1.0 - (double)c;   // 1 - c is exact in double
}
__device__ __forceinline__ double robust_eps(double e, const EtaIn& eta, size_t idx) {
  const float h = eta.eta ? eta.eta[idx] : eta.uniform;
  return fmin(1.0, e + fmax((double)h, 0.0));
}

struct SelectIO {
  const float* conf;
  const float* eps;           // may be null
  uint8_t* mask;              // read; cleared at commits when reveal
  const int32_t* bstart;
  const int32_t* bend;
  uint8_t* commit;            // may be null
  int32_t* n_commit;          // may be null
  const int32_t* tokens;      // reveal source (may be null: no reveal)
  int32_t* x;                 // reveal target (may be null: no reveal)
  EtaIn eta;                  // calibration allowance (robust rule)
};

// Host side, defined with the selection kernels: selection and reveal of
// every block from conf / eps (the kernels of fdllm_select_*).
hipError_t launch_select(fdllm_selector sel, const SelectIO& io, int B, int L, float param,
                         hipStream_t st);

inline size_t align256(size_t n) { return (n + 255) & ~(size_t)255; }

// Host side, defined with the decode-step kernels: fdllm_decode_step, whose
// large batches may run their last sequences on a side stream beside the
// one-kernel part.  Without side_stream_ok those sequences run after it on
// `stream` instead (same kernels, same bits), so the call creates no stream
// and no event (fdllm_decode_step_static).
fdllm_status decode_step(const void* logits, fdllm_dtype dtype, int B, int L, int V, uint8_t* mask,
                         const int32_t* block_start, const int32_t* block_end, int32_t* x,
                         fdllm_selector sel, float param, const float* eta, float eta_uniform,
                         int32_t* tokens, float* conf, float* eps, float* lse, uint8_t* commit,
                         int32_t* n_commit, void* workspace, size_t workspace_bytes,
                         fdllm_stream stream, bool side_stream_ok);

}  // namespace fdllm

#endif  // FDLLM_PASS_COMMON_H
