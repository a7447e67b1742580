/*
 * fdllm.h -- C ABI of the Fast-dLLM++ commit selector for AMD Instinct MI355X
 * (gfx950).  Implements one decoding step of Frechet profile decoding
 * (arXiv 2606.02955, Alg. 1): per masked position of the active block the
 * greedy token and its softmax confidence, per block the commit set chosen by
 * the Frechet profile rule (its calibration-robust variant, or the factor /
 * threshold baselines), and the reveal of the chosen tokens.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every array pointer is DEVICE memory owned by the caller
 *   (allocated with hipMalloc or by a framework such as PyTorch).  The library
 *   never allocates, frees or retains a pointer beyond the call.
 * Layout.  Arrays are contiguous and row-major:
 *   logits [B, L, V]            bf16 (FDLLM_BF16) or fp32 (FDLLM_F32)
 *   mask   [B, L]  uint8        1 = position still masked
 *   x      [B, L]  int32        sequence tokens
 *   tokens [B, L]  int32        greedy token (argmax over V)
 *   conf   [B, L]  float        confidence c = max_v softmax(logits)_v
 *   eps    [B, L]  float        1 - c, computed without cancellation
 *   lse    [B, L]  float        log sum_v exp(logits_v)
 *   commit [B, L]  uint8        1 = position revealed this step
 *   n_commit [B]   int32        number of revealed positions per sequence
 *   block_start, block_end [B] int32: sequence b's active block is the
 *   half-open span [block_start[b], block_end[b]) of its L positions.
 *   The L rows may be the active block itself (start 0, end L: logits of a
 *   cached model call) or a longer span of which the bounds select the block.
 * Candidates.  Position i of sequence b is a candidate when
 *   block_start[b] <= i < block_end[b] and mask[b, i] != 0 (Alg. 1 visits the
 *   masked positions of the active block).  Logits of other rows are never
 *   read; their outputs are tokens = -1, conf = 0, eps = 1, lse = 0,
 *   commit = 0.
 * Bounds.  A block needs 0 <= start <= end <= L and end - start <= 1024
 *   (FDLLM_MAX_BLOCK).  Blocks of up to 64 positions are selected within one
 *   64-lane wavefront, larger ones (block-size ablations) by a workgroup.
 *   Bounds live in device memory and are checked on the device: a sequence
 *   with invalid bounds gets no commits, default outputs and n_commit = -1
 *   (where n_commit is written).  fdllm_check_inputs reports such sequences
 *   to the host.
 * Logits.  Must be finite with |logit| <= FDLLM_MAX_ABS_LOGIT (1e7).  Within
 *   that range every row's exponent reference is exact (the row maximum's own
 *   term lies in (1/2, 1]), so results do not depend on the logits' offset.
 *   NaN, inf and larger magnitudes are outside the contract (results are
 *   unspecified, no fault); fdllm_check_inputs detects them.
 * Ties.  The argmax takes the lowest vocabulary index; the confidence sort
 *   puts equal values at the lower position first.
 * Streams.  Every call only enqueues work on `stream` (NULL = the null
 *   stream) and returns; results are visible after stream synchronisation.
 *   Kernel faults surface at that synchronisation.
 * Errors.  Argument checks are done on the host before anything is enqueued;
 *   a failing check returns a negative status and enqueues nothing.
 * Determinism.  For fixed (B, L, V, dtype) every call is bitwise
 *   reproducible, identical rows give bitwise identical outputs, and
 *   fdllm_decode_step gives bitwise the same tokens/conf/eps/lse as
 *   fdllm_confidence and the same commits as fdllm_select_* fed with them.
 */
#ifndef FDLLM_H
#define FDLLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A hipStream_t (same underlying type); NULL selects the null stream. */
typedef struct ihipStream_t* fdllm_stream;

/* Logits element type.  Plain int, so that any value a caller passes is a
 * value of the type (an out-of-range value of a C++ enum would not be, and the
 * range check that rejects it could then be compiled away). */
typedef int fdllm_dtype;
enum { FDLLM_BF16 = 0, FDLLM_F32 = 1 };

/* Selection rule (plain int, as fdllm_dtype). */
typedef int fdllm_selector;
enum {
  FDLLM_SEL_THRESHOLD = 0, /* commit every c >= tau, else the single highest        */
  FDLLM_SEL_FACTOR = 1,    /* largest n with (n+1)(1 - c_(n)) < f                   */
  FDLLM_SEL_PROFILE = 2,   /* largest n with G_n > 1 - f (Frechet profile rule)     */
  FDLLM_SEL_ROBUST = 3     /* profile rule on c_low = max(0, c - eta) (robust rule) */
};

typedef int fdllm_status;
#define FDLLM_OK 0
#define FDLLM_ERR_INVALID_ARG (-1)       /* null pointer, negative size, bad enum   */
#define FDLLM_ERR_UNSUPPORTED_DTYPE (-2) /* dtype not FDLLM_BF16 / FDLLM_F32         */
#define FDLLM_ERR_SIZE (-3)              /* V < 1, or B*L*V beyond 2^62 elements     */
#define FDLLM_ERR_WORKSPACE (-4)         /* workspace missing or too small           */
#define FDLLM_ERR_HIP (-5)               /* the HIP runtime rejected a launch        */
#define FDLLM_ERR_BOUNDS (-6)            /* fdllm_check_inputs: a window outside [0, L] */
#define FDLLM_ERR_BLOCK_TOO_LARGE (-7)   /* fdllm_check_inputs: end - start > FDLLM_MAX_BLOCK */
#define FDLLM_ERR_NONFINITE (-8)         /* fdllm_check_inputs: a candidate logit is NaN,
                                            inf or beyond FDLLM_MAX_ABS_LOGIT           */
#define FDLLM_ERR_SCRATCH (-9)           /* fdllm_decode_step_static: the call needs more
                                            than FDLLM_STATIC_SCRATCH_BYTES of scratch  */

#define FDLLM_MAX_BLOCK 1024
#define FDLLM_MAX_ABS_LOGIT 1.0e7f
#define FDLLM_STATIC_SCRATCH_BYTES (8u << 20)   /* fdllm_decode_step_static, per GPU */

/*
 * Greedy token, confidence, complement and log-sum-exp of every candidate
 * position (Sec. 3 "Notation": x*_i = argmax_v p_i(v), c_i = p_i(x*_i); Alg. 1
 * per-position loop; softmax at temperature 1 as in greedy decoding).  Each
 * logit of a candidate row is read exactly once.
 *   logits  [B,L,V] bf16/fp32 per `dtype`        (in)
 *   mask    [B,L] uint8                           (in)
 *   block_start, block_end [B] int32              (in)
 *   tokens  [B,L] int32                           (out, required)
 *   conf    [B,L] float                           (out, required)
 *   eps     [B,L] float                           (out, may be NULL)
 *   lse     [B,L] float                           (out, may be NULL)
 */
fdllm_status fdllm_confidence(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                              const uint8_t* mask, const int32_t* block_start,
                              const int32_t* block_end, int32_t* tokens, float* conf, float* eps,
                              float* lse, fdllm_stream stream);

/*
 * Commit set of each block from per-position confidences (phase after the
 * vocabulary pass).  Candidates are ordered by confidence descending --
 * by eps ascending when `eps` is given, else by conf descending -- with
 * ties to the lower position; this is the sort of Alg. 1.
 *
 * fdllm_select_profile: Frechet profile rule (Sec. 3 "Frechet profile
 *   quantities"; Alg. 1 selection).  With c_(j) the sorted confidences,
 *   L_n = max{0, sum_{j<=n} c_(j) - (n-1)}, U_n = 1 - c_(n), G_n = L_n - U_n,
 *   n* = max{n : G_n > delta}, delta = 1 - f (matched parameterisation,
 *   equal-confidence corollary and Sec. 5), n* = 1 when no n qualifies.  It
 *   is evaluated as (n+1)(1 - c_(n)) - B_n < f with the heterogeneity bonus
 *   B_n = sum_{j<n} (c_(j) - c_(n)) (adaptive-factor remark), which accepts
 *   exactly the same n as the clipped definition for f <= 1 and is the rule
 *   used for f > 1.
 * fdllm_select_factor: Fast-dLLM factor rule (Sec. 2; Sec. 5 "Baselines"):
 *   largest n with (n+1)(1 - c_(n)) < f, else 1.
 * fdllm_select_threshold: (Sec. 2) every candidate with conf >= tau; when
 *   none qualifies, the single highest-confidence candidate.
 * Arguments:
 *   conf [B,L] float (in, required); eps [B,L] float (in, may be NULL: then
 *   eps = 1 - conf exactly); mask, block_start, block_end as above (in);
 *   param: f for profile/factor, tau for threshold;
 *   commit [B,L] uint8 (out, required; every entry written);
 *   n_commit [B] int32 (out, may be NULL).
 * The criterion is evaluated in double precision on the given float values.
 */
fdllm_status fdllm_select_profile(const float* conf, const float* eps, const uint8_t* mask,
                                  const int32_t* block_start, const int32_t* block_end, int B,
                                  int L, float f, uint8_t* commit, int32_t* n_commit,
                                  fdllm_stream stream);
fdllm_status fdllm_select_factor(const float* conf, const float* eps, const uint8_t* mask,
                                 const int32_t* block_start, const int32_t* block_end, int B,
                                 int L, float f, uint8_t* commit, int32_t* n_commit,
                                 fdllm_stream stream);
fdllm_status fdllm_select_threshold(const float* conf, const float* eps, const uint8_t* mask,
                                    const int32_t* block_start, const int32_t* block_end, int B,
                                    int L, float tau, uint8_t* commit, int32_t* n_commit,
                                    fdllm_stream stream);

/*
 * Calibration-robust Frechet profile rule (appendix "Calibration-Robust
 * Frechet Certificates"): each reported confidence c_i is replaced by the
 * conservative lower confidence c_low_i = max{0, c_i - eta_i}, where eta_i
 * >= 0 is a calibration allowance (negative values count as 0), and the
 * profile rule above is applied to the c_low profile (sorted by c_low,
 * ties to the lower position).  With uniform eta and no clipping the score
 * drops by exactly (n+1) eta (the calibration-penalty corollary).  The
 * paper states the robust certificate for a set; the selector takes the
 * largest certified prefix of the c_low order, as the plain rule does.
 *   eta [B,L] float (in, may be NULL: then every eta_i = eta_uniform);
 *   other arguments as for fdllm_select_profile.  eta_uniform must not be NaN.
 */
fdllm_status fdllm_select_robust(const float* conf, const float* eps, const float* eta,
                                 float eta_uniform, const uint8_t* mask, const int32_t* block_start,
                                 const int32_t* block_end, int B, int L, float f, uint8_t* commit,
                                 int32_t* n_commit, fdllm_stream stream);

/*
 * Reveal (Alg. 1, reveal step): for every (b,i) with commit[b,i] != 0 set
 * x[b,i] = tokens[b,i] and mask[b,i] = 0.  Other entries are untouched.
 *   commit [B,L] uint8 (in); tokens [B,L] int32 (in); x [B,L] int32 (in/out);
 *   mask [B,L] uint8 (in/out).
 */
fdllm_status fdllm_reveal(const uint8_t* commit, const int32_t* tokens, int32_t* x, uint8_t* mask,
                          int B, int L, fdllm_stream stream);

/*
 * One whole decoding step (Alg. 1, loop body after the model call):
 * fdllm_confidence, then the selector `sel` with `param` (f, or tau for the
 * threshold rule), then the reveal, fused.  Large batches run as one kernel
 * (one workgroup per sequence); small batches as two kernels.  When a large
 * batch exceeds a multiple of the GPU's compute-unit count by at most 64
 * sequences, those last sequences run with the small-batch kernels on a
 * stream the library keeps per device, at the same time as the one-kernel
 * part; the call stays asynchronous and can be captured into a HIP graph
 * (the side stream is forked from and joined back to `stream` by events).  That needs the workspace, or tokens,
 * conf and eps all given; without either, they run in the one kernel.
 *   eta, eta_uniform: calibration allowance of FDLLM_SEL_ROBUST (as in
 *   fdllm_select_robust); ignored by the other selectors.
 *   mask [B,L] uint8 (in/out: committed positions are cleared);
 *   x    [B,L] int32 (in/out: committed positions receive their token);
 *   tokens, conf, eps, lse [B,L], commit [B,L], n_commit [B]: optional
 *   outputs (NULL to skip), with the meanings above.
 *   workspace: device memory of at least fdllm_workspace_size() bytes
 *   (may be NULL when that size is 0); its contents need no initialisation
 *   and are scratch between calls.  With tokens, conf and eps all given a
 *   smaller workspace (or NULL) is accepted: the results are the same, but a
 *   small batch of blocks of at most 64 positions then streams each row
 *   from one workgroup instead of several.  (The one exception: a large
 *   batch's last sequences, above, run in the one kernel when neither the
 *   workspace nor those three outputs are given; the decisions are the
 *   oracle's either way, but conf, eps and lse of those sequences are then
 *   not bitwise fdllm_confidence's.)
 */
fdllm_status fdllm_decode_step(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                               uint8_t* mask, const int32_t* block_start, const int32_t* block_end,
                               int32_t* x, fdllm_selector sel, float param, const float* eta,
                               float eta_uniform, int32_t* tokens, float* conf, float* eps,
                               float* lse, uint8_t* commit, int32_t* n_commit, void* workspace,
                               size_t workspace_bytes, fdllm_stream stream);

/*
 * fdllm_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same step, with the same arguments minus the workspace, the same plans
 * and bitwise the same results as fdllm_decode_step given a workspace of
 * fdllm_workspace_size() bytes.  The scratch it needs instead lives in the
 * library: a static array of FDLLM_STATIC_SCRATCH_BYTES (8 MiB) on every GPU
 * the library runs on, held until the process ends.  The call allocates and
 * frees nothing.
 *   Sizes whose workspace exceeds FDLLM_STATIC_SCRATCH_BYTES are refused with
 *   FDLLM_ERR_SCRATCH (nothing enqueued).  Small batches need 12 B per
 *   position of the span (when tokens, conf or eps are not given) plus up to
 *   384 B per position of blocks of at most 64 positions; batches of 256
 *   sequences or more need scratch only for the at most 64 sequences beyond a
 *   multiple of the compute-unit count, which run as a small batch.  Those
 *   run on `stream` after the one-kernel part instead of beside it on a side
 *   stream (the call creates no stream and no event), with the same bits.
 *   Every call on one GPU uses that GPU's one array: calls that overlap on one
 *   GPU (other streams, other threads) race and must be serialised by the
 *   caller.  The array keeps the last call's contents; the step needs none of
 *   them (its scratch needs no initialisation).
 *   The first call on a device, with that device current, looks up the
 *   array's device address (hipGetSymbolAddress) once; later calls on that
 *   device reuse it.
 */
fdllm_status fdllm_decode_step_static(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                                      uint8_t* mask, const int32_t* block_start,
                                      const int32_t* block_end, int32_t* x, fdllm_selector sel,
                                      float param, const float* eta, float eta_uniform,
                                      int32_t* tokens, float* conf, float* eps, float* lse,
                                      uint8_t* commit, int32_t* n_commit, fdllm_stream stream);

/*
 * ---------------------------------------------------------------------------
 * LM head fused with the vocabulary pass (Alg. 1: the model call's last
 * layer followed by the per-position confidence)
 * ---------------------------------------------------------------------------
 * The logits of candidate position (b, i) are l_v = sum_k h[b,i,k] W[v,k],
 * formed on the matrix cores with float32 accumulation (bf16 operands) and
 * folded into the online (max, sum, argmax) of the vocabulary pass; no full
 * logit row is stored (for 33..64 positions the two halves of the hidden
 * dimension's partial logits pass through the workspace, 2 x 64 x V floats).
 * From the logits on, the outputs are those of fdllm_confidence (token,
 * conf, eps, lse; defaults for non-candidates).
 *   hidden [B, L, d] bf16, 16-byte aligned (in): final hidden states;
 *   weight [V, d] bf16, 16-byte aligned (in): output embedding, row v for token v;
 *   d: a multiple of 64, hidden at most 4 GiB (B*L*d*2 < 2^32 bytes) and
 *   V*d/8 < 2^31 (FDLLM_ERR_SIZE otherwise);
 *   mask, block_start, block_end: candidates as above;
 *   workspace: at least fdllm_lmhead_workspace_size() bytes of device memory
 *   (FDLLM_ERR_WORKSPACE otherwise), scratch between calls.
 */
fdllm_status fdllm_lmhead_workspace_size(int B, int L, int d, int V, size_t* bytes);
fdllm_status fdllm_lmhead_confidence(const void* hidden, const void* weight, int B, int L, int d,
                                     int V, const uint8_t* mask, const int32_t* block_start,
                                     const int32_t* block_end, int32_t* tokens, float* conf,
                                     float* eps, float* lse, void* workspace,
                                     size_t workspace_bytes, fdllm_stream stream);

/*
 * One decoding step from hidden states: fdllm_lmhead_confidence, then the
 * selector and the reveal as in fdllm_decode_step (same selector arguments;
 * tokens, conf, eps, lse, commit, n_commit optional).
 */
fdllm_status fdllm_lmhead_decode_step(const void* hidden, const void* weight, int B, int L, int d,
                                      int V, uint8_t* mask, const int32_t* block_start,
                                      const int32_t* block_end, int32_t* x, fdllm_selector sel,
                                      float param, const float* eta, float eta_uniform,
                                      int32_t* tokens, float* conf, float* eps, float* lse,
                                      uint8_t* commit, int32_t* n_commit, void* workspace,
                                      size_t workspace_bytes, fdllm_stream stream);

/*
 * ---------------------------------------------------------------------------
 * The decoding loop on the device (Alg. 1 outer loops)
 * ---------------------------------------------------------------------------
 * A generation of B sequences over a span of G positions in blocks of blk:
 * every position starts masked, each sequence works on its first block that
 * still has a masked position, and every step is a model call followed by
 * fdllm_decode_step.  Here the model call is replaced by a synthetic,
 * counter-based logits producer, so the whole loop runs without the host.
 *
 * Synthetic logits (bf16, row-major [B, G, V]).  Philox4x32-10 (Salmon,
 * Moraes, Dror and Shaw, SC 2011) with key (seed mod 2^32, seed >> 32); for
 * row (b, i) at step t and vocabulary index v:
 *   background  w = philox(v >> 2, i, b, t)[v & 3]; (sum of w's 4 bytes - 510) * 2^-7
 *   spike token philox(0xFFFFFFFF, i, b, 0xFFFFFFFF)[0] mod V (fixed over steps)
 *   spike height y = philox(0xFFFFFFFE, i, b, t); u1 = (y[0] >> 8) 2^-24,
 *               u2 = (y[1] >> 8) 2^-24; h = 8 + 6 u2 if u1 < 0.6 else 6 u2
 *   logit       bf16(background + h) at the spike token, bf16(background)
 *               elsewhere; float32 with every operation rounded to nearest,
 *               bf16 by round-to-nearest-even.
 * Only the rows of each sequence's active block are written.
 */

/*
 * Writes the synthetic logits of the rows [block_start[b], block_end[b]) of
 * every sequence b at step `step` (rows beyond blk slots of a window and
 * rows outside it are untouched).
 *   logits [B, L, V] bf16 (out); block_start, block_end [B] int32 (in);
 *   blk: largest window (1..FDLLM_MAX_BLOCK).
 */
fdllm_status fdllm_synth_logits(void* logits, int B, int L, int V, int blk,
                                const int32_t* block_start, const int32_t* block_end,
                                uint64_t seed, int step, fdllm_stream stream);

/*
 * Block advance (Alg. 1: a block is decoded until none of its positions is
 * masked, then the next block starts).  For every sequence, the window moves
 * from its current block to the first block of blk positions at or after it
 * that has a masked position; a sequence with none left gets [G, G).
 *   mask [B, G] uint8 (in); block_start, block_end [B] int32 (in/out:
 *   block_start must be a multiple of blk or G);
 *   n_active [1] int32 (out, may be NULL): sequences left with a block.
 */
fdllm_status fdllm_advance_blocks(const uint8_t* mask, int32_t* block_start, int32_t* block_end,
                                  int B, int G, int blk, int32_t* n_active, fdllm_stream stream);

typedef struct {
  int B, G, blk, V;          /* sequences, span, block size (<= FDLLM_MAX_BLOCK), vocabulary */
  uint64_t seed;             /* synthetic logits generator seed */
  fdllm_selector sel;        /* selector and its parameter (f, or tau), as fdllm_decode_step */
  float param;
  const float* eta;          /* robust rule: [B, G] allowances or NULL */
  float eta_uniform;
  int max_steps;             /* upper bound on steps; G always suffices */
  int chunk;                 /* steps per launch; the host checks for completion between chunks */
  int use_graph;             /* 1: capture `chunk` steps into a HIP graph and replay it;
                                0: launch the kernels of each chunk directly */
  void* logits;              /* [B, G, V] bf16 device buffer; active rows rewritten each step */
  uint8_t* mask;             /* [B, G] out: final mask (all 0 when every block finished) */
  int32_t* x;                /* [B, G] out: generated tokens (-1 where never revealed) */
  int32_t* block_start;      /* [B] scratch/out: final windows */
  int32_t* block_end;        /* [B] */
  int32_t* n_commit_hist;    /* [max_steps, B] out (may be NULL): n_commit of every step */
  void* workspace;           /* >= fdllm_generation_workspace_size() bytes of device memory */
  size_t workspace_bytes;
} fdllm_generation_desc;

typedef struct fdllm_generation_s* fdllm_generation;

/* Device workspace a generation needs (counters, n_commit, decode-step scratch). */
fdllm_status fdllm_generation_workspace_size(const fdllm_generation_desc* desc, size_t* bytes);

/*
 * Prepares a generation: validates the description and, with use_graph,
 * captures `chunk` steps (producer, decode step, advance, step counter) into
 * a HIP graph.  All device memory is the caller's (the description's
 * buffers); the object holds host-side runtime state only (a graph, a
 * capture stream, two events and 64 bytes of pinned host memory).  The
 * buffers must stay valid until fdllm_generation_destroy.
 */
fdllm_status fdllm_generation_create(const fdllm_generation_desc* desc, fdllm_generation* gen);

/*
 * Runs one whole generation on `stream`: resets mask = 1, x = -1, the
 * windows to the first block and the counters, then launches chunks of
 * steps until no sequence has a block left (read back once per chunk, one
 * chunk behind the device) or max_steps is reached.  Blocks until the
 * stream is idle; *steps (host, may be NULL) receives the number of steps
 * in which some sequence still had a block (the NFE).  Runs of one object
 * must not overlap.
 */
fdllm_status fdllm_generation_run(fdllm_generation gen, fdllm_stream stream, int32_t* steps);

/*
 * Releases the object's graph, capture stream, events and pinned memory (all
 * of them, also when one release fails; FDLLM_ERR_HIP then).  NULL is a
 * no-op.  The caller's buffers are not touched.
 */
fdllm_status fdllm_generation_destroy(fdllm_generation gen);

/*
 * Opt-in input check (debug aid; the other entry points never read the
 * logits of non-candidates and do not validate values).  Scans every
 * candidate row (as defined above) for a logit that is NaN, inf or of
 * magnitude above FDLLM_MAX_ABS_LOGIT, and every sequence's window.
 *   logits, dtype, B, L, V, mask, block_start, block_end: as fdllm_confidence;
 *   counts [3] int32 device memory (out): sequences whose window is not
 *   0 <= start <= end <= L; sequences whose window is longer than
 *   FDLLM_MAX_BLOCK; candidate rows holding a bad logit (rows of sequences
 *   with an invalid window are not scanned).
 * Unlike the other entry points this call SYNCHRONISES `stream` and returns
 * the verdict: FDLLM_ERR_BOUNDS, else FDLLM_ERR_BLOCK_TOO_LARGE, else
 * FDLLM_ERR_NONFINITE when the matching count is non-zero, else FDLLM_OK.
 * It reads every candidate logit once (the same traffic as the pass).
 */
fdllm_status fdllm_check_inputs(const void* logits, fdllm_dtype dtype, int B, int L, int V,
                                const uint8_t* mask, const int32_t* block_start,
                                const int32_t* block_end, int32_t* counts, fdllm_stream stream);

/* Workspace bytes fdllm_decode_step needs for these sizes (0 = none) on the
 * current device (the large-batch remainder above depends on its
 * compute-unit count). */
fdllm_status fdllm_workspace_size(int B, int L, int V, fdllm_dtype dtype, size_t* bytes);

/* Static, human-readable text for a status code. */
const char* fdllm_status_string(fdllm_status status);

#ifdef __cplusplus
}
#endif

#endif /* FDLLM_H */
