/*
 * radar.h -- C ABI of the Radar decode path on MI355X (gfx950).
 *
 * Radar ("Radar: Fast Long-Context Decoding for Any Transformer", ICLR 2025)
 * keeps a two-level index over the key cache: the keys are cut into segments
 * of c tokens and every segment is summarised by the mean of the positive
 * random features of its keys (Section 2.2, Eq. 4 and Eq. 5). A decode query
 * is mapped to the same random features, every segment is scored by one dot
 * product (Eq. 6), the top-k segments are selected, and exact softmax
 * attention (Section 2.1, Eq. 1-2) runs over the selected segments' tokens
 * together with the recent tokens that belong to no summarised segment
 * (Appendix A, Algorithm 1).
 *
 * Conventions shared by every call
 * --------------------------------
 *  - Every tensor argument is a DEVICE pointer owned by the caller; `cfg` is a
 *    host pointer. K and V may instead point to pinned host memory mapped
 *    into the device's address space at the same address (hipHostMalloc);
 *    the kernels then read over the host link only the rows a call needs
 *    (a decode: the selected segments, the window and the sinks; an append:
 *    the closed segment it summarises; an index build: every key), and write
 *    appended rows there. Summaries, Omega, q and the outputs stay in device
 *    memory. The library allocates no device memory, keeps no device
 *    state between calls, never synchronises, and launches only on `stream`
 *    (the path override and the profiling switch are host-side settings of
 *    the calling thread). The one device buffer of its own is the scratch
 *    array of radar_append_decode_noalloc, whose contents no call depends on.
 *  - Layouts are dense, row-major, element type `kv_dtype` for q / K / V /
 *    k_new / v_new / out, `omega_dtype` for Omega, fp32 for summaries and
 *    scores, int32 for segment ids:
 *        q, out          [B][Hq][d]
 *        K, V            [B][Hkv][capacity][d]     (token-major per head)
 *        k_new, v_new    [B][Hkv][d]
 *        omega           [n][d]                    (row i is omega_i)
 *        summaries       [B][Hkv][capacity / c][n]
 *        selected        [B][Hq][k]   int32, -1 padded
 *        scores          [B][Hq][k]   fp32,  NaN padded
 *  - Every pointer must be 16-byte aligned.
 *  - Positions are 0-based. "t" is the current context length: tokens
 *    0 .. t-1 are valid in K and V.
 *  - Errors: every argument is checked before anything is launched, so a
 *    call that returns an error has no side effect. A failed launch returns
 *    RADAR_EHIP; radar_last_error() then holds the HIP error text. No C++
 *    exception crosses this boundary.
 *
 * Numerical contract
 * ------------------
 *  phi(x)_i = n^(-1/2) exp(omega_i . x' - |x'|^2 / 2),  x' = x / d^(1/4)
 *  (Eq. 4; omega_i is the i-th row of Omega, and queries and keys are both
 *  scaled by d^(-1/4)). Summaries hold the Eq. 5 means, scores the Eq. 6
 *  dot products, both in fp32. All accumulation is fp32. For bf16 caches the
 *  projection runs on bf16 matrix cores with Omega rounded to bf16 (round to
 *  nearest even); pass a bf16-representable Omega for results that do not
 *  depend on that rounding. exp arguments must stay below ~88 (fp32 range);
 *  unit-scale keys and queries keep them far below.
 *
 * Segments, window and candidates
 * -------------------------------
 *  Segment s covers tokens [s*c, s*c + c); only full segments are summarised.
 *  At a decode step with context length t the recent window is
 *  W = [ws, t) with ws = c * floor(max(0, t - w) / c); it is always attended.
 *  The candidate segments are the n_cand = ws / c segments wholly before ws.
 *  Each query head selects k_eff = min(k, n_cand) of them, ordered by score
 *  descending and then by segment index ascending. With grouped-query
 *  attention (Hq = G * Hkv) every query head of a group attends the union of
 *  the group's selections plus W (RADAR_GQA_UNION), or only its own
 *  selection plus W (RADAR_GQA_PER_HEAD).
 *
 *  Attention sinks (n_sink > 0, as in the sink token of Appendix E): tokens
 *  [0, min(n_sink, t)) are attended by every query head and belong to no
 *  segment. Segment s then covers [n_sink + s*c, n_sink + s*c + c), and the
 *  window rule above applies to the tokens after the sinks:
 *  ws = n_sink + c * floor(max(0, t - n_sink - w) / c) (W is empty while
 *  t <= n_sink). Summary row s still holds segment s.
 *
 *  Ragged batches: radar_decode, radar_decode_exact and radar_attend_selected
 *  take an optional device array lens[B] (int64) of per-sequence context
 *  lengths; the call's t is then their upper bound (grid sizes derive from
 *  it) and sequence b is decoded exactly as a call with t = lens[b] would
 *  decode it. A length outside [1, t] is not checked on the host: that
 *  sequence selects nothing (ids -1, scores NaN) and its outputs are NaN.
 *  radar_append takes pos[B] likewise. Build the index of a ragged batch
 *  with t = the longest length: a segment that a shorter sequence has not
 *  yet filled is summarised again by the append that completes it, before
 *  it can become a candidate.
 */
#ifndef RADAR_H
#define RADAR_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RADAR_ABI_VERSION 7

typedef enum {
  RADAR_OK = 0,
  RADAR_EINVAL = 1,       /* null pointer, bad shape, misaligned pointer    */
  RADAR_ECAPACITY = 2,    /* t or a position outside [.., capacity]         */
  RADAR_EUNSUPPORTED = 3, /* valid but outside the instantiated shapes      */
  RADAR_EHIP = 4,         /* a HIP launch failed; see radar_last_error()    */
  RADAR_EWORKSPACE = 5    /* workspace null or smaller than required        */
} radar_status;

typedef enum { RADAR_F32 = 0, RADAR_BF16 = 1 } radar_dtype;

typedef enum {
  RADAR_GQA_UNION = 0,    /* each head attends its group's union (default)  */
  RADAR_GQA_PER_HEAD = 1  /* each head attends its own selection            */
} radar_gqa;

typedef struct {
  int32_t batch;       /* B >= 1                                            */
  int32_t n_q_heads;   /* Hq; Hq % Hkv == 0, G = Hq / Hkv in {1, 2, 4, 8}   */
  int32_t n_kv_heads;  /* Hkv >= 1; B * Hkv <= 65535                        */
  int32_t head_dim;    /* d in {64, 128}                                    */
  int32_t n_features;  /* n in {64, 128, ..., 2048} (powers of two)         */
  int32_t seg_len;     /* c >= 1 (any value; need not divide anything)      */
  int32_t window;      /* w >= 0                                            */
  int64_t capacity;    /* token rows per head in K and V, 1 .. 2^31 - 1     */
  radar_dtype kv_dtype;
  int32_t n_sink;      /* attention-sink tokens, 0 .. capacity (0: none)    */
  radar_gqa gqa_mode;  /* which segments a grouped query head attends       */
  radar_dtype omega_dtype;  /* element type of Omega: RADAR_F32, or
                          RADAR_BF16 with a bf16 cache only (its projection
                          rounds Omega to bf16 anyway, so a bf16 copy gives
                          the same results and halves the Omega bytes every
                          decode reads); a zero-initialised config means
                          fp32                                             */
} radar_config;

/* Index build (Eq. 4 and Eq. 5; Algorithm 1's restructuring step that
 * pre-computes the segment embeddings). Writes summaries rows
 * 0 .. floor((t - n_sink) / c) - 1 of every (b, kv head) from the rows of K
 * before t. Rows beyond are not touched. Requires 1 <= t <= capacity. */
radar_status radar_build_index(const radar_config* cfg, const void* K,
                               const void* omega, int64_t t,
                               float* summaries, hipStream_t stream);

/* Append one token (Algorithm 1: the new key joins the buffer W). Writes
 * k_new / v_new ([B][Hkv][d]) to row t of K / V. If the row completes a
 * segment (r = t - n_sink >= 0 and (r + 1) % c == 0) the summary of segment
 * (r + 1) / c - 1 is computed with exactly the code path of
 * radar_build_index, so appending and rebuilding give bit-identical
 * summaries. Requires 0 <= t < capacity; the caller's context length
 * becomes t + 1. With pos (nullable, device int64 [B]) sequence b writes
 * row pos[b] instead and t is ignored; a pos[b] outside [0, capacity) is
 * skipped (no write, no summary). */
radar_status radar_append(const radar_config* cfg, void* K, void* V,
                          const void* k_new, const void* v_new,
                          const void* omega, int64_t t, const int64_t* pos,
                          float* summaries, hipStream_t stream);

/* Decode one query per (b, q head) (Algorithm 1, querying step): phi(q)
 * (Eq. 4), scores of the n_cand candidate segments (Eq. 6), top-k, and exact
 * softmax attention (Eq. 1-2) over the selected segments plus W, with the
 * softmax scale 1/sqrt(d). t is the context length including the query's own
 * token (append first, then decode); lens (nullable, device int64 [B])
 * gives per-sequence lengths with t their bound (see Ragged batches).
 * k >= 1. `selected` and `scores` may be NULL. `workspace` must hold at
 * least radar_decode_workspace_bytes(cfg, k) bytes; its contents on entry do
 * not matter and it must not be used by another call at the same time. */
radar_status radar_decode(const radar_config* cfg, const void* q,
                          const void* K, const void* V, const void* omega,
                          const float* summaries, int64_t t,
                          const int64_t* lens, int32_t k, void* out,
                          int32_t* selected, float* scores, void* workspace,
                          size_t workspace_bytes, hipStream_t stream);

/* One decode step with its append (Algorithm 1: the new key joins W, then
 * the query step), the same result as radar_append(..., t - 1, pos, ...)
 * followed by radar_decode(..., t, lens = pos + 1, ...), in fewer kernels:
 * the first per-(b, kv head) kernel of the decode writes the new rows
 * k_new / v_new ([B][Hkv][d]) before the attention reads them, and the
 * summary of a segment the rows complete is computed after the decode, with
 * radar_append's code (that segment lies inside W at this step, so the
 * decode does not read its summary; with w = 0 it would, and the call then
 * runs append, refresh and decode in that order).
 * t: the context length after the append, 1 <= t <= capacity. Without pos
 * every sequence writes row t - 1 and attends t tokens. With pos (nullable,
 * device int64 [B]) sequence b writes row pos[b] (skipped outside
 * [0, capacity), as radar_append) and is decoded at length pos[b] + 1, with
 * t their bound: a pos[b] outside [0, t) makes that sequence's outputs NaN
 * and its ids -1 (see Ragged batches). Everything else as for radar_append
 * and radar_decode; the workspace is radar_decode's. */
radar_status radar_append_decode(const radar_config* cfg, const void* q,
                                 void* K, void* V, const void* k_new,
                                 const void* v_new, const void* omega,
                                 float* summaries, int64_t t,
                                 const int64_t* pos, int32_t k, void* out,
                                 int32_t* selected, float* scores,
                                 void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/* Bytes of the library's own decode scratch (one copy per GPU). */
#define RADAR_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): exactly
 * radar_append_decode, with the same arguments, kernels and results, except
 * that the decode's scratch is a device array of the library's own of
 * RADAR_NOALLOC_SCRATCH_BYTES bytes instead of a caller workspace. The call
 * allocates nothing: each GPU the library runs on holds one copy of the
 * array (placed by the loader with the library's code), found on the first
 * call on that device, until the process ends. `stream` must belong to the
 * current device (else RADAR_EINVAL). A shape and k whose
 * radar_decode_workspace_bytes exceeds RADAR_NOALLOC_SCRATCH_BYTES return
 * RADAR_EWORKSPACE before anything is launched. The array keeps what the
 * last call wrote; no call depends on its contents on entry. Every call on
 * one GPU uses the same array, so calls that may overlap on one GPU (other
 * streams, other host threads) race on it and must be serialised by the
 * caller. */
radar_status radar_append_decode_noalloc(const radar_config* cfg,
                                         const void* q, void* K, void* V,
                                         const void* k_new, const void* v_new,
                                         const void* omega, float* summaries,
                                         int64_t t, const int64_t* pos,
                                         int32_t k, void* out,
                                         int32_t* selected, float* scores,
                                         hipStream_t stream);

/* Exact segment search (the exact-selection ablation of Section 3.3): like
 * radar_decode, but each query head selects the k candidate segments with
 * the largest exact attention mass beta_s = sum over the segment's keys of
 * exp(q . k / sqrt(d)) (the quantity Theorem 2's proof calls beta) instead
 * of the random-feature estimate. It reads every candidate key, O(t) bytes
 * per query: a reference selector for recall measurements, not the fast
 * path. `scores` (nullable) receives ln(beta) of the selected segments.
 * Workspace as for radar_decode; summaries and Omega are not used. */
radar_status radar_decode_exact(const radar_config* cfg, const void* q,
                                const void* K, const void* V, int64_t t,
                                const int64_t* lens, int32_t k, void* out,
                                int32_t* selected, float* scores,
                                void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/* The exact segment masses behind radar_decode_exact's selection, for
 * recall measurements of Radar's selection against the exact segment search
 * (Section 3.3): for every (b, q head), ln(beta_s) of each candidate segment
 * s < n_cand (beta_s = sum over the segment's keys of exp(q . k / sqrt(d)),
 * the beta of Theorem 2's proof), and at index n_cand the same log-sum of
 * the tokens that belong to no candidate segment (the window W and the
 * sinks), which every selection attends; exp(ln_beta - logsumexp(ln_beta))
 * over indices 0 .. n_cand is then each part's share of the full softmax.
 * ln_beta: device fp32 [B][Hq][capacity / c + 1]; entries after index
 * n_cand of a row are not written (a sequence with an invalid length in
 * lens gets -inf at index 0 and nothing else). t and lens as for
 * radar_decode; the summaries, Omega and k are not involved. Needs no
 * workspace. */
radar_status radar_segment_mass(const radar_config* cfg, const void* q,
                                const void* K, int64_t t, const int64_t* lens,
                                float* ln_beta, hipStream_t stream);

/* Scratch bytes radar_decode, radar_append_decode, radar_decode_exact and
 * radar_attend_selected need for this shape and k (0 if cfg is invalid). */
size_t radar_decode_workspace_bytes(const radar_config* cfg, int32_t k);

/* Exact attention over caller-chosen segments (the last step of Algorithm 1
 * with the selection supplied): selected [B][Hq][k] holds segment ids, -1
 * for none; ids outside [0, n_cand) are ignored. Each query head attends the
 * union of its group's ids (or its own ids, RADAR_GQA_PER_HEAD) plus the
 * sinks and W, exactly as radar_decode does; a head that attends no token
 * gets a zero output. lens as for radar_decode. */
radar_status radar_attend_selected(const radar_config* cfg, const void* q,
                                   const void* K, const void* V,
                                   const int32_t* selected, int32_t k,
                                   int64_t t, const int64_t* lens, void* out,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream);

/* Algorithm 1's dynamic restructuring (Section 2.2, Appendix A): the
 * segment length becomes sqrt(t) whenever t is a perfect square, the c
 * segments of c tokens then cover [0, c^2), and later tokens wait in the
 * buffer W until the next perfect square. For context length t >= 1 this
 * writes c = floor(sqrt(t)) to *seg_len and t - c^2 to *window: a config
 * with these two fields makes radar_decode attend exactly Algorithm 1's
 * candidates (the c restructured segments) and buffer W = [c^2, t). At a
 * perfect square the caller rebuilds the summaries with radar_build_index
 * under the new seg_len (summaries then need capacity / c rows for the
 * smallest c used). Host-only; launches nothing. */
radar_status radar_schedule_sqrt(int64_t t, int32_t* seg_len, int32_t* window);

/* Decode paths. The split path runs phi(q), scores, top-k, attention and
 * merge as separate kernels spread over the whole chip; the fused path runs
 * the whole step of one (b, kv head) in R workgroups that each repeat the
 * pair's selection and share its attention (R = 1 when the pairs fill the
 * chip or a step is small; with R > 1 a merge kernel follows); the select
 * path runs phi(q), scores, top-k and union of each pair in one workgroup
 * and then the split path's attention and merge. All compute the same
 * method; their fp32 summation orders differ. */
typedef enum {
  RADAR_PATH_AUTO = 0,   /* fused when the shape fits and either B * Hkv >=
                            #CUs, one pair's step reads <= 256 KB, or a
                            pair's summary rows are <= 384 KB; else select
                            when the rows are <= 384 KB; else scored when
                            G <= 4 and not fp32 with d = 128; split
                            otherwise                                       */
  RADAR_PATH_SPLIT = 1,
  RADAR_PATH_FUSED = 2,  /* used when the shape fits (G <= 4, at most 1024
                            candidate segments, not fp32 with d = 128),
                            else split                                      */
  RADAR_PATH_SELECT = 3, /* used when G <= 4 and at most 1024 candidate
                            segments, else split                            */
  RADAR_PATH_SCORED = 4  /* phi(q) and the scores as the split path's
                            chip-wide kernels, then R workgroups per pair
                            that each take the pair's top-k and union from
                            those scores and share its attention (the fused
                            kernel from its top-k on); used when G <= 4 and
                            not fp32 with d = 128, else split              */
} radar_path;

/* Choose the decode path for later calls from this host thread (default
 * RADAR_PATH_AUTO). For tests and tuning; results stay within tolerance. */
radar_status radar_set_decode_path(int32_t path);

/* The path radar_decode would take for this shape, t (the length, or the
 * bound of a ragged call's lengths) and k on this thread (RADAR_PATH_SPLIT,
 * RADAR_PATH_FUSED or RADAR_PATH_SELECT; -1 if the arguments are invalid). */
int32_t radar_decode_path(const radar_config* cfg, int64_t t, int32_t k);

/* Kernel kinds reported by the measurement hook below. */
typedef enum {
  RADAR_K_APPEND = 0,   /* k/v row write                                   */
  RADAR_K_BUILD = 1,    /* segment summaries (build or segment close)      */
  RADAR_K_PHI_Q = 2,    /* phi(q)                                          */
  RADAR_K_SCORE = 3,    /* Eq. 6 segment scores (exact mass: its kernel)   */
  RADAR_K_TOPK = 4,     /* top-k and per-kv-head union (or given union)    */
  RADAR_K_ATTEND = 5,   /* gather-attention partials                       */
  RADAR_K_COMBINE = 6,  /* merge of the partials                           */
  RADAR_K_FUSED = 7,    /* the whole decode step, fused path               */
  RADAR_K_SELECT = 8,   /* phi(q) to union of one pair, select path        */
  RADAR_K_SCORED = 9,   /* top-k, union, attention from given scores,
                           scored path                                     */
  RADAR_K_COUNT = 10
} radar_kernel;

/* Measurement hook (not part of the method). While enabled on the calling
 * host thread, every kernel the library launches is bracketed by a HIP event
 * pair recorded at that kernel's start and end on its stream. Results do not
 * change. radar_profile_enable(0) stops recording; pending records are kept
 * until read. */
radar_status radar_profile_enable(int32_t on);

/* Waits for the recorded kernels, adds their durations per radar_kernel kind
 * into ms[0 .. n) and their launch counts into launches[0 .. n) (n >=
 * RADAR_K_COUNT; both arrays are host memory, zeroed by this call), and
 * releases the records. Their events stay with the calling thread for the
 * next profiled launches, so a profiled pass that follows another creates
 * no events. */
radar_status radar_profile_read(double* ms, int64_t* launches, int32_t n);

/* Measurement hook (not part of the method): phase clocks of the fused
 * decode kernel (fused, select and scored paths). While a buffer is set on
 * the calling host thread, workgroup w < max_wgs of every such launch writes
 * RADAR_CLOCK_STAMPS readings of the GPU's constant-rate wall clock
 * (hipDeviceAttributeWallClockRate kHz) to clocks[w * RADAR_CLOCK_STAMPS +
 * i]: 0 entry, 1 phi(q) done, 2 segment scores done, 3 top-k and window
 * tiles done, 4 union done, 5 segment tiles done (every wave), 6 output or
 * partial written, 7 unused. Each is taken by the workgroup's first thread
 * after the barrier that ends the phase; a phase the launch does not run
 * keeps the stamp before it. clocks: device memory of max_wgs *
 * RADAR_CLOCK_STAMPS uint64 values, rewritten by every launch (the last
 * launch's stamps remain); clocks = NULL stops. Results do not change. */
#define RADAR_CLOCK_STAMPS 8
radar_status radar_set_phase_clock(uint64_t* clocks, int32_t max_wgs);

/* The rate of that clock on the current device, in kHz (0 on error). */
int64_t radar_wall_clock_khz(void);

/* Measurement microkernels (not part of the method), for reporting the
 * index build against what this GPU sustains: radar_peak_mfma runs dense
 * bf16 16x16x32 matrix-core chains, radar_peak_exp chains of exp2 on the
 * vector ALUs, each over the whole chip for `iters` rounds on `stream`.
 * *work (host) receives the launch's work: FLOP, or exp2 evaluations. The
 * caller times the launch. sink: device buffer of at least
 * radar_peak_sink_floats() floats, overwritten. */
size_t radar_peak_sink_floats(void);
radar_status radar_peak_mfma(int32_t iters, float* sink, double* work,
                             hipStream_t stream);
radar_status radar_peak_exp(int32_t iters, float* sink, double* work,
                            hipStream_t stream);

/* Measurement microkernel (not part of the method), for reporting the decode
 * kernels against the read rate this GPU sustains: one pass of non-temporal
 * 16-byte loads (the loads the decode kernels stream K, V and the summaries
 * with) over `bytes` bytes of the device buffer `buf` (16-byte aligned, a
 * multiple of 16 bytes), on `stream`; the caller times the launch. sink as
 * for radar_peak_mfma. */
radar_status radar_peak_read(const void* buf, size_t bytes, float* sink,
                             hipStream_t stream);

/* Static text for a status code. */
const char* radar_status_string(radar_status status);

/* Text of the last HIP error seen by this thread ("" if none). */
const char* radar_last_error(void);

/* RADAR_ABI_VERSION of the built library. */
int32_t radar_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RADAR_H */
