/*
 * eta.h -- C ABI of the Elastic Threshold Attention (ETA) decode path on
 * AMD Instinct MI355X (gfx950).
 *
 * One decode step of ETA attention for a batch of sequences, each with one new
 * query token per query head, over a KV cache split into contiguous blocks of
 * b tokens:
 *
 *   1. block summaries (built once per cache, at prefill):   mu, sigma, M per full block
 *   2. threshold prediction:                                  tau = concat_h(q_h) W + bias
 *   3. screening of every full block by its score bound against tau_eff = tau - a,
 *      per-head top-1 rescue, GQA union of the surviving blocks
 *   4. shifted-SiLU-gated softmax attention over the surviving blocks plus the
 *      partial tail, split over the union and merged by log-sum-exp.
 *
 * Paper references are to "Elastic Threshold Attention: Learned Contextual
 * Sparsity for Long-Context Decoding" (section / equation / algorithm names).
 *
 * Conventions shared by every entry point
 *   - All data pointers are DEVICE pointers owned by the caller.  The library
 *     allocates no device memory in any entry point; scratch space is the
 *     caller's `workspace`.
 *   - Work is enqueued on the caller's HIP stream (`stream`, a hipStream_t;
 *     NULL = the null stream) and returns without synchronising.  Outputs are
 *     valid once the stream reaches that point.
 *   - Arguments are validated on the host before anything is enqueued.  A
 *     failed call enqueues nothing and returns a non-zero eta_status_t;
 *     eta_last_error_string() names the argument.  Device-side values (the
 *     contents of seq_lens, q, tau, K, V) cannot be checked without a
 *     synchronisation and are not: seq_lens[b] is clamped to
 *     [0, capacity_tokens] before use, so no access leaves the buffers; NaN
 *     in q, tau, K or V propagates to the outputs.
 *   - Supported shapes: head_dim in {64, 128}; block_size in {64, 128};
 *     G = num_q_heads / num_kv_heads in {1, 2, 4, 8}; K/V dtype fp32 or
 *     bf16; q / output dtype fp32 or bf16.  Anything else returns
 *     ETA_ERR_UNSUPPORTED -- there is no fallback path.
 *   - Every device pointer must be 16-byte aligned; K/V strides must keep
 *     token rows 16-byte aligned; the workspace must be 256-byte aligned.
 *   - Functions never throw across the ABI and are safe to call from several
 *     host threads (the error string is per thread).  Calls that share a
 *     workspace must be ordered on one stream.
 */
#ifndef ETA_H_
#define ETA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ETA_OK = 0,
  ETA_ERR_INVALID_ARG = 1,   /* null pointer, bad size, misalignment, inconsistent shapes */
  ETA_ERR_UNSUPPORTED = 2,   /* valid but outside the supported shape / dtype set */
  ETA_ERR_WORKSPACE = 3,     /* workspace missing, misaligned or too small */
  ETA_ERR_HIP = 4            /* a HIP runtime call or kernel launch failed */
} eta_status_t;

/* Element types.  q, K and V are ETA_DT_F32 or ETA_DT_BF16; block-index
 * records (mu, sigma) are ETA_DT_F32, ETA_DT_F16 or ETA_DT_FP8 (8-bit E4M3:
 * bias 7, 3 fraction bits, largest finite 448). */
typedef enum { ETA_DT_F32 = 0, ETA_DT_BF16 = 1, ETA_DT_F16 = 2, ETA_DT_FP8 = 3 } eta_dtype_t;

/*
 * KV cache geometry.  K and V share it.  Element (b, h, t, i) of K lives at
 * k[b*stride_b + h*stride_h + t*stride_t + i] (strides in elements, the head
 * dimension contiguous); the contiguous layout is [batch][num_kv_heads]
 * [capacity_tokens][head_dim].  Token t of sequence b is valid for
 * t < seq_lens[b] <= capacity_tokens.  Block j covers tokens [j*b, (j+1)*b);
 * it is "full" when (j+1)*b <= seq_lens[b] (Sec. "Block-Based Scanning via
 * Dual Metadata Caching": the cache is cut into contiguous blocks of b tokens).
 */
typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t block_size;
  int32_t kv_dtype;            /* eta_dtype_t */
  int64_t capacity_tokens;
  int64_t stride_b, stride_h, stride_t;
} eta_kv_desc_t;

/*
 * Block index (the "Dual Probabilistic-Geometric Block Index" of Sec.
 * "Block-Based Scanning via Dual Metadata Caching"), dimension-major so that a
 * wavefront reading coordinate i of 64 consecutive blocks issues one
 * coalesced load:
 *   mu[((b*num_kv_heads + h)*head_dim + i)*n_blk_cap + j]     centroid
 *   sigma[((b*num_kv_heads + h)*head_dim + i)*n_blk_cap + j]  coordinate std (population)
 *   max_norm[(b*num_kv_heads + h)*n_blk_cap + j]              largest key L2 norm, fp32
 * mu and sigma are stat_dtype: fp32, or fp16 as in the paper's compact record
 * (App. "GQA-Grouped Execution and Compact Metadata Layout": half-precision
 * centroid and standard deviation, fp32 maximum norm).  The statistics are
 * computed in fp32 and rounded to nearest-even when stored as fp16; the bound
 * is evaluated in fp32 either way.  The standard deviation (not the variance)
 * is stored, as the paper does, so small spreads do not underflow in fp16.
 * ETA_DT_FP8 stores mu and sigma as 8-bit E4M3 codes (the FP8 metadata of Sec.
 * "Limitations and Conclusion"): nearest-even rounding of the fp32 statistic,
 * magnitudes from 464 saturated to 448; a quarter of the fp32 record bytes.
 * n_blk_cap >= max(1, capacity_tokens / block_size), n_blk_cap < 2^24 and
 * n_blk_cap <= 131072 (2048 screening tiles of 64 blocks).  A multiple of 4
 * lets screening read four blocks' records per load (any other value is
 * accepted and read one record at a time).
 */
typedef struct {
  void* mu;
  void* sigma;
  float* max_norm;
  int64_t n_blk_cap;
  int32_t stat_dtype;          /* ETA_DT_F32 (0), ETA_DT_F16 or ETA_DT_FP8 */
  int32_t reserved;            /* 0 */
} eta_summary_t;

/* Decode hyper-parameters (Alg. "Hardware-Aligned Block-Sparse Decoding (Inference)"). */
typedef struct {
  float beta;                   /* gate temperature, Eq. (soft_mask); finite, >= 0 */
  float z;                      /* z-score of the bound, Eq. (dual_bound_eq); finite, >= 0 */
  float offset_a;               /* slack: tau_eff = tau - offset_a, used by screen and gate */
  int32_t rescue_window_blocks; /* c: top-1 rescue over blocks [0, min(c, N)); 0 disables; <= 256 */
  int32_t pin_recent_blocks;    /* lwb: the last lwb full blocks are always selected; >= 0 */
  int32_t self_ungated;         /* 1: key seq_len-1 uses S~ = S (Eq. (mult_attn), M_tt = 1) */
  int32_t screen_all;           /* 1: every full block selected (dense gated attention) */
  int32_t num_splits;           /* splits per (sequence, kv head), for several sequences their
                                   average (the splits are dealt to the (sequence, kv head)
                                   groups in proportion to their unions); 0: library default;
                                   <= 1024; 1 with one sequence (or a uniform split layout):
                                   each (sequence, kv head) is decoded by one workgroup that
                                   writes the results itself, with no merge launch (App.
                                   "Chunked Decoding and Two-Stage Reduction", one chunk) */
} eta_decode_params_t;

/*
 * eta_build_block_summaries -- one pass over K that writes mu, sigma, M of
 * every full block of every (sequence, kv head) (Sec. "Block-Based Scanning
 * via Dual Metadata Caching"; the single O(L d) prefill pass of App.
 * "End-to-End Systems Accounting").
 *   kv        cache geometry (num_q_heads is not used but must be valid)
 *   k         keys, kv->kv_dtype, layout of eta_kv_desc_t
 *   seq_lens  device int32 [batch]
 *   out       summary buffers; entries of blocks that are not full are not written
 * Statistics are accumulated in fp32: mean first, then the mean squared
 * deviation from it (two passes over an on-chip copy of the block).
 */
eta_status_t eta_build_block_summaries(const eta_kv_desc_t* kv, const void* k,
                                       const int32_t* seq_lens, const eta_summary_t* out,
                                       void* stream);

/*
 * eta_build_block_summaries_envelope -- as eta_build_block_summaries, with
 * sigma replaced by the sub-block envelope (App. "Sub-Block Variance
 * Envelope", Eq. subblock_envelope_appx): per coordinate i, the largest over
 * the block's contiguous sub-blocks B_m of sub_block tokens of
 *   sqrt( (1/sub_block) * sum_{k in B_m} (k_i - mu_i)^2 ),
 * mu the centroid of the whole block.  The decode path uses it where it uses
 * sigma (the paper's b = 64 configuration).
 *   sub_block  a power of two in [1, block_size]; 0 gives the flat sigma
 *              (sub_block = block_size gives the same values as the flat sigma)
 */
eta_status_t eta_build_block_summaries_envelope(const eta_kv_desc_t* kv, const void* k,
                                                const int32_t* seq_lens, int32_t sub_block,
                                                const eta_summary_t* out, void* stream);

/*
 * eta_update_block_summaries -- incremental decode-time index update (App.
 * "End-to-End Systems Accounting": the metadata update that follows each
 * appended token).  Writes the records of the blocks that became full since
 * an earlier state of the cache: for each sequence b, blocks
 *   prev_lens[b] / block_size  ..  min(seq_lens[b] / block_size,
 *                                      prev_lens[b] / block_size + max_new_blocks) - 1
 * with exactly the values eta_build_block_summaries(_envelope) writes for them;
 * every other entry is left as it is.  The tail is never summarised (it is
 * always attended), so a block's record is emitted once, when it fills.
 *   prev_lens       device int32 [batch], the lengths the index was built for
 *   seq_lens        device int32 [batch], the current lengths
 *   max_new_blocks  >= 0, upper bound on blocks completed per sequence since
 *                   prev_lens (1 for one appended token per step); it sizes the
 *                   grid without reading the lengths on the host
 *   sub_block       0 (flat sigma) or the envelope's sub-block, as above
 * Lengths are clamped to [0, capacity_tokens]; prev_lens[b] > seq_lens[b]
 * writes nothing for b.
 */
eta_status_t eta_update_block_summaries(const eta_kv_desc_t* kv, const void* k,
                                        const int32_t* prev_lens, const int32_t* seq_lens,
                                        int32_t max_new_blocks, int32_t sub_block,
                                        const eta_summary_t* out, void* stream);

/*
 * eta_predict_threshold -- Eq. (tau_pred): tau[b][h] = sum_j qbar[b][j] W[h][j] + bias[h],
 * qbar[b] the concatenation of the num_q_heads query heads of sequence b
 * (post-RoPE queries).  W == NULL gives frozen per-head constants tau[b][h] =
 * bias[h] (Sec. "Runtime Contextuality and Domain-Specific Offline
 * Calibration").
 *   q        [batch][num_q_heads][head_dim], q_dtype (eta_dtype_t)
 *   W        fp32 [num_q_heads][num_q_heads*head_dim] row-major (head-major: row h holds
 *            the weights of head h's threshold, i.e. the (H d) x H matrix of Eq.
 *            (tau_pred) transposed, so that a workgroup predicting a few heads reads
 *            only their rows), or NULL
 *   bias     fp32 [num_q_heads] (required)
 *   tau_out  fp32 [batch][num_q_heads]
 * fp32 accumulation.  head_dim here may be any value in [1, 1024].
 */
eta_status_t eta_predict_threshold(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                   int32_t q_dtype, const void* q, const float* W,
                                   const float* bias, float* tau_out, void* stream);

/*
 * Bytes of workspace eta_decode / eta_decode_predicted need for this geometry,
 * these params and a summary of block capacity n_blk_cap (the n_blk_cap of the
 * eta_summary_t the decode will read: the workspace holds per-block id lists
 * and per-tile counts laid out with that capacity, and the default split count
 * depends on it).  n_blk_cap is checked as eta_summary_t states
 * (>= max(1, capacity_tokens / block_size), <= 131072): ETA_ERR_INVALID_ARG /
 * ETA_ERR_UNSUPPORTED otherwise.  *bytes is host memory, written on success.
 */
eta_status_t eta_decode_workspace_size(const eta_kv_desc_t* kv, int64_t n_blk_cap,
                                       const eta_decode_params_t* p, size_t* bytes);

/*
 * eta_decode -- one ETA decode step (Alg. "Hardware-Aligned Block-Sparse
 * Decoding (Inference)"; GQA-grouped execution of App. "GQA-Grouped Execution
 * and Compact Metadata Layout").  For every sequence b and query head h
 * (kv head g = h / G), with s = 1/sqrt(head_dim), N = floor(T_b / block_size):
 *   bound_j  = s * min(<q,mu_j> + z*sqrt(sum_i q_i^2 sigma_ji^2), |q| M_j)  (Eq. dual_bound_eq)
 *   sel_j    = bound_j >= tau_eff | j >= N - lwb | screen_all
 *   rescue   if no block in [0, min(c, N)) is selected, the first block of that
 *            window with the largest bound is selected (top-1 rescue)
 *   attended = selected full blocks + the tail [N*block_size, T_b)
 *   S_t      = s <q, k_t>,  S~_t = S_t * sigmoid(beta (S_t - tau_eff))     (Eq. mult_attn)
 *   out      = sum_t softmax(S~)_t v_t over the attended tokens
 * A kv block is read from HBM once per (sequence, kv head) if any of its G
 * query heads selected it (GQA union); each head attends only the blocks it
 * selected.  A head that attends nothing (possible only with rescue disabled,
 * no selection and no tail, or T_b = 0) gets a zero output.
 *   q                  [batch][num_q_heads][head_dim], q_dtype
 *   k, v               kv->kv_dtype, layout of eta_kv_desc_t
 *   seq_lens           device int32 [batch]
 *   summ               block index built by eta_build_block_summaries
 *   tau                fp32 [batch][num_q_heads] (eta_predict_threshold output)
 *   out                [batch][num_q_heads][head_dim], q_dtype (bf16: round to nearest even)
 *   block_mask         uint8 [batch][num_q_heads][summ->n_blk_cap]: 1 = block attended
 *                      by that head (threshold, pin or rescue); 0 elsewhere, including
 *                      every entry j >= N
 *   head_token_counts  int32 [batch][num_q_heads] attended tokens per head, or NULL
 *   union_counts       int32 [batch][num_kv_heads] blocks of the GQA union (the full blocks
 *                      read from HBM for that kv head: selected by any of its G query
 *                      heads), or NULL; the count App. "Top-1 Rescue, Tail Handling, and
 *                      Kernel Validation" checks as "GQA union blocks"
 *   workspace          >= eta_decode_workspace_size() bytes, 256-byte aligned
 * Results are deterministic: the same inputs give bitwise-identical outputs.
 */
eta_status_t eta_decode(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q, const void* k,
                        const void* v, const int32_t* seq_lens, const eta_summary_t* summ,
                        const float* tau, const eta_decode_params_t* p, void* out,
                        uint8_t* block_mask, int32_t* head_token_counts, int32_t* union_counts,
                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * eta_decode_predicted -- eta_decode with the threshold predictor of Eq.
 * (tau_pred) fused into the screening launch: tau = concat(q) W + bias (W ==
 * NULL: the frozen constants bias), computed with the same summation order as
 * eta_predict_threshold, so the thresholds are bit-identical to it.  When the
 * screening workgroups' re-reads of W would exceed 64 MiB per step (batch x
 * kv heads x screening tiles x num_q_heads x head_dim x group x 4 bytes; e.g.
 * 32 sequences at 32/8 heads and 64K capacity), the thresholds are predicted
 * once per step in a launch of their own instead, with the same result.  This
 * is one whole decode step of the paper's layer: predict, screen, attend.
 *   W, bias   as in eta_predict_threshold (bias required)
 *   tau_out   fp32 [batch][num_q_heads] receives the thresholds, or NULL
 * Every other argument, the results and the workspace size are as for eta_decode.
 */
eta_status_t eta_decode_predicted(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                                  const void* k, const void* v, const int32_t* seq_lens,
                                  const eta_summary_t* summ, const float* W, const float* bias,
                                  const eta_decode_params_t* p, void* out, uint8_t* block_mask,
                                  int32_t* head_token_counts, int32_t* union_counts,
                                  float* tau_out, void* workspace, size_t workspace_bytes,
                                  void* stream);

/*
 * eta_decode_predicted_noalloc -- eta_decode_predicted for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the same kernels and results, with the
 * workspace taken from a scratch array the library holds on each GPU instead of
 * a caller's buffer.  The call allocates nothing (no hipMalloc, hipFree or
 * allocating library routine); the caller still passes inputs and outputs.
 *   scratch      ETA_DECODE_NOALLOC_SCRATCH_BYTES (32 MiB) per GPU, a device array
 *                in the library, held by each GPU the library runs on until the
 *                process ends; its device address is looked up on the first call
 *                on a device (with that device current)
 *   size limit   a call whose eta_decode_workspace_size() exceeds that size is
 *                rejected with ETA_ERR_WORKSPACE before anything is enqueued (e.g.
 *                32 ragged 64K sequences at 32/8 heads need ~9.6 MB; 8 x 128K at
 *                16/4 heads ~4.5 MB)
 *   contents     no scratch entry needs to start at zero: every value a kernel reads
 *                was written earlier in the same call
 *   concurrency  every call on a GPU shares that GPU's scratch: calls that can
 *                overlap (other streams, other host threads) race and give wrong
 *                results; order them on one stream
 * Every other argument and every result are as for eta_decode_predicted
 * (bit-identical to it at the same arguments).
 */
#define ETA_DECODE_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
eta_status_t eta_decode_predicted_noalloc(const eta_kv_desc_t* kv, int32_t q_dtype,
                                          const void* q, const void* k, const void* v,
                                          const int32_t* seq_lens, const eta_summary_t* summ,
                                          const float* W, const float* bias,
                                          const eta_decode_params_t* p, void* out,
                                          uint8_t* block_mask, int32_t* head_token_counts,
                                          int32_t* union_counts, float* tau_out, void* stream);

/*
 * Offline density-matched calibration of static per-head thresholds (App.
 * "Offline Threshold Calibration via 1/t-Weighted Histograms"; Alg.
 * "Density-Matched Offline Threshold Calibration"): the frozen constants that
 * replace the predictor (eta_predict_threshold with W = NULL) for a stationary
 * deployment.  Over calibration sequences of T steps, step t (0-based) of head
 * h sees the t + 1 causal keys of kv head h / G, and each causal pair (t, s <= t)
 * weighs 1 / (t + 1).  eta_calib_accumulate adds, per head,
 *   hist[h][bin(S)]  += 1 / (t + 1),   S = <q_t, k_s> / sqrt(head_dim),
 *                      bin(S) = floor((S - lo) / w), w = (hi - lo) / num_bins,
 *                      clamped to [0, num_bins)
 *   density[h]       += sigmoid(beta (S - tau[x][h][t])) / (t + 1)
 * in fixed point (units of 2^-40, integer adds, so the sums do not depend on
 * the order of the adds); eta_calib_solve then finds, per head, the c with
 *   sum_b H_b sigmoid(beta (s_b - c)) = density / total      (bisection, fp64)
 * H the normalised histogram, s_b = lo + (b + 1/2) w, total the sum of the
 * weights (sequences x T).  Scores are computed on the matrix cores from bf16
 * q and K with fp32 accumulation.
 */
typedef struct {
  int32_t num_seqs;            /* N sequences in this call's q, k, tau */
  int32_t num_q_heads;
  int32_t num_kv_heads;        /* num_q_heads / num_kv_heads in {1, 2, 4, 8} */
  int32_t head_dim;            /* 64 or 128 */
  int32_t seq_len;             /* T >= 1 steps (= keys) per sequence */
  int32_t dtype;               /* q and K element type: ETA_DT_BF16 */
  float beta;                  /* gate inverse temperature, finite, > 0 */
  float lo, hi;                /* histogram range of raw scores, finite, lo < hi */
  int32_t num_bins;            /* 1 .. 4096 */
} eta_calib_desc_t;

/* Accumulators, device memory owned by the caller, zeroed before the first
 * eta_calib_accumulate; sequences x T per head must stay below 2^23. */
typedef struct {
  uint64_t* hist;              /* [num_q_heads][num_bins] */
  uint64_t* density;           /* [num_q_heads] */
} eta_calib_state_t;

/*
 * eta_calib_accumulate -- add N calibration sequences to the accumulators.
 *   q    bf16 [num_seqs][num_q_heads][seq_len][head_dim] (the query of every step)
 *   k    bf16 [num_seqs][num_kv_heads][seq_len][head_dim]
 *   tau  fp32 [num_seqs][num_q_heads][seq_len]  the dynamic thresholds of the steps
 *        (e.g. eta_predict_threshold over the steps' concatenated queries)
 * All pointers 16-byte aligned; tensors contiguous.
 */
eta_status_t eta_calib_accumulate(const eta_calib_desc_t* cd, const void* q, const void* k,
                                  const float* tau, const eta_calib_state_t* st, void* stream);

/*
 * eta_calib_solve -- the static threshold of every head.
 *   c_out       fp32 [num_q_heads]
 *   target_out  fp64 [num_q_heads] or NULL: the target density density / total
 * A head with nothing accumulated gets NaN.
 */
eta_status_t eta_calib_solve(const eta_calib_desc_t* cd, const eta_calib_state_t* st,
                             float* c_out, double* target_out, void* stream);

/*
 * Gated prefill / training forward (App. "Hardware-Aligned Forward Kernel"):
 * for every sequence b, query head h (kv head h / G) and row i < seq_lens[b],
 * over the causal keys j <= i:
 *   S_ij = <q_i, k_j> / sqrt(head_dim),  sigma_ij = sigmoid(beta (S_ij - tau_i))
 *   S~_ij = S_ij sigma_ij, or S_ij + C sigma_ij - C when additive; S~_ii = S_ii
 *   out_i = sum_j softmax_j(S~_ij) v_j,  R_i = sum_j sigma_ij,  L_i = log sum_j exp(S~_ij)
 * Rows i >= seq_lens[b] (up to capacity_tokens): out 0, R 0, L -inf.  Scores
 * and p.V on the matrix cores (bf16 operands, fp32 accumulation; the softmax
 * weights are rounded to bf16 for p.V), everything else fp32.
 *   q, out   bf16 [batch][num_q_heads][capacity_tokens][head_dim]
 *   k, v     bf16 [batch][num_kv_heads][capacity_tokens][head_dim]
 *   tau      fp32 [batch][num_q_heads][capacity_tokens]  per-row thresholds
 *   R, L     fp32 [batch][num_q_heads][capacity_tokens]
 *   seq_lens device int32 [batch]
 */
typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;        /* num_q_heads / num_kv_heads in {1, 2, 4, 8} */
  int32_t head_dim;            /* 64 or 128 */
  int32_t capacity_tokens;     /* rows per (sequence, head) in every tensor, >= 1 */
  int32_t dtype;               /* q, k, v, out: ETA_DT_BF16 */
  float beta;                  /* finite, >= 0 */
  int32_t additive;            /* 0: multiplicative gate S sigma; 1: S + C sigma - C */
  float C;                     /* additive mask depth, finite (ignored when multiplicative) */
} eta_prefill_desc_t;

eta_status_t eta_gated_prefill(const eta_prefill_desc_t* pd, const void* q, const void* k,
                               const void* v, const float* tau, const int32_t* seq_lens,
                               void* out, float* R, float* L, void* stream);

/*
 * eta_block_bounds -- the screening bound of Eq. (dual_bound_eq) for every
 * full block and query head, as eta_decode computes it, without selecting or
 * attending.  For threshold calibration and diagnostics.
 *   bounds  fp32 [batch][num_q_heads][summ->n_blk_cap]; NaN for j >= N
 */
eta_status_t eta_block_bounds(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                              const int32_t* seq_lens, const eta_summary_t* summ, float z,
                              float* bounds, void* stream);

/* Bytes of workspace eta_dense_decode needs. */
eta_status_t eta_dense_workspace_size(const eta_kv_desc_t* kv, int32_t num_splits, size_t* bytes);

/*
 * eta_dense_decode -- plain softmax attention decode over all T_b tokens (the
 * dense attention output of Sec. "Elastic Threshold Attention"), split over
 * the context and merged by log-sum-exp: the dense baseline the ETA path is
 * measured against (the paper compares with FlashAttention-2 decode).  Same
 * layouts as eta_decode; num_splits 0 = library default.
 */
eta_status_t eta_dense_decode(const eta_kv_desc_t* kv, int32_t q_dtype, const void* q,
                              const void* k, const void* v, const int32_t* seq_lens, void* out,
                              int32_t num_splits, void* workspace, size_t workspace_bytes,
                              void* stream);

/* Human-readable detail of the last failure on this host thread ("" if none). */
const char* eta_last_error_string(void);

/* ABI version of this header: 5 (2: eta_summary_t carries the record type;
 * 3: ETA_DT_FP8 records; 4: eta_decode / eta_decode_predicted return the
 * per-(sequence, kv head) union counts; 5: eta_decode_workspace_size takes the
 * summary's n_blk_cap, which is at least 1). */
int32_t eta_abi_version(void);

/*
 * Kernel timing.  Between eta_profile_begin() and eta_profile_end(), every
 * kernel the library launches is bracketed by a pair of HIP events recorded
 * on the launch stream (at most 65536 launches).  eta_profile_end waits for
 * the events and writes, per kernel kind, the summed duration in milliseconds
 * and the launch count.
 */
typedef enum {
  ETA_KERNEL_SUMMARIES = 0,
  ETA_KERNEL_PREDICT = 1,
  ETA_KERNEL_SCREEN = 2,
  ETA_KERNEL_SPLIT_DECODE = 3,
  ETA_KERNEL_COMBINE = 4,
  ETA_KERNEL_DENSE_SPLIT = 5,
  ETA_KERNEL_DENSE_COMBINE = 6,
  ETA_KERNEL_BOUNDS = 7,
  ETA_KERNEL_CALIB_ACCUMULATE = 8,
  ETA_KERNEL_CALIB_SOLVE = 9,
  ETA_KERNEL_PREFILL = 10,
  ETA_KERNEL_KINDS = 11
} eta_kernel_kind_t;

typedef struct {
  double ms_total;
  int64_t launches;
} eta_kernel_time_t;

eta_status_t eta_profile_begin(void);
eta_status_t eta_profile_end(eta_kernel_time_t* out /* [ETA_KERNEL_KINDS] */);

#ifdef __cplusplus
}
#endif

#endif /* ETA_H_ */
