/*
 * moeq -- forward pass of one pruned, mixed-precision, block-quantized
 * Mixture-of-Experts layer on an AMD Instinct MI355X (gfx950).
 *
 * The layer is the compressed DeepSeek MoE block of "Collaborative
 * Compression for Large-Scale MoE Deployment on Edge" (arXiv 2509.25689):
 *
 *   - expert pruning (Section 3.1) leaves a subset of the routed experts; the
 *     survivors are given here as a mask over the original expert ids;
 *   - activation adjustment (Section 3.2) sets how many experts each token
 *     activates (top_k) and how grouped routing restricts them (topk_group);
 *   - mixed-precision quantization (Section 3.3) gives every weight tensor
 *     its own low bit width.  This library stores tensors in a symmetric
 *     block format (32 weights per binary16 scale, 2/3/4-bit codes, and
 *     5/6/8-bit codes for the tensors the allocation upgrades) instead
 *     of the paper's llama.cpp formats;
 *   - each expert is a SwiGLU feed-forward network and the layer output is
 *     the routing-weighted sum of the chosen experts plus the shared
 *     expert(s) (Fig. 1, middle).
 *
 * Weight format ("canonical packing", the only layout callers ever see):
 *   a tensor is a row-major [rows x K] matrix, K a multiple of 32.  Every run
 *   of 32 consecutive weights in a row (a block) has one scale d (binary16 bit
 *   pattern) and every weight a b-bit code c; the weight's value is
 *   d * (c - 2^(b-1)).  The 32 codes of a block form one little-endian bit
 *   string of 32*b bits: code i occupies bits [i*b, i*b + b).  Blocks follow
 *   each other along the row, rows follow each other; scales are a separate
 *   row-major [rows x K/32] array.  Projections: 0 = gate [inter x hidden],
 *   1 = up [inter x hidden], 2 = down [hidden x inter].
 *
 * Conventions for every entry point:
 *   - return value: MOEQ_OK or a negative moeq_status; nothing is thrown
 *     across this interface.  moeq_last_error() gives the calling thread's
 *     text for its last failing call;
 *   - every argument and configuration check happens on the host before any
 *     HIP runtime call, so all validation errors are reported the same way on
 *     a machine without a GPU;
 *   - "DEVICE" pointers are HIP device memory on the device the layer was
 *     created on (that device must be current when calling); "HOST" pointers
 *     are ordinary host memory;
 *   - stream arguments are hipStream_t values passed as void*; NULL means the
 *     default stream.  Work is enqueued asynchronously; no entry point except
 *     moeq_layer_create, moeq_set_router_weight and moeq_destroy synchronizes
 *     the host;
 *   - a layer handle owns one workspace, so calls on one handle must not run
 *     concurrently on different streams.
 */
#ifndef MOEQ_H
#define MOEQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MOEQ_OK = 0,
  MOEQ_ERR_INVALID_ARG = -1,   /* a NULL pointer, an out-of-range value, an inconsistent config */
  MOEQ_ERR_UNSUPPORTED = -2,   /* valid in the format but not supported by these kernels */
  MOEQ_ERR_OUT_OF_MEMORY = -3, /* a device allocation failed */
  MOEQ_ERR_DEVICE = -4,        /* a HIP runtime call or a kernel launch failed */
  MOEQ_ERR_CAPACITY = -5       /* n_tokens exceeds the layer's max_tokens */
} moeq_status;

enum { MOEQ_PROJ_GATE = 0, MOEQ_PROJ_UP = 1, MOEQ_PROJ_DOWN = 2 };
enum { MOEQ_WEIGHTS_HOST = 0, MOEQ_WEIGHTS_DEVICE = 1 };
enum { MOEQ_PATH_AUTO = 0, MOEQ_PATH_DECODE = 1, MOEQ_PATH_PREFILL = 2 };

typedef struct moeq_layer moeq_layer; /* opaque; owns every device buffer it allocates */

/* Layer configuration.
 *   hidden, inter   H and I; both multiples of 128 (the format needs 32, the
 *                   kernels' 128-weight units need 128: else UNSUPPORTED)
 *   n_experts       E, routed experts before pruning (= mask length), 1..1024,
 *                   a multiple of n_group
 *   n_shared        shared experts, 0..4; always active, weight 1
 *   n_group         routing groups: experts [g*E/G, (g+1)*E/G) form group g
 *   topk_group      groups each token may draw from (Section 3.2), 1..n_group
 *   top_k           experts per token (num_experts_per_tok), 1..32
 *   group_topn      best scores summed into a group's score, >= 1 (V3: 2)
 *   norm_topk       1: weights are the chosen sigmoid scores renormalised to
 *                   sum to 1, then times routed_scale; 0: scores times routed_scale
 *   routed_scale    the routed scaling factor (V3: 2.5), finite
 *   max_tokens      largest n_tokens a forward may use; sizes the workspace
 *   decode_max_tokens  forward takes the decode path (dequant-GEMV) for
 *                   n_tokens <= this and the prefill path (grouped GEMM on
 *                   MFMA) above it; 0 selects the library default (64).
 *                   From 24 tokens on, the decode path sends the buckets of
 *                   more than 2 tokens to the grouped GEMMs as well
 *   regroup         0: routing groups are the original id ranges with pruned
 *                   experts masked; 1: the kept experts, in ascending id order,
 *                   are cut into n_group equal contiguous groups (Section 3.2's
 *                   partition of the pruned expert pool; the kept count must be
 *                   a multiple of n_group)
 */
typedef struct {
  int32_t hidden;
  int32_t inter;
  int32_t n_experts;
  int32_t n_shared;
  int32_t n_group;
  int32_t topk_group;
  int32_t top_k;
  int32_t group_topn;
  int32_t norm_topk;
  float routed_scale;
  int32_t max_tokens;
  int32_t decode_max_tokens;
  int32_t regroup;
} moeq_config;

/* One quantized tensor in the canonical packing described above.
 *   bits    2, 3, 4, 5, 6 or 8 (any tensor may take any of them)
 *   codes   rows * K * bits / 8 bytes
 *   scales  rows * K / 32 binary16 bit patterns */
typedef struct {
  int32_t bits;
  const void* codes;
  const void* scales;
} moeq_qtensor;

/* Build a layer (Sections 3.1-3.3: the pruned expert set, the routing
 * hyper-parameters and the per-tensor bit widths).
 *   cfg          HOST; copied
 *   expert_mask  HOST uint8 [n_experts]; nonzero = expert kept by pruning
 *   score_bias   HOST float [n_experts] added to the sigmoid scores for
 *                selection only, or NULL for zeros
 *   routed       [n_experts * 3] descriptors, index e*3 + proj; entries of
 *                pruned experts are ignored (may be zeroed)
 *   shared       [n_shared * 3] descriptors, index s*3 + proj; NULL if n_shared = 0
 *   weights_location  MOEQ_WEIGHTS_HOST: codes/scales are HOST pointers;
 *                MOEQ_WEIGHTS_DEVICE: DEVICE pointers on the current device
 *   out          receives the handle
 * The routing must be feasible: topk_group must not exceed the number of
 * groups with a kept expert, and the topk_group smallest non-empty groups
 * must hold at least top_k kept experts (with regroup: topk_group groups of
 * kept / n_group experts must hold top_k) (else INVALID_ARG).
 * All weight data is copied and re-laid-out on the device; the caller may
 * free its buffers when this returns.  The copies and the re-layout run on
 * the null stream, which create waits for before it returns (DEVICE weights
 * must be complete in null-stream order).
 * Errors: INVALID_ARG (including widths outside {2,3,4,5,6,8}), UNSUPPORTED
 * (shapes), OUT_OF_MEMORY, DEVICE;
 * on error *out is set to NULL and nothing is leaked. */
moeq_status moeq_layer_create(const moeq_config* cfg, const uint8_t* expert_mask,
                              const float* score_bias, const moeq_qtensor* routed,
                              const moeq_qtensor* shared, int32_t weights_location,
                              moeq_layer** out);

/* The layer forward (the whole hot path: route, bucket, expert products,
 * SwiGLU, weighted combine, shared expert).
 *   x        DEVICE bfloat16 [n_tokens x hidden], row-major
 *   logits   DEVICE float32 [n_tokens x n_experts] router logits (finite), or
 *            NULL when a router weight is set: the forward then first
 *            computes them as moeq_router_logits does, into layer memory
 *   n_tokens 0..max_tokens; 0 enqueues nothing and returns OK
 *   y        DEVICE float32 [n_tokens x hidden]; fully overwritten
 * Borrowed pointers must stay valid until the stream work completes.  No
 * allocation, no memset, no host synchronization: safe to capture in a HIP
 * graph.  For 2..64 tokens on the decode path, and on the prefill path,
 * part of the work runs on an auxiliary stream (one per device, shared by
 * the device's layers, default priority), ordered after `stream` by an event
 * of the layer and joined back into `stream` by another before the forward's
 * last kernels, so all of it completes in `stream` order (a capture records
 * the fork and join).  Deterministic: identical inputs give bitwise-identical y.
 * Arithmetic: code values are exact; products accumulate in float32.  x and
 * the SwiGLU activations h enter the products in binary16 after power-of-two
 * prescales that put the largest magnitude of each group in [2^14, 2^15).
 * The groups are blocks of 32 on the decode path, except x of the buckets of
 * 2-64 tokens, which stays bfloat16.  On the prefill path they are tokens for
 * x and rows for h.  x is therefore exact, except values more than 2^28
 * below their group's largest.  h is rounded once to 11 significant bits.  The per-token error max|y - y_exact| / max|y_exact| is
 * about 2e-4 on synthetic layers.
 * Errors: INVALID_ARG, CAPACITY (n_tokens > max_tokens), DEVICE. */
moeq_status moeq_forward(moeq_layer* layer, const void* x, const float* logits,
                         int32_t n_tokens, float* y, void* stream);

/* The router's gate weight W_r, so that a forward needs only x: the logits
 * l = x W_r^T are the token-to-expert affinities whose sigmoid the router of
 * Section 3.2 (and the statistics of Section 3.1) score.
 *   w         float32 [n_experts x hidden], row-major, finite; HOST or
 *             DEVICE (current device) per location (MOEQ_WEIGHTS_*); NULL
 *             removes the weight and frees its memory
 * Copied; the caller may free w on return.  Allocates, on the first set,
 * n_experts * hidden * 4 bytes for the weight and max_tokens * n_experts * 4
 * for the logits a forward computes.  Synchronizes the device (do not call
 * while a forward of this layer is being captured).
 * Errors: INVALID_ARG (location, a non-finite HOST element), OUT_OF_MEMORY,
 * DEVICE. */
moeq_status moeq_set_router_weight(moeq_layer* layer, const float* w, int32_t location);

/* The gate alone: logits = x W_r^T with the set weight, float32 products and
 * sums.  Each logit is accumulated in a fixed order that depends only on
 * whether n_tokens <= 8 (one streaming pass per expert, per-thread partial
 * sums over strided columns combined by a fixed tree) or not (one fused
 * multiply-add chain over the hidden index), so results are deterministic.
 *   x        DEVICE bfloat16 [n_tokens x hidden], 16-byte aligned
 *   n_tokens 0..max_tokens
 *   logits   DEVICE float32 [n_tokens x n_experts] (written)
 * Errors: INVALID_ARG (no weight set, arguments), CAPACITY, DEVICE. */
moeq_status moeq_router_logits(moeq_layer* layer, const void* x, int32_t n_tokens, float* logits,
                               void* stream);

/* Frees everything the layer owns after synchronizing the device (the handle
 * does not know every stream its calls ran on).  NULL-safe. */
void moeq_destroy(moeq_layer* layer);

/* Text for the calling thread's last failing call ("" if none). */
const char* moeq_last_error(void);

/* Choose the forward path: MOEQ_PATH_AUTO (by decode_max_tokens),
 * MOEQ_PATH_DECODE or MOEQ_PATH_PREFILL (any n_tokens).  INVALID_ARG otherwise. */
moeq_status moeq_set_path(moeq_layer* layer, int32_t path);

/* Diagnostic: the router stage of the forward alone (Section 3.2 grouped
 * top-k over the experts kept by Section 3.1).  Runs the same device code
 * the forward would run for this n_tokens.
 *   logits  DEVICE float32 [n_tokens x n_experts]
 *   idx     DEVICE int32 [n_tokens x top_k]: chosen experts, best first
 *   w       DEVICE float32 [n_tokens x top_k]: their combine weights */
moeq_status moeq_route(moeq_layer* layer, const float* logits, int32_t n_tokens,
                       int32_t* idx, float* w, void* stream);

/* Diagnostic: the bucketing stage alone, on given expert ids.
 *   idx      DEVICE int32 [n_tokens x top_k]; every id a kept expert, ids of
 *            one token distinct (as the router produces)
 *   offsets  DEVICE int32 [n_experts + 1]: exclusive prefix sum of counts
 *   perm     DEVICE int32 [n_tokens * top_k]: value t*top_k + j, ordered by
 *            expert, then token */
moeq_status moeq_bucket(moeq_layer* layer, const int32_t* idx, int32_t n_tokens,
                        int32_t* offsets, int32_t* perm, void* stream);

/* Diagnostic: one stored tensor decoded to float32 (exact: d * (c - 2^(b-1))).
 *   expert   0..n_experts-1 (a kept expert) or -1 - s for shared expert s
 *   proj     MOEQ_PROJ_*
 *   out      DEVICE float32 [rows x K] */
moeq_status moeq_dequant(moeq_layer* layer, int32_t expert, int32_t proj, float* out,
                         void* stream);

/* Diagnostic: one stored tensor through one of the decoders the products use
 * (each width's code unpacking of Section 3.3's per-tensor formats), so each
 * can be compared with the format's definition d * (c - 2^(b-1)).
 *   decoder  MOEQ_DECODER_EXACT: the bfloat16-form unpacking (the matrix-vector
 *            kernels for 5/6/8-bit tensors),
 *            out = float32 [rows x K], exact (this is moeq_dequant);
 *            MOEQ_DECODER_GEMV_SUBNORMAL: the binary16-subnormal code pairs
 *            (the 2-4-bit gate/up and down matrix-vector kernels), each code
 *            rebuilt from its pair value c * 2^(k-24),
 *            out = float32 [rows x K], exact; widths 2-4 only (else
 *            UNSUPPORTED);
 *            MOEQ_DECODER_GEMM_F16: the grouped GEMMs' weight decoder, out =
 *            binary16 bit patterns (uint16) [rows x K] of d * (c - 2^(b-1))
 *            rounded once to nearest even, the value the matrix cores use
 *   expert, proj as for moeq_dequant; out DEVICE
 * Errors: INVALID_ARG, UNSUPPORTED, DEVICE. */
enum { MOEQ_DECODER_EXACT = 0, MOEQ_DECODER_GEMV_SUBNORMAL = 1, MOEQ_DECODER_GEMM_F16 = 2 };
moeq_status moeq_dequant_as(moeq_layer* layer, int32_t expert, int32_t proj, int32_t decoder, void* out,
                            void* stream);

/* Quantize a float32 matrix into the canonical format (Section 3.3's
 * "quantize to the base precision" step, in this library's block format):
 * per block d = binary16(max|w| / (2^(b-1)-1)) rounded to nearest even from
 * the exact quotient, codes clamp(rint(w/d)) + 2^(b-1) (ties to even; all
 * codes 2^(b-1) when d = 0).
 *   w       DEVICE float32 [rows x K], K a multiple of 32, finite
 *   bits    2, 3, 4, 5, 6 or 8
 *   codes   DEVICE [rows * K * bits / 8] bytes
 *   scales  DEVICE uint16 [rows * K / 32] */
moeq_status moeq_quantize(const float* w, int32_t rows, int32_t K, int32_t bits,
                          void* codes, uint16_t* scales, void* stream);

/* Sizes: weight bytes as stored (codes plus scales of every kept expert and
 * shared expert) and workspace bytes.  Either pointer may be NULL. */
moeq_status moeq_layer_bytes(const moeq_layer* layer, uint64_t* weight_bytes,
                             uint64_t* workspace_bytes);

/* Expert importance and the pruning mask (Section 3.1): the statistics of the
 * unpruned router over calibration tokens.  Every expert is kept for routing;
 * cfg's grouped top-k fields and score_bias apply as in a forward.  For each
 * expert e:
 *   f_e    = (tokens that selected e) / n_tokens            (float32)
 *   sbar_e = mean sigmoid score of e over those tokens, 0 if none (float32;
 *            the scores are summed in float32 in token order)
 *   I_e    = alpha * f_e + (1 - alpha) * sbar_e              (float64, two
 *            products and one sum, each rounded)
 * and mask_e = 1 for the ceil(retain * E) experts with the largest I_e (ties:
 * lower id first; the product is taken with a 1e-9 tolerance so that e.g.
 * 0.7 * 10 keeps 7).  The result is deterministic.
 *   cfg         HOST; a valid layer configuration (its routing fields are used)
 *   score_bias  HOST float [n_experts] or NULL (zeros); copied before return
 *   logits      DEVICE float32 [n_tokens x n_experts], finite
 *   n_tokens    1..2^24
 *   alpha       in [0, 1]; retain in (0, 1]
 *   importance  DEVICE double [n_experts] (written)
 *   mask        DEVICE uint8 [n_experts] (written): usable as create's expert_mask
 *   counts      DEVICE int32 [n_experts] (written) or NULL
 * Scratch memory (about 16 * n_tokens * top_k bytes) is allocated and released
 * in stream order; nothing synchronizes the host.
 * Errors: INVALID_ARG (arguments, configuration, routing infeasible with all
 * experts kept), OUT_OF_MEMORY (scratch), DEVICE. */
moeq_status moeq_expert_importance(const moeq_config* cfg, const float* score_bias, const float* logits,
                                   int32_t n_tokens, double alpha, double retain, double* importance,
                                   uint8_t* mask, int32_t* counts, void* stream);

/* moeq_expert_importance without any allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops, hosts
 * that forbid hipMalloc): identical arguments, results and errors, but the
 * scratch lives in a 16 MiB array compiled into the library, one per device,
 * held until the process ends.  The scratch of a call is
 *   the sum, each part rounded up to a multiple of 256, of
 *                       16 * n_tokens * top_k  (ids, weights, ranks, permutation)
 *                     + 4 * ceil(n_tokens / 64) * n_experts  (per-chunk counts)
 *                     + 13 * n_experts + 8  (offsets, active list, mask, bias)
 * bytes; a call that needs more than 16 MiB returns CAPACITY (e.g. about
 * 100k tokens at top_k 8 over 256 experts fit).  The array keeps the last
 * call's contents and no part of it needs to start cleared.  Calls on one
 * device share the array, so calls that overlap in time on one device (two
 * streams, or two host threads) race: order them on one stream.  The first
 * call on a device looks up the array's device address (no allocation).
 * Errors: INVALID_ARG, CAPACITY, DEVICE. */
moeq_status moeq_expert_importance_noalloc(const moeq_config* cfg, const float* score_bias, const float* logits,
                                           int32_t n_tokens, double alpha, double retain, double* importance,
                                           uint8_t* mask, int32_t* counts, void* stream);

/* ---- Mixed-precision bit allocation (Section 3.3), host only ----------------
 * These entry points run on the host, make no HIP call and need no device.
 *
 * Sensitivity of each tensor (Section 3.3's tensor-level analysis):
 *   sens[t] = (ppl_low - ppl_high[t]) / rho_t,  rho_t = params[t] / layer_params[t]
 * in float64 (rho_t first, then one subtraction and one division).
 *   ppl_low       perplexity with every tensor at the base width
 *   ppl_high      HOST double [n]: perplexity with tensor t alone raised
 *   params, layer_params  HOST int64 [n], positive, params[t] <= layer_params[t]
 *   sens          HOST double [n] (written)
 * Errors: INVALID_ARG (NULL, n < 0, non-finite perplexity, bad counts). */
moeq_status moeq_sensitivity(int32_t n, double ppl_low, const double* ppl_high, const int64_t* params,
                             const int64_t* layer_params, double* sens);

/* The order in which rule 3 of the back-off visits MoE layers: a breadth-first
 * binary partition of the layer positions 0..n_layers-1 over half-open
 * intervals [lo, hi), each contributing position ceil((lo + hi) / 2) (lo for an
 * interval of one) and splitting into [lo, mid) and [mid + 1, hi).  For 58
 * layers it begins 29, 15, 44, 8, 23, 37, 52.
 *   order  HOST int32 [n_layers] (written), n_layers 1..4096 */
moeq_status moeq_layer_order(int32_t n_layers, int32_t* order);

/* Tensor kinds for moeq_plan_bits. */
enum {
  MOEQ_TENSOR_OTHER = 0,        /* may be upgraded by its size tier */
  MOEQ_TENSOR_ROUTED_GATE = 1,  /* routed-expert tensors: never upgraded, */
  MOEQ_TENSOR_ROUTED_UP = 2,    /* lowered to Q_low' by rule 3 */
  MOEQ_TENSOR_ROUTED_DOWN = 3
};

#define MOEQ_PLAN_MAX_LEVELS 8

/* The width ladder and budget of a plan.  Widths are bits per weight,
 * scales included, in units of 1/64 bit (so 1.75 -> 112, 4.5 -> 288), strictly
 * increasing.  Level indices satisfy low_prime < low < floor <= medium_level
 * <= small_level < n_levels. */
typedef struct {
  int32_t n_levels;                       /* 3..MOEQ_PLAN_MAX_LEVELS */
  int32_t width64[MOEQ_PLAN_MAX_LEVELS];  /* 1..4096 each */
  int32_t low_prime;                      /* Q_low': rule 3's target for routed experts */
  int32_t low;                            /* Q_low: every tensor's starting width */
  int32_t floor;                          /* Q4: no upgraded tensor ends below it */
  int32_t small_level;                    /* target below small_params parameters (Q8) */
  int32_t medium_level;                   /* target up to medium_params parameters (Q6) */
  int64_t small_params;                   /* 10,000,000 in the paper */
  int64_t medium_params;                  /* 50,000,000 in the paper */
  uint64_t m_limit_bytes;                 /* M_limit, at most 2^50 */
  int32_t n_moe_layers;                   /* positions of routed tensors: 0..n_moe_layers-1 */
} moeq_plan_params;

/* Budget figures of a plan; GB are 10^9 bytes. */
typedef struct {
  double s_low_gb;     /* S_low: every tensor at Q_low */
  double b_base_gb;    /* B_base = M_limit - S_low */
  double b_delta_gb;   /* released by rule 3 (sum of B_delta) */
  double b_total_gb;   /* B_base + b_delta */
  double upgrade_gb;   /* the upgrades' extra bytes, <= b_total when feasible */
  double total_gb;     /* size of the planned model */
  int32_t n_upgraded;  /* tensors left above Q_low */
  int32_t n_rule2;     /* one-level downgrades of earlier upgrades */
  int32_t n_rule3;     /* routed tensors lowered to Q_low' */
  int32_t feasible;    /* 1 if total <= M_limit */
} moeq_plan_report;

/* Dynamic allocation with back-off (Section 3.3): every tensor starts at
 * Q_low; tensors that are not routed experts are taken in descending
 * sensitivity (ties: lower index first) and raised to small_level (fewer than
 * small_params parameters) or medium_level (up to medium_params; larger ones
 * are not raised) while the upgrades' extra bits fit B_total.  When one does
 * not fit: (1) it is tried one, then two levels lower (not below floor);
 * (2) failing that, the upgraded tensor with the most parameters (ties: the
 * later in sensitivity order) is lowered one level, never below floor, and
 * (3) when none is left, the next routed tensor in rule 3's order (the gate
 * and up tensors of the layers in moeq_layer_order, then their down tensors;
 * ties by index) is lowered from Q_low to Q_low', raising B_total, until the
 * tensor fits at the lowest level rule 1 tried.  Rules 2 and 3 run only if
 * together they can make it fit; otherwise it stays at Q_low.  If Q_low alone
 * exceeds M_limit, rule 3 runs first.  All fit decisions are exact integer
 * comparisons in 1/64-bit units, so the plan is deterministic.
 *   p         HOST; the ladder and budget
 *   n         number of tensors, 1..2^20; sum of params <= 2^45
 *   params    HOST int64 [n], positive
 *   sens      HOST double [n], finite
 *   kind      HOST int32 [n], MOEQ_TENSOR_*
 *   layer     HOST int32 [n]: MoE layer position of routed tensors (ignored
 *             for others); NULL only if no tensor is routed
 *   level     HOST int32 [n] (written): each tensor's ladder level
 *   report    HOST (written) or NULL
 * Errors: INVALID_ARG (arguments, ladder, sizes).  An infeasible budget is
 * not an error: the plan is returned with report->feasible = 0. */
moeq_status moeq_plan_bits(const moeq_plan_params* p, int32_t n, const int64_t* params, const double* sens,
                           const int32_t* kind, const int32_t* layer, int32_t* level, moeq_plan_report* report);

/* Benchmark instrumentation: stage boundaries of moeq_forward.
 *   events  NULL (count 0) to stop, or MOEQ_STAGE_EVENTS hipEvent_t handles
 *           (as void*) owned by the caller.  Every following moeq_forward on
 *           this layer records, on its stream, events[0] before its first
 *           kernel, events[1] after routing and bucketing (and the gate,
 *           when the forward computes the logits), events[2] after the
 *           gate/up kernel, events[3] after the down kernel and events[4]
 *           after the combine, so hipEventElapsedTime between neighbours is
 *           the duration of one stage.
 * The handles are copied; the caller keeps them alive while they are set.
 * Errors: INVALID_ARG (count neither 0 nor MOEQ_STAGE_EVENTS, NULL handle). */
#define MOEQ_STAGE_EVENTS 5
moeq_status moeq_set_stage_events(moeq_layer* layer, void* const* events, int32_t count);

#ifdef __cplusplus
}
#endif

#endif /* MOEQ_H */
