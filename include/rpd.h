/*
 * rpd.h -- C ABI of the MI355X (gfx950) commit step of Reliable Parallel
 * Decoding (RPD).
 *
 * One call performs one decoding iteration's commit step (Sections 2.2, 3.1
 * and 3.2 of the paper; Appendix A.6 "Layerwise projection"): every masked
 * canvas position is projected through the unembedding at each of the final
 * K layers, each layer's full-vocabulary softmax is reduced to its argmax,
 * top probability and entropy (Eq. 1), layerwise stability is scored
 * (persistence Eq. 2, confidence drop Eq. 3, stability Eq. 4), candidates
 * are formed (Eq. 5), and the candidates whose cumulative upstream entropy
 * stays within the budget are committed, with the progress fallback
 * (Section 3.2).
 *
 * Conventions for every entry point:
 *  - Pointers marked "device" are HIP device (or managed) memory on the
 *    current device; "host" pointers are read during the call only.
 *  - The caller owns every buffer. The library allocates no device memory,
 *    keeps no pointer after it returns, and never writes its inputs.
 *  - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the
 *    default stream). Results are valid once the stream has completed.
 *  - Arrays are dense and row-major in the shapes given. The final layer of
 *    the window is layer K-1.
 *  - Errors: every argument is validated on the host before anything is
 *    enqueued, so a status other than RPD_OK and RPD_ERR_HIP means nothing
 *    was enqueued and the outputs are untouched. RPD_ERR_HIP reports a HIP
 *    runtime call or launch that failed part-way: the work enqueued before
 *    it stays enqueued and may have written the outputs and the workspace
 *    in part, so the outputs are then undefined (and the stream may be in
 *    an error state, as HIP reports it). rpd_last_error() describes the
 *    failure (thread-local). No C++ exception crosses this interface.
 *  - Calls on distinct streams with distinct workspaces may overlap.
 */
#ifndef RPD_H
#define RPD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RPD_ABI_VERSION 3

/* element type of `hidden` and `w_u` (both must have the same type) */
enum { RPD_DTYPE_BF16 = 0, RPD_DTYPE_F32 = 1 };

typedef enum rpd_status {
  RPD_OK = 0,
  RPD_ERR_NULL_POINTER = 1,        /* a required pointer is NULL */
  RPD_ERR_BAD_SHAPE = 2,           /* a dimension is out of range */
  RPD_ERR_BAD_PARAM = 3,           /* a hyperparameter is out of range or NaN */
  RPD_ERR_WORKSPACE_TOO_SMALL = 4, /* workspace_bytes < the required size */
  RPD_ERR_UNSUPPORTED = 5,         /* dtype / alignment / size not supported */
  RPD_ERR_HIP = 6                  /* a HIP runtime call or launch failed */
} rpd_status;

/* bits of rpd_params.flags */
#define RPD_PARAM_LAZY 1u     /* lazy layerwise projection (see rpd_params) */
#define RPD_PARAM_LAZY_ALL 2u /* with RPD_PARAM_LAZY: every masked position walks its layers */

/* per-position flag bits written to rpd_outputs.flags */
#define RPD_FLAG_CANDIDATE 1u  /* in the candidate set C_t (Eq. 5) */
#define RPD_FLAG_HIGH_CONF 2u  /* admitted because c_i >= theta_h */
#define RPD_FLAG_STABLE    4u  /* admitted through the stability test */
#define RPD_FLAG_COMMITTED 8u  /* in the commitment set A_t */
#define RPD_FLAG_FALLBACK  16u /* committed by the progress fallback */

/* bits of the optional device status word */
#define RPD_DEVICE_STATUS_MASKED_OVERFLOW 1 /* more masked positions than max_masked */

/*
 * The problem of one call (Section 3: the masked positions M_t of the canvas
 * and the hidden states of the final layers of one forward pass).
 *   K           number of final layers supplied, 1 <= K <= 64 (the paper
 *               projects layers l0..L, Appendix A.6; here the K supplied)
 *   B, L        sequences and canvas positions per sequence (B >= 1, L >= 1,
 *               B*L <= 2^24)
 *   d, V        hidden size and vocabulary size (1 <= d <= 2^20, 1 <= V < 2^31);
 *               bf16 requires d % 8 == 0
 *   dtype       RPD_DTYPE_BF16 or RPD_DTYPE_F32
 *   hidden      device [K][B][L][d]; hidden states already passed through the
 *               model's final normalisation; rows of unmasked positions are
 *               never read (they may hold anything, NaN included)
 *   w_u         device [V][d]; the unembedding (output head), d contiguous;
 *               16-byte aligned
 *   mask        device [B][L] uint8; nonzero = masked (in M_t)
 *   norm_weight optional device [d], same type as hidden: the gain g of the
 *               model's final normalization (RMS normalization). NULL: every
 *               supplied state is already normalized and is projected as is.
 *               Otherwise the states of layers 0 .. K-2 (and of layer K-1
 *               too if norm_final != 0) are first replaced by
 *               g * x / sqrt(mean(x^2) + norm_eps), evaluated in float64 and
 *               rounded (to nearest, ties to even) to the input type, as the
 *               model's normalization hands the output head (Appendix A.2
 *               "Intermediate-layer readout", A.6 "Layerwise projection":
 *               the final layer uses the native, already normalized state).
 *               16-byte aligned for bf16.
 *   norm_eps    >= 0, finite; the normalization's epsilon (unused without g)
 *   norm_final  0: layer K-1 is the model's native normalized state (the
 *               paper); 1: normalize it like the others
 *   max_masked  an upper bound on the number of masked positions summed over
 *               the batch, or -1. With -1 the call reads the exact count back
 *               from the device once (one stream synchronisation). If the
 *               bound is exceeded, only the first max_masked masked positions
 *               (batch-major, canvas order) are scored, the results for the
 *               rest are undefined, and RPD_DEVICE_STATUS_MASKED_OVERFLOW is
 *               raised in the optional status word.
 */
typedef struct rpd_problem {
  int32_t K, B, L, d, V;
  int32_t dtype;
  const void* hidden;
  const void* w_u;
  const uint8_t* mask;
  int32_t max_masked;
  const void* norm_weight;
  float norm_eps;
  int32_t norm_final;
} rpd_problem;

/*
 * Hyperparameters (Table 4, Appendix A.6; LLaDA: theta_s 3.5, w 15; Dream:
 * theta_s 2.5, w 20; both theta_h 0.9, theta_c 0.6, K_max 6, beta 4 nats,
 * W 32). Requirements: 0 <= theta_c <= theta_h, w >= 0, k_max >= 1,
 * beta >= 0 (may be +inf), window >= 1, flags only RPD_PARAM_LAZY and
 * RPD_PARAM_LAZY_ALL (the latter only with the former), block >= 0; no NaN.
 *
 * block selects the commitment rule. 0: full RPD (Section 3.2), the
 * cumulative-entropy budget beta over the whole canvas with the fallback
 * over the first `window` masked positions. > 0: RPD-block (Section 3.2
 * "Variants", Appendix A.6 "RPD-block"; the paper uses 32): the canvas of
 * each sequence is cut into runs of `block` positions starting at 0, the
 * active block is the first run holding a masked position, every candidate
 * (Eq. 5) inside it is committed with no budget (beta and window are then
 * unused), and without one its most confident masked position is. The
 * reported upstream entropy is then the entropy over earlier masked
 * positions outside the commitment set.
 *
 * RPD_PARAM_LAZY in flags: lazy layerwise projection (Appendix A.6
 * "Layerwise projection": a position's intermediate layers are projected
 * from the final one down, no further than its agreement suffix needs). The
 * final layer of every masked position is projected first; then the
 * positions that walk project layer K-2, K-3, ..., each stopping after its
 * first disagreeing layer. With RPD_PARAM_LAZY_ALL as well, every masked
 * position with a finite final confidence walks (the procedure as the paper
 * states it), and persistence, drop and stability equal the eager
 * projection's everywhere. Without it only the positions with
 * theta_c <= c < theta_h walk: the only ones whose candidacy the stability
 * test decides (Eq. 5), a further saving of this library beyond the
 * paper's procedure that leaves every decision unchanged; outside that band
 * persistence, drop and stability are then not evaluated (persistence -1,
 * drop and stability NaN). Either way tokens, candidacy and commitment are
 * those of the eager projection, and the per-layer outputs of layers never
 * projected hold -1 / NaN. One projection
 * pass per layer (each streams W_U again): it pays where the projection is
 * compute-bound (many masked positions), not where streaming W_U dominates.
 * While the bound on a pass's rows (max_masked, then the last count read
 * back) is at most 256, the pass reads its count on the device and is
 * launched once per size class the count may fall in (<= 64, <= 128, up to
 * the bound), all but one exiting at once; above, the previous pass's count
 * is read back (one stream synchronisation) and the pass planned for it. So
 * with max_masked <= 256 the call never synchronises.
 *
 * logit_scale multiplies every logit before the softmax statistics (an
 * inverse temperature). The paper reads probabilities before any
 * temperature (Appendix A.2), i.e. 1; 0 is read as 1; otherwise it must be
 * finite and > 0. rpd_gate_commit ignores it.
 */
typedef struct rpd_params {
  float theta_h;   /* high-confidence threshold (bypasses stability), Eq. 5 */
  float theta_c;   /* minimum confidence for stability admission, Eq. 5 */
  float theta_s;   /* stability threshold, Eq. 5 */
  float w;         /* weight of the confidence-drop penalty, Eq. 4 */
  int32_t k_max;   /* cap on persistence, Eq. 4 */
  float beta;      /* cumulative entropy budget in nats, Section 3.2 */
  int32_t window;  /* fallback window W, Section 3.2 */
  uint32_t flags;  /* RPD_PARAM_* bits */
  int32_t block;   /* 0: full RPD; > 0: RPD-block with blocks of this many positions */
  float logit_scale; /* inverse temperature of the scoring softmax; 0 or 1: none */
} rpd_params;

/*
 * Outputs, all device memory, shape [B][L] unless noted. Unmasked positions
 * receive: commit 0, token -1, persistence 0, flags 0 and 0.0f elsewhere.
 *   commit            1 if the position is in A_t (Section 3.2)
 *   token             y_i, the final-layer argmax, for every masked
 *                     position, committed or not. Ties go to the lowest
 *                     index: logits equal in exact arithmetic are found
 *                     exactly while |logit_scale| * sum_k |W_U[y,k] x_k|
 *                     <= 256 (|max logit| + 1) at d = 4096 (the bound
 *                     scales with 1/(d+1)); a positive gap below the fp32
 *                     accumulation error 4 (d+1) 2^-24 sum_k |W_U[y,k] x_k|
 *                     may go either way
 *   entropy           H(p_i^(K-1)) in nats (Eq. 1)
 *   confidence        c_i = p_i^(K-1)(y_i)
 *   persistence       K_i (Eq. 2), counted within the K supplied layers
 *   drop              r_i (Eq. 3)
 *   stability         S_i = min(K_i, k_max) - w r_i (Eq. 4)
 *   flags             RPD_FLAG_* bits
 *   upstream_entropy  E_i: entropy summed over earlier masked positions of
 *                     the sequence that are not in A_t (Section 3.2),
 *                     evaluated before the fallback
 *   n_commit          [B] number of committed positions per sequence
 * Optional (NULL to skip):
 *   layer_argmax, layer_conf, layer_entropy   [K][B][L] per-layer argmax,
 *                     top probability and entropy at masked positions
 *                     (unmasked entries are left untouched)
 *   status            one int32 of RPD_DEVICE_STATUS_* bits, overwritten
 */
typedef struct rpd_outputs {
  uint8_t* commit;
  int32_t* token;
  float* entropy;
  float* confidence;
  int32_t* persistence;
  float* drop;
  float* stability;
  uint8_t* flags;
  float* upstream_entropy;
  int32_t* n_commit;
  int32_t* layer_argmax;
  float* layer_conf;
  float* layer_entropy;
  int32_t* status;
} rpd_outputs;

/* Device workspace bytes that rpd_score_commit needs for problem `p`
 * (pointers in `p` are not read; norm_weight is only tested for NULL).
 * Returns 0 if the shape is invalid. */
size_t rpd_workspace_size(const rpd_problem* p);

/*
 * The whole commit step (Sections 2.2, 3.1, 3.2). `workspace` is device
 * memory of at least rpd_workspace_size(p) bytes, 256-byte aligned, used only
 * during the call's stream work; its prior contents do not matter.
 */
rpd_status rpd_score_commit(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                            void* workspace, size_t workspace_bytes, void* stream);

/*
 * rpd_score_commit, recording caller-created HIP events (hipEvent_t, cast to
 * void*) on `stream` at its stage boundaries, for callers that time the
 * stages: events[0] before the masked-position compaction, [1] before the
 * projection (logit lens + fused softmax statistics; with a norm_weight, the
 * final normalization of the rows comes first, after [1]), [2] after it, [3]
 * after the cross-tile reduction and stability scoring, [4] after the
 * commitment scan. Only the first n_events (0..5) are used;
 * NULL entries are skipped (with RPD_PARAM_LAZY, [1] precedes the first
 * pass and [2] follows the last). Everything else is exactly
 * rpd_score_commit.
 */
rpd_status rpd_score_commit_timed(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                                  void* workspace, size_t workspace_bytes, void* stream,
                                  void* const* events, int32_t n_events);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * rpd_score_commit without a workspace argument. The workspace is a
 * library-owned static device array of RPD_NOALLOC_SCRATCH_BYTES on each
 * GPU the library runs on, held until the process ends; the call allocates
 * nothing (no hipMalloc, no allocating library routine). Problems whose
 * rpd_workspace_size exceeds RPD_NOALLOC_SCRATCH_BYTES are rejected with
 * RPD_ERR_WORKSPACE_TOO_SMALL before anything is enqueued (at the LLaDA-8B
 * vocabulary, up to about 8,400 projected rows: K * max_masked). Every call
 * on one GPU shares that GPU's array: calls that overlap on one GPU (other
 * streams, other threads) race and must be serialised by the caller. The
 * array's prior contents never matter (every kernel writes what it reads).
 * The first call on a device, with that device current, looks the array's
 * address up (RPD_ERR_HIP if that fails). Otherwise exactly
 * rpd_score_commit, including its validation and error reporting.
 */
#define RPD_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
rpd_status rpd_score_commit_noalloc(const rpd_problem* p, const rpd_params* q, const rpd_outputs* o,
                                    void* stream);

/*
 * Scoring and commitment from per-layer statistics that the caller already
 * has (Eq. 2-5 and Section 3.2), for callers whose logits come from
 * elsewhere. layer_argmax / layer_conf / layer_entropy are device [K][B][L]
 * in the layout rpd_score_commit writes them (only masked positions are
 * read; only the final layer's entropy is used). Inside the agreement suffix
 * the probability of the final token equals that layer's top probability,
 * which is how Eq. 3 is evaluated. Writes the required outputs of `o`; the
 * optional per-layer pointers and status of `o` are ignored. Needs no
 * workspace.
 */
rpd_status rpd_gate_commit(int32_t K, int32_t B, int32_t L, const uint8_t* mask,
                           const int32_t* layer_argmax, const float* layer_conf,
                           const float* layer_entropy, const rpd_params* q,
                           const rpd_outputs* o, void* stream);

/* projection kernel variants (values of rpd_projection_variant) */
enum {
  RPD_PROJ_BF16_S32 = 0,  /* bf16, at most 32 projected rows: W_U streamed once from HBM */
  RPD_PROJ_BF16_S64 = 1,  /* bf16, 33..64 rows, same kernel family */
  /* 2: no longer planned (a 65..128-row streaming form, replaced by 7) */
  RPD_PROJ_F32 = 3,       /* fp32 inputs, any row count */
  RPD_PROJ_BF16_BIG = 4,  /* bf16, more than 128 rows: MFMA tiles of 256 x 256 */
  /* 5: no longer planned (a 129..192-row streaming form, replaced by 6) */
  RPD_PROJ_BF16_BIG192 = 6, /* bf16, more than 128 rows where 256 x 192 tiles pad the rows less (129..192 rows
                               always; above, whenever ceil(R/192)*192 < ceil(R/256)*256) */
  RPD_PROJ_BF16_BIG128 = 7  /* bf16, 65..128 rows: one MFMA tile of 256 x 128 per vocabulary tile */
};

/*
 * The projection kernel variant (RPD_PROJ_*) that rpd_score_commit launches
 * for problem `p` (pointers in `p` are not read), where the projected rows
 * are K * max_masked; with max_masked < 0 this assumes every position is
 * masked (the call itself plans for the count it reads back). Returns -1 if
 * the shape or dtype is invalid. For instrumentation and tests.
 */
int32_t rpd_projection_variant(const rpd_problem* p);

/*
 * The end of an iteration (Section 3.2: the positions of A_t are filled with
 * their predictions y_i; every other position keeps its mask): for every
 * masked position with commit != 0, canvas = token and mask = 0.
 *   mask     [B][L] uint8, updated in place
 *   canvas   [B][L] int32, written only at the positions committed here
 *   commit, token  [B][L] uint8 / int32 as rpd_score_commit writes them
 *   progress optional int32 [1 + progress_len], zeroed by the caller before
 *            the first call: progress[0] counts the calls made with it and
 *            progress[1 + t] receives the number of positions still masked
 *            after call t (for t < progress_len), so a loop of iterations
 *            learns when the canvas is full without a read-back per
 *            iteration. With it the update runs in one workgroup (meant for
 *            canvases of up to some tens of thousands of positions); without
 *            it, over the whole GPU.
 *   step     optional int32 [B][L] (needs progress): at each position
 *            committed here, the call index progress[0] had on entry.
 * All pointers are device memory owned by the caller. NULL mask, canvas,
 * commit or token, or step without progress, -> RPD_ERR_NULL_POINTER; B or L
 * < 1 or B*L > 2^24 -> RPD_ERR_BAD_SHAPE; progress_len < 0 ->
 * RPD_ERR_BAD_PARAM. Enqueued on `stream`; it allocates nothing and never
 * synchronises, so a loop body of rpd_score_commit (max_masked >= 0, and at
 * most 256 with lazy projection) followed by this call can be captured in a
 * HIP graph.
 */
rpd_status rpd_apply_commit(int32_t B, int32_t L, uint8_t* mask, int32_t* canvas, const uint8_t* commit,
                            const int32_t* token, int32_t* progress, int32_t progress_len, int32_t* step,
                            void* stream);

/* Static text for a status code. */
const char* rpd_status_string(rpd_status s);

/* Detail of the calling thread's most recent non-OK status ("" if none). */
const char* rpd_last_error(void);

/* RPD_ABI_VERSION of the library. */
int32_t rpd_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* RPD_H */
