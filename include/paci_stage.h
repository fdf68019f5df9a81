/*
 * paci_stage.h -- C ABI of one PACI pipeline stage on an MI355X (gfx950).
 *
 * PACI (arXiv 2606.07881) runs asynchronous 1F1B pipeline training in which a
 * stage accumulates the gradients of K local backwards before each optimizer
 * update. This bounds how many parameter versions a micro-batch's backward can
 * be behind its forward (Eq. 2: Delta <= ceil((N - i) / a)). This library is
 * the per-stage hot path. For each micro-batch it runs the forward and the
 * backward of a stack of pre-LN GPT blocks. It accumulates the local gradient
 * into an fp32 buffer G and applies AdamW with G every K backwards. A stage
 * at pipeline position p has delay = N - 1 - p micro-batches in flight
 * (the paper's N - i).
 *
 * Notation: the paper's accumulation factor a is K here, and its downstream
 * depth N - i (one-indexed stage i) is `delay`.
 *
 * Conventions for every call
 *   - Every call returns an int status: PACI_OK (0), PACI_STEP_DUE (1) or a
 *     negative PACI_E_* code. On a negative status the handle's counters and
 *     buffers are unchanged (checks run before any device work is enqueued),
 *     except for PACI_E_HIP, which leaves the handle unusable.
 *   - Device work is enqueued on the HIP stream given to paci_stage_init and
 *     is asynchronous to the host. Versions, counters and stamps are host
 *     integers, so they are final when the call returns; device buffers are
 *     final only after the stream is synchronized (paci_stage_sync).
 *   - A handle is single-threaded: calls on one handle must not overlap.
 *   - Pointers named `dev_*` or documented as device buffers are device
 *     memory on the stage's GPU; the caller owns them and keeps them alive
 *     until the stream has consumed them.
 *   - Activations use the stage dtype (fp32 or bf16), row-major [T, d_model]
 *     with T = micro_batch * seq tokens, token t = b * seq + s.
 */
#ifndef PACI_STAGE_H
#define PACI_STAGE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes -------------------------------------------------------- */
#define PACI_OK 0
#define PACI_STEP_DUE 1          /* backward completed the K-th micro-batch of a window */
#define PACI_E_INVAL (-1)        /* bad argument (null pointer, size, shape relation) */
#define PACI_E_UNSUPPORTED (-2)  /* valid but not implemented (head_dim, dtype) */
#define PACI_E_NOMEM (-3)        /* arena smaller than paci_stage_arena_bytes */
#define PACI_E_ORDER (-4)        /* micro-batch out of FIFO order */
#define PACI_E_BACKPRESSURE (-5) /* forward refused: q > delay (admission rule) */
#define PACI_E_STEP_PENDING (-6) /* forward/backward while an update is due */
#define PACI_E_NOT_DUE (-7)      /* step before K backwards of the window */
#define PACI_E_HIP (-8)          /* a HIP runtime call failed; see paci_last_hip_error */
#define PACI_E_SCRATCH (-9)      /* the call needs more than the library's static scratch buffer */

/* ---- stage description ---------------------------------------------------- */
enum paci_kind { PACI_MIDDLE = 0, PACI_FIRST = 1, PACI_LAST = 2 };
enum paci_dtype { PACI_FP32 = 0, PACI_BF16 = 1 };

typedef struct paci_shapes {
  int32_t n_layers;     /* pre-LN decoder blocks in this stage (>= 1) */
  int32_t d_model;      /* d = n_heads * head_dim */
  int32_t n_heads;
  int32_t head_dim;     /* 32, 64 or 128 */
  int32_t d_ff;         /* FFN width f, multiple of 32 */
  int32_t seq;          /* S, tokens per sequence, <= max_pos for PACI_FIRST */
  int32_t micro_batch;  /* mu, sequences per micro-batch */
  int32_t vocab;        /* V (PACI_FIRST / PACI_LAST only) */
  int32_t max_pos;      /* rows of the position table (PACI_FIRST only) */
  int32_t kind;         /* enum paci_kind */
  int32_t dtype;        /* enum paci_dtype: arithmetic type of the activations */
  float lr, beta1, beta2, eps, weight_decay; /* AdamW hyper-parameters */
  float ln_eps;         /* LayerNorm epsilon */
  int32_t recompute;    /* 1: activation-checkpointed stage (appendix "Activation checkpointing"):
                           a forward keeps only the stage input, the backward recomputes the
                           activations under the current parameters first; 0: stored activations */
  int32_t lr_warmup;    /* learning-rate schedule (appendix "Detailed experimental setup"): update t
                           (1-based) uses lr * t / lr_warmup while t <= lr_warmup, then a cosine
                           from lr down to lr * lr_min_ratio at update lr_total, flat after it */
  int32_t lr_total;     /* 0: no schedule, every update uses lr */
  float lr_min_ratio;
  int32_t fused_head;   /* PACI_LAST, bf16, d % 8 == 0, delay 0 only. 1: no [T, V] logits are stored;
                           the LM-head forward product reduces each row to its log-sum-exp and target
                           logit as it goes, and the backward recomputes the product (same parameters,
                           since a delay-0 stage's backward follows its forward before any update) and
                           turns it into dL/dz inside the same kernel. 0: fp32 logits per slot */
  float dropout;        /* rate p in [0, 1) of inverted dropout at GPT-2's four places (appendix
                           "Detailed experimental setup": 0.1): the embedding sum (first stage), the
                           attention probabilities, and the attention-projection and FFN outputs
                           before their residual adds; kept values are scaled by 1 / (1 - p). 0: off */
  uint32_t dropout_seed; /* masks are a pure function of (dropout_seed, micro-batch index, block,
                           site, element) through Philox4x32-10, so a backward (and a recomputed
                           forward) uses its forward's masks; the element -> bits map is given with
                           paci_stage_forward */
  int32_t window;       /* 0 (default): Alg. 1's accumulate step as written, every backward adds its
                           block weight gradients to G, and the store holds delay + 1 micro-batch
                           slots (the in-flight count of the appendix "Memory and synchronization
                           properties"). 1: windowed block weight gradients (bf16, micro_batch * seq
                           a multiple of 64, d and d_ff multiples of 8, recompute 0; else
                           E_UNSUPPORTED): each backward keeps its blocks' output gradients, and
                           one contraction per weight over the K micro-batches of a window adds
                           them to G before the update or an earlier read of G. Same sum up to fp32
                           rounding order; costs K - 1 more activation slots plus the window's
                           output gradients */
} paci_shapes;

typedef struct paci_counters {
  int32_t version;      /* t: local optimizer updates applied so far */
  int32_t c;            /* backwards in the current accumulation window */
  int32_t q;            /* forwards whose backward has not yet run */
  int32_t next_f;       /* micro-batch index the next forward must carry */
  int32_t next_b;       /* micro-batch index the next backward must carry */
  int32_t K, delay;
} paci_counters;

/* Description of one parameter tensor in the canonical order. */
typedef struct paci_param_info {
  char name[32];        /* e.g. "h3.w_qkv", "wte", "lnf_g" */
  int32_t rows, cols;   /* matrices: [rows, cols] = [out, in]; vectors: [rows, 1] */
  int64_t offset;       /* element offset in the flat canonical vector */
  int64_t numel;
  int32_t decay;        /* 1 if AdamW weight decay applies */
} paci_param_info;

typedef struct paci_stage paci_stage; /* opaque handle */
typedef struct paci_fsm paci_fsm;     /* opaque host-only protocol object */

/* ---- host-only protocol (Alg. 1 counters) --------------------------------
 * The event rule of one stage (Alg. 1, appendix "Stage-level execution rule"),
 * with no device work. A forward of micro-batch mb is admitted only if
 * mb == next_f, no update is due and q <= delay (Sec. 3.2, admission rule
 * q_i < N + 1 - i); it returns the version t it ran at (t^F) and increments q.
 * A backward must carry mb == next_b < next_f (FIFO, 1F1B); it returns t^B,
 * increments c, decrements q and returns PACI_STEP_DUE when c == K. A step is
 * legal only when c == K; it resets c and increments t. paci_stage_* use this
 * same object, so the stage and its protocol cannot disagree. */
int paci_fsm_create(int K, int delay, paci_fsm** out);      /* E_INVAL: K < 1, delay < 0 */
int paci_fsm_forward(paci_fsm* f, int mb, int* version);   /* E_ORDER, E_BACKPRESSURE, E_STEP_PENDING */
int paci_fsm_backward(paci_fsm* f, int mb, int* version);  /* E_ORDER, E_STEP_PENDING; may return STEP_DUE */
int paci_fsm_step(paci_fsm* f, int* new_version);          /* E_NOT_DUE */
int paci_fsm_counters(const paci_fsm* f, paci_counters* out);
int paci_fsm_destroy(paci_fsm* f);

/* Canonical asynchronous 1F1B order of one stage (Alg. 1 with every forward
 * issued as soon as it is admitted and every update right after the backward
 * that completes its window): F_0 .. F_min(delay, M-1); then for j = 0..M-1:
 * B_j, S if (j+1) % K == 0, F_{j+delay+1} if j+delay+1 < M.
 * kinds[e] is 0 (forward), 1 (backward) or 2 (step); idx[e] is the micro-batch
 * (-1 for a step). Host arrays of capacity `cap`; *n receives the event count
 * (2M + floor(M/K)). E_INVAL if M < 0, K < 1, delay < 0 or cap is too small
 * (then *n still receives the required count). */
int paci_schedule(int M, int K, int delay, int32_t* kinds, int32_t* idx, int cap, int* n);

/* Synchronous 1F1B with a flush, the comparison schedule of Sec. 2 and Eq. (3),
 * at one stage: window by window (micro-batches wK .. wK+K-1), the forwards
 * F_wK .. F_wK+min(delay, K-1), then B_j followed by F_j+delay+1 while it lies
 * in the window, and the update after the window's last backward. No forward of
 * a window runs before the previous window's update, so every stamp has
 * Delta = 0. Same arrays, count and errors as paci_schedule; a trailing partial
 * window (M % K != 0) has no update. */
int paci_schedule_flush(int M, int K, int delay, int32_t* kinds, int32_t* idx, int cap, int* n);

/* ---- parameter layout (host only) ------------------------------------------
 * The canonical order: first stage prefix wte [V, d], wpe [max_pos, d]; per
 * block l: h{l}.ln1_g, ln1_b, w_qkv [3d, d], b_qkv, w_o [d, d], b_o, ln2_g,
 * ln2_b, w_1 [f, d], b_1, w_2 [d, f], b_2; last stage suffix lnf_g, lnf_b,
 * w_lm [V, d]. The flat canonical vector is the concatenation in this order
 * with no padding. Weight decay applies to the w_* matrices only (appendix
 * "Detailed experimental setup": no decay on biases, LayerNorm parameters or
 * embeddings). */
int paci_param_count(const paci_shapes* s, int* n_tensors, int64_t* n_elements);
int paci_param_info_at(const paci_shapes* s, int index, paci_param_info* out); /* E_INVAL: bad index */

/* ---- stage lifetime --------------------------------------------------------- */
/* Bytes of device memory the stage needs: fp32 parameters, G, AdamW moments,
 * the bf16 working copy (bf16 stages), the activation store and the backward
 * workspace. The sizes follow the stage's memory model (appendix "Memory and
 * synchronization properties": one parameter copy, no weight stash, the
 * activations of the micro-batches in flight). The store has delay + 1
 * micro-batch slots (a stage admits at most delay + 1 forwards whose backward
 * has not run, Sec. 3.2), or K + delay with windowed weight gradients
 * (paci_shapes.window = 1): such a stage also keeps every block's output
 * gradients of the K micro-batches of a window. A checkpointed stage
 * (recompute = 1) has delay + 1 slots holding only the stage input (ids,
 * targets) plus one work slot for the activations. Pure host computation;
 * E_INVAL / E_UNSUPPORTED as for paci_stage_init. */
int paci_stage_arena_bytes(const paci_shapes* s, int K, int delay, size_t* bytes);

/* stage_init(shapes, K, delay): one pipeline stage of Alg. 1 (appendix
 * "Stage-level execution rule") with a single parameter copy theta, the
 * accumulator G and the AdamW moments (appendix "Memory and synchronization
 * properties"), counters t = c = q = 0 (appendix "Pipeline setup and notation":
 * versions count local updates from 0). `dev_arena` is caller-owned device memory of
 * at least paci_stage_arena_bytes bytes, 256-byte aligned, that must outlive
 * the handle; `hip_stream` is the hipStream_t all work is enqueued on (NULL =
 * the null stream). Parameters start at zero and G, m, v are cleared; load the
 * initial parameters with paci_stage_load. Counters start at t = c = q = 0.
 * Errors: E_INVAL (null pointer, d != n_heads * head_dim, K < 1, delay < 0,
 * seq > max_pos on a first stage, non-positive size), E_UNSUPPORTED (head_dim
 * not 32/64/128, d_ff or d not multiples of 32, unknown kind or dtype),
 * E_NOMEM (arena too small), E_HIP. */
int paci_stage_init(const paci_shapes* s, int K, int delay, void* dev_arena, size_t arena_bytes,
                    void* hip_stream, paci_stage** out);
int paci_stage_destroy(paci_stage* h); /* frees host state only; the arena stays the caller's */

/* ---- state transfer --------------------------------------------------------- */
enum paci_what { PACI_PARAMS = 0, PACI_GRADS = 1, PACI_EXP_AVG = 2, PACI_EXP_AVG_SQ = 3 };
/* State transfer of the stage's single parameter copy, its accumulator G
 * (Alg. 1's local gradient sum) and the AdamW moments (appendix "Detailed
 * experimental setup": AdamW). Copy n fp32 values in the canonical order into / out of the stage. n must
 * equal the stage's element count (paci_param_count). `src`/`dst` are device
 * pointers if `on_device` is non-zero, else host pointers (the call then
 * synchronizes the stream). Loading PARAMS also rewrites the bf16 working copy.
 * Reading or loading GRADS first adds any windowed weight gradients still
 * pending, so G always holds every backward so far. E_INVAL on a wrong count
 * or null pointer. */
int paci_stage_load(paci_stage* h, int what, const float* src, int64_t n, int on_device);
int paci_stage_read(paci_stage* h, int what, float* dst, int64_t n, int on_device);

/* ---- the three events of Alg. 1 ----------------------------------------------- */
/* stage_forward(mb, &version): F_i of micro-batch mb at the current parameters
 * (Alg. 1's forward event, admitted only while q <= delay, Sec. 3.2; the
 * version it returns is t^F of the appendix "Pipeline setup and notation").
 * Middle/last stage: `dev_in` is the stage input [T, d] (stage dtype). First
 * stage: `dev_in` is int32 token ids [micro_batch, seq] in [0, vocab).
 * Middle/first stage: `dev_out` receives [T, d] (stage dtype). Last stage:
 * `dev_targets` are int32 [micro_batch, seq] in [0, vocab) and `dev_out`
 * receives one fp32, the mean cross-entropy over the T tokens.
 * The input is copied into the activation store (slot mb modulo the slot
 * count), so the caller may reuse `dev_in` once the stream has passed this call. *version
 * receives t^F; q is incremented.
 * Errors (state unchanged): E_ORDER (mb != next_f), E_BACKPRESSURE (q > delay),
 * E_STEP_PENDING (an update is due), E_INVAL (null pointer). */
int paci_stage_forward(paci_stage* h, int mb, const void* dev_in, const int32_t* dev_targets,
                       void* dev_out, int* version);

/* stage_backward(mb, grad_out): B_i of micro-batch mb. It differentiates the
 * activations stored by F_mb at the parameters current now (Eq. 1: a stale
 * backward reads the newest version, with no weight stash), adds the local
 * gradient to the fp32 accumulator G, and writes the input gradient. On a
 * windowed stage the block weight gradients are added later, all K of the
 * window in one contraction per weight, before the update (or an earlier
 * read of G): the same sum up to fp32 rounding order. On a checkpointed stage
 * (recompute = 1) the backward first recomputes the stage forward from the
 * stored input under the current parameters and differentiates those
 * activations (appendix "Activation checkpointing").
 * Middle/first stage: `dev_grad_out` is dL/d(out) [T, d] (stage dtype). Last
 * stage: `dev_grad_out` must be NULL; the backward is seeded with
 * (softmax(z) - onehot(target)) / (T * K). `dev_grad_in` receives dL/d(in)
 * [T, d] (NULL to discard; always NULL for a first stage).
 * *version receives t^B; c is incremented, q decremented. Returns PACI_STEP_DUE
 * when this backward completes the window (c == K): paci_stage_step must run
 * before the next forward or backward.
 * Errors (state unchanged): E_ORDER (mb != next_b or no forward pending),
 * E_STEP_PENDING, E_INVAL. */
int paci_stage_backward(paci_stage* h, int mb, const void* dev_grad_out, void* dev_grad_in,
                        int* version);

/* For callers that cannot allocate device memory or rely on a caller-sized
 * workspace at call time (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): paci_stage_backward with the same
 * arguments, results and errors, except that the attention backward's
 * per-query scratch, the (lse2, D) pairs of micro_batch * n_heads *
 * roundup(seq, 64) queries (8 bytes each in bf16, micro_batch * n_heads * seq
 * * 4 bytes in fp32), comes from one static device buffer of 8 MiB that the
 * library holds per GPU until the process ends, not from the stage's arena.
 * It calls no allocating routine (no device allocation, no timing events: while
 * timing is on, this call's launches are not timed). Every call rewrites all of
 * the pairs it reads, so the buffer needs no clearing; it is shared by every
 * stage on the GPU, so calls that overlap on one GPU (stages on different
 * streams) race. Error: PACI_E_SCRATCH (state unchanged) if the pairs exceed
 * 8 MiB. */
int paci_stage_backward_static(paci_stage* h, int mb, const void* dev_grad_out, void* dev_grad_in,
                               int* version);

/* stage_step(): one AdamW update with G (the plain sum of the window's K local
 * gradients, Alg. 1), decoupled weight decay on the w_* matrices; then G <- 0,
 * c <- 0, t <- t + 1 and the bf16 working copy is rewritten. *new_version
 * receives t. E_NOT_DUE if c != K.
 * Non-finite guard (the paper has none; its limitations section leaves invalid
 * gradients unhandled): if any element of G is NaN or infinite, parameters and
 * moments are left unchanged, G is still cleared and t still advances, so the
 * version stamps stay a function of the event order alone. The decision is
 * taken on the device (no host synchronization). AdamW's bias correction and
 * the learning-rate schedule use a = (updates applied so far) + 1, which equals
 * t + 1 while no update was skipped. */
int paci_stage_step(paci_stage* h, int* new_version);

/* ---- schedule driver --------------------------------------------------------- */
/* The schedule driver: the event order of Alg. 1 at one stage, each forward
 * issued as soon as admission allows and each update right after the backward
 * that completes its window (Sec. 3.2; the order whose worst case Eq. (2)
 * bounds). Replays paci_schedule(M, K, delay) on the handle by calling forward,
 * backward and step. Micro-batch i reads dev_in_all + i * (input bytes) (ids
 * for a first stage), dev_targets_all + i * T (last stage), dev_grad_out_all
 * + i * (T * d elements) (middle/first), and writes dev_out_all + i * (output
 * bytes) and dev_grad_in_all + i * (T * d elements); either output may be NULL
 * to discard. host_stamps (host int32 [M][3], may be NULL) receives
 * (t^F, t^B, Delta) per micro-batch. The handle must be fresh for the replay
 * (next_f == next_b == 0, c == 0); the first error is returned. */
int paci_stage_run(paci_stage* h, int M, const void* dev_in_all, const int32_t* dev_targets_all,
                   const void* dev_grad_out_all, void* dev_out_all, void* dev_grad_in_all,
                   int32_t* host_stamps);

/* Replays the event list (kinds[e], idx[e]) for e < n, in the encoding of
 * paci_schedule (e.g. paci_schedule_flush's order), with the buffers and
 * stamps of paci_stage_run (host_stamps needs 3 entries per micro-batch index
 * used). Host arrays. The list is checked first (kinds in {0, 1, 2}, idx >= 0
 * for forwards and backwards: else E_INVAL and nothing runs); each event then
 * goes through the protocol, and the first error is returned with the events
 * before it done. Micro-batch indices are absolute: the handle may be in any
 * state the list continues (e.g. after paci_stage_resume), and the buffers are
 * indexed by them. host_stamps[3 i + 2] (Delta) is valid for micro-batches whose
 * forward ran in the same call. */
int paci_stage_run_events(paci_stage* h, int n, const int32_t* kinds, const int32_t* idx,
                          const void* dev_in_all, const int32_t* dev_targets_all,
                          const void* dev_grad_out_all, void* dev_out_all, void* dev_grad_in_all,
                          int32_t* host_stamps);

/* Rewinds the counters to t = c = q = 0, next_f = next_b = 0 and the applied /
 * skipped update counts to 0, keeping parameters, moments and G (pending
 * windowed weight gradients are added to G first); used to replay again from
 * the current state. */
int paci_stage_reset_counters(paci_stage* h);

/* Checkpoint / resume. A checkpoint of a drained stage (q = 0, c = 0) is
 * PARAMS, EXP_AVG and EXP_AVG_SQ (paci_stage_read), its counters and its
 * update counts (paci_stage_updates). To resume, load the three arrays into a
 * stage of the same shapes, K and delay, then call paci_stage_resume: it sets
 * the version t, the index of the next micro-batch (next_f = next_b; dropout
 * masks are keyed by it) and the applied / skipped update counts (AdamW's bias
 * correction and the rate schedule continue from applied + 1). Synchronizes
 * the stream. Errors: E_INVAL (a negative value), E_ORDER (micro-batches in
 * flight or a window partly accumulated; nothing changes), E_HIP. */
int paci_stage_resume(paci_stage* h, int32_t version, int32_t next_mb, int32_t applied, int32_t skipped);

/* Number of updates paci_stage_step applied and skipped (non-finite G) since
 * creation or the last paci_stage_reset_counters, which clears both.
 * Synchronizes the stream. Errors: E_INVAL (null pointer), E_HIP. */
int paci_stage_updates(paci_stage* h, int32_t* applied, int32_t* skipped);

/* ---- introspection ------------------------------------------------------------- */
int paci_stage_counters(const paci_stage* h, paci_counters* out);
int paci_stage_sync(paci_stage* h);              /* hipStreamSynchronize; E_HIP on failure */
int paci_last_hip_error(const paci_stage* h);    /* the hipError_t behind the last E_HIP (NULL: of paci_stage_init) */
const char* paci_strerror(int status);

/* Kernel timing: while enabled, each kernel launch of the stage is bracketed by
 * HIP events on the stage stream. paci_stage_kernel_times (after a sync) reports,
 * per kernel family, the number of launches, the summed device time in
 * milliseconds and the summed algorithmic work (FLOP for matrix kernels, bytes
 * for streaming kernels) since timing was enabled. Families are numbered
 * 0 .. paci_kernel_family_count() - 1 and named by paci_kernel_family_name. */
int paci_kernel_family_count(void);
const char* paci_kernel_family_name(int family);
int paci_stage_set_timing(paci_stage* h, int enable);
int paci_stage_kernel_times(paci_stage* h, int family, int64_t* launches, double* ms, double* work);

/* ---- stage planning (host only) --------------------------------------------------
 * Memory-constrained partition of a sequential stack of L layers over N
 * pipeline stages (appendix "Memory-constrained pipeline partitioning").
 * Layer l (0-based) has forward time t[l], static bytes s[l] (parameters,
 * gradients, optimizer state) and activation bytes a[l] per micro-batch. The
 * stages hold contiguous, non-empty layer ranges; stage j (1-based) keeps
 * w_j = N - j + 1 micro-batches in flight, so its memory is
 * sum s + w_j * sum a over its layers. The result minimises the largest stage
 * time subject to every stage's memory <= budget. If no partition fits, it
 * minimises the largest overshoot max(0, memory - budget) first and the
 * largest stage time second.
 * cuts (host int32 [N + 1]) receives 0 = c_0 < c_1 < ... < c_N = L (stage j
 * holds layers c_{j-1} .. c_j - 1); *max_time and *max_overshoot (nullable)
 * the optimum, with *max_overshoot == 0 exactly when a partition fits. Among
 * equal optima any one may be returned. Sums run left to right over each
 * stage's layers, so integer-valued inputs give exact results. O(L^2 N) time.
 * Errors: E_INVAL (N < 1, L < N, a null array, a negative or non-finite
 * t/s/a, or a budget that is negative or NaN; it may be +infinity). */
int paci_partition(int L, int N, const double* t, const double* s, const double* a, double budget,
                   int32_t* cuts, double* max_time, double* max_overshoot);

/* Bubble efficiency of synchronous 1F1B with a flush, m / (m + N - 1) (Eq. 3),
 * and of interleaved 1F1B with V model chunks per device, mV / (mV + N - 1)
 * (Eq. 4), for m micro-batches (real m > 0 allowed, as in the paper's worked
 * values) on N stages; NaN if m <= 0, N < 1 or V < 1. */
double paci_eta_flush(double m, int N);
double paci_eta_interleaved(double m, int N, int V);
/* Projected bubble-free throughput from a measured 1F1B-flush throughput,
 * t_flush / eta_flush(m, N) (Eq. 5). */
double paci_throughput_proxy(double t_flush, double m, int N);

#ifdef __cplusplus
}
#endif
#endif /* PACI_STAGE_H */
