/*
 * iefwd.h -- C ABI of libiefwd: the batched transformer forward pass of
 * co-located serverless DL instances on one MI355X (gfx950), each with a
 * compute quota expressed as a number of compute units (CUs).
 *
 * Problem statement this interface follows (Dilu, ASPLOS '25):
 *  - every serverless DL instance holds its own model and serves requests in
 *    batches of at most its inference batch size (Sec. 3.2, "Multi-Factor
 *    Profiling");
 *  - each instance has a compute quota that is not an integer number of GPUs
 *    but a continuous share, scaled up and down at run time (Sec. 3.4,
 *    "Adaptive 2D Co-Scaling"; Table 1, <request, limit> quotas);
 *  - a quota change acts between iterations (one batch execution is one
 *    iteration of an inference instance, Sec. 3.4.1 and Alg. 2);
 *  - co-located instances are isolated from each other (Sec. 3.4.1, Discussion).
 * Here the quota is a set of CUs: each instance launches on a HIP stream whose
 * hardware queue carries a CU mask, and a new mask takes effect at the next
 * batch boundary.
 *
 * Conventions
 *  - Every function returns an int status (IEFWD_OK = 0, negative = error)
 *    unless stated otherwise.  No C++ exception crosses the ABI; nothing aborts.
 *  - On error, iefwd_last_error() returns a message for the calling thread.
 *  - The caller owns every input/output buffer; an instance owns its weights,
 *    workspace and streams.  Calls on one instance must be serialised by the
 *    caller; distinct instances are independent and may be driven from
 *    different threads.
 *  - Results are a function of (config, seed, input) only: bit-identical
 *    across CU quotas, co-location, repeats and batch composition.  One
 *    exception: a decode step (iefwd_decode) sums its products in an order
 *    chosen by the batch-size class (1-4, 5-8 or 9-16 sequences), so its bits
 *    may differ between classes (never across quotas or co-location); prefill
 *    and decode agree within rounding, not bit for bit.
 *  - Device pointers are HIP device addresses on the instance's device.
 *  - After a HIP runtime error an instance is poisoned: every later call on it
 *    returns IEFWD_EHIP; destroy and re-create it (weights are a pure function
 *    of the config, so re-creation restores the same model).
 */
#ifndef IEFWD_H
#define IEFWD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define IEFWD_ABI_VERSION 1u

/* ---- status codes --------------------------------------------------------- */
#define IEFWD_OK        0
#define IEFWD_EINVAL   (-1)  /* bad argument: NULL, size out of range, bad shape */
#define IEFWD_ENODEV   (-2)  /* no usable gfx950 device with that index */
#define IEFWD_ENOMEM   (-3)  /* device or host allocation failed, or would exceed limits */
#define IEFWD_EHIP     (-4)  /* HIP runtime error; the instance is poisoned */
#define IEFWD_ESTATE   (-5)  /* call not valid in the instance's current state */
#define IEFWD_EVERSION (-6)  /* config.abi_version != IEFWD_ABI_VERSION */

typedef struct iefwd_instance iefwd_instance;   /* opaque, library-owned */

/* ---- model configuration ----------------------------------------------------
 * One transformer stack.  post-LN (pre_ln = 0): X1 = LN1(X + Attn(X)),
 * X' = LN2(X1 + FFN(X1)).  pre-LN (pre_ln = 1): X1 = X + Attn(LN1(X)),
 * X' = X1 + FFN(LN2(X1)), plus a final LN after the last layer.
 * FFN(Y) = GELU(Y W1 + b1) W2 + b2 with the exact erf GELU.  Attention scores
 * are Q K^T / sqrt(d_model / n_heads); causal = 1 keeps keys j <= i.
 * Output: n_out > 0 -> per-token logits X_L Wh + bh, fp32 [batch, seq, n_out];
 *         n_out = 0 -> final hidden states, fp32 [batch, seq, d_model].
 * Limits: d_model % 128 == 0, d_model <= 4096, d_model / n_heads in {64, 128},
 *         d_ff % 64 == 0, n_out <= 16, n_layers >= 1.
 * Weights are drawn on the host from the seeded init spec: element e of the
 * tensor with uid 32*layer + slot is sigma * N(0,1) from SplitMix64 +
 * Box-Muller, rounded fp64 -> fp32 -> bf16 (see iefwd_export_tensor for slots).
 */
typedef struct iefwd_config {
    uint32_t abi_version;   /* must be IEFWD_ABI_VERSION */
    uint32_t n_layers;
    uint32_t d_model;
    uint32_t n_heads;
    uint32_t d_ff;
    uint32_t max_batch;     /* workspace is sized for max_batch * max_seq tokens */
    uint32_t max_seq;
    uint32_t n_out;         /* head width; 0 = return hidden states */
    uint32_t pre_ln;        /* 0 = post-LN (BERT-style), 1 = pre-LN + final LN */
    uint32_t causal;        /* 0 = bidirectional, 1 = causal mask */
    uint32_t kv_cache;      /* 1 = keep every layer's K and V for iefwd_decode (needs pre_ln = causal
                               = 1 and max_seq <= 8192), and a packed copy of the four weight
                               matrices per layer for the decode step (the weights' device memory
                               roughly doubles); 0 = prefill only (default) */
    float    ln_eps;        /* LayerNorm epsilon (default 1e-5) */
    float    w_std;         /* std of weight matrices (default 0.02) */
    float    b_std;         /* std of biases (default 0: biases are zero) */
    float    ln_std;        /* gamma = 1 + ln_std*n, beta = ln_std*n (default 0) */
    float    qk_std;        /* std of the Q and K column blocks of Wqkv; 0 = w_std */
    uint64_t seed;          /* weight seed */
} iefwd_config;

/* Fills *cfg with the defaults above (abi_version set, all sizes 0). No status. */
void iefwd_config_init(iefwd_config *cfg);

/* ---- device ------------------------------------------------------------------ */

/* Number of CUs and XCDs of HIP device `device`.  ENODEV if there is no such
 * device or it is not gfx950. */
int iefwd_device_info(int device, uint32_t *n_cu, uint32_t *n_xcd);

/* Pure host function: the CU mask the library uses for a quota of `quota` CUs
 * starting at mask bit `first` on a device with n_cu CUs in n_xcd equal XCDs:
 * bits first, first + 1, ..., first + quota - 1 (mod n_cu).  Bit i of word
 * i/32 enables mask bit i (the bit order of hipExtStreamCreateWithCUMask),
 * which drives CU i / n_xcd of XCD i % n_xcd; a run of consecutive bits is
 * therefore spread evenly over the XCDs (each gets quota/n_xcd CUs or one
 * more; with first = 0 the first quota % n_xcd XCDs get the extra CU), so
 * every XCD's L2 serves an equal share.  Co-located instances placed at
 * first = 0, q0, q0 + q1, ... get disjoint CUs while their quotas sum to at
 * most n_cu, and overlap cyclically beyond that.
 * n_words must be >= ceil(n_cu / 32); extra words are zeroed.
 * EINVAL if quota is 0 or > n_cu, first >= n_cu, n_xcd is 0 or does not
 * divide n_cu. */
int iefwd_build_cu_mask(uint32_t n_cu, uint32_t n_xcd, uint32_t quota, uint32_t first,
                        uint32_t *mask, uint32_t n_words);

/* ---- instance lifecycle -------------------------------------------------------- */

/* Creates an instance on `device`: validates cfg, generates the weights on the
 * host (multi-threaded), uploads them, allocates the workspace and a stream
 * masked to all CUs.  On error *out is set to NULL. */
int iefwd_create(const iefwd_config *cfg, int device, iefwd_instance **out);

/* Waits for in-flight work and frees everything.  NULL is accepted (no-op). */
int iefwd_destroy(iefwd_instance *inst);

/* ---- quota (compute share) ------------------------------------------------------ */

/* Requests a quota of n_cu CUs (1 .. device CUs) starting at mask bit `first`
 * (0 .. device CUs - 1), spread evenly over the XCDs as by iefwd_build_cu_mask.
 * Takes effect at the next iefwd_submit; a batch already in flight keeps its
 * CUs.  EINVAL if n_cu or first is out of range.  Measured on MI355X: give
 * quotas in multiples of 32 CUs.  Each XCD's CUs sit in 4 shader engines and
 * workgroups are dealt to the engines in equal numbers, so a quota of 5-7 CUs
 * per XCD runs at about the speed of 4 (the BERT-base batch-32 forward: 6.99 ms
 * at 32 CUs, 6.42-6.50 ms at 40-56, 3.76 ms at 64). */
int iefwd_set_quota_at(iefwd_instance *inst, uint32_t n_cu, uint32_t first);

/* iefwd_set_quota_at(inst, n_cu, 0). */
int iefwd_set_quota(iefwd_instance *inst, uint32_t n_cu);

/* Creates the CU-masked stream for this quota and placement ahead of time, so
 * that a later iefwd_set_quota_at with the same arguments switches without
 * creating a hardware queue at the next submit (creation takes about 5 ms).
 * Unlike the other calls on an instance, this one may run on another thread
 * concurrently with them (a controller thread preparing the next quotas while
 * the serving thread submits).  The instance caches 2 masked streams (the one
 * in use, never evicted, and one more), since every live masked stream is a
 * hardware queue.  EINVAL as iefwd_set_quota_at. */
int iefwd_prepare_quota_at(iefwd_instance *inst, uint32_t n_cu, uint32_t first);

/* Sets how many masked streams (hardware queues) the instance keeps cached:
 * 1 .. 16, default 2 (the one in use and one more).  Lowering it destroys the
 * least recently used streams beyond the new size (never the one in use).
 * Measured on MI355X, and the reason the cache is small: creating or
 * destroying a masked queue stalls every other queue of the process for
 * about 3 ms, and with more than about 20-24 live queues in a process the
 * hardware scheduler time-slices them (12-33 ms stalls).  A serving loop that
 * moves quotas every control period should therefore prepare a fixed set of
 * placements once (iefwd_prepare_quota_at), size the cache to hold them, and
 * keep the whole process within that queue budget.  Also measured: the order
 * the queues are created in matters.  Created in rounds (one per instance per
 * round, the instances always in the same order), co-located instances keep
 * their batch times; created instance by instance, a latency-sensitive
 * instance's batches ran 5-8 times slower whenever another instance's long
 * GEMM launches ran, on whatever CUs.  The queues appear to be dealt to the
 * device's dispatch pipes in creation order.  A placement still cached is not
 * created again, which shifts every later queue of a round order: shrink the
 * caches to 1 (the stream in use) before creating a set of placements in
 * rounds.  EINVAL outside 1 .. 16. */
int iefwd_set_stream_cache(iefwd_instance *inst, uint32_t capacity);

/* Requests an explicit CU mask (n_words 32-bit words, bit order as above);
 * same timing as iefwd_set_quota.  EINVAL if the mask enables no existing CU. */
int iefwd_set_cu_mask(iefwd_instance *inst, const uint32_t *mask, uint32_t n_words);

/* Copies the mask of the stream the instance currently launches on (the one
 * applied at the last submit, or the initial all-CU mask). */
int iefwd_get_cu_mask(const iefwd_instance *inst, uint32_t *mask, uint32_t n_words);

/* ---- serving ---------------------------------------------------------------------- */

/* Submits one batch: x is fp32 [batch, seq, d_model], row-major.  Asynchronous.
 * x_is_device = 0: x is host memory, copied before the call returns.
 * x_is_device = 1: x is device memory that must stay valid and unmodified
 *                  until iefwd_wait / iefwd_read_logits returns.
 * 1 <= batch <= max_batch, 1 <= seq <= max_seq.  One batch may be in flight per
 * instance: submitting while one is in flight returns ESTATE.  A pending quota
 * change is applied first (the new stream waits for the previous one). */
int iefwd_submit(iefwd_instance *inst, const float *x, uint32_t batch, uint32_t seq,
                 int x_is_device);

/* Decode step (instances created with kv_cache = 1): one new token per
 * sequence at position `pos`.  x is fp32 [batch, d_model], the embeddings of
 * the new tokens (host or device, as for iefwd_submit).  Every layer appends
 * the tokens' K and V to its cache at `pos` and attends to positions
 * 0 .. pos; the output (iefwd_read_logits) is fp32 [batch, 1, n_out or
 * d_model].  The cache holds what the last iefwd_submit (the prompt,
 * positions 0 .. seq - 1) and the decode steps since wrote: 1 <= batch <=
 * the prompt's batch, pos <= the cached length (pos < length rewrites from
 * there on) and pos < max_seq; otherwise EINVAL, or ESTATE without a prompt
 * or a KV cache.  Asynchronous; one batch in flight per instance. */
int iefwd_decode(iefwd_instance *inst, const float *x, uint32_t batch, uint32_t pos, int x_is_device);

/* Blocks until the in-flight batch (if any) is complete. */
int iefwd_wait(iefwd_instance *inst);

/* Waits for the last submitted batch, then copies its output (fp32
 * [batch, seq, n_out], or [batch, seq, d_model] when n_out = 0) to out.
 * n_floats must equal that element count exactly (else EINVAL).
 * ESTATE if nothing was submitted yet. */
int iefwd_read_logits(iefwd_instance *inst, float *out, size_t n_floats, int out_is_device);

/* Device time of the last completed batch in milliseconds, from HIP events on
 * the instance's stream (the per-iteration time an elasticity controller
 * watches, Sec. 3.4.1).  ESTATE if no batch has completed. */
int iefwd_last_batch_ms(iefwd_instance *inst, float *ms);

/* Number of kernels the instance has launched since it was created (every
 * kernel of every submitted batch).  An elasticity controller samples it once
 * per control period to get the instance's kernel rate (Sec. 3.4.1). */
int iefwd_kernels_launched(const iefwd_instance *inst, uint64_t *count);

/* The hipStream_t the instance currently launches on (for external ordering). */
int iefwd_get_stream(iefwd_instance *inst, void **hip_stream);

/* ---- per-kernel timing ------------------------------------------------------------- */

/* Kernel classes of the forward pass. */
#define IEFWD_K_QKV      0u   /* QKV projection GEMM + bias + head scatter */
#define IEFWD_K_ATTN     1u   /* fused softmax attention */
#define IEFWD_K_OUTPROJ  2u   /* output projection GEMM + bias + residual */
#define IEFWD_K_FFN1     3u   /* FFN up GEMM + bias + GELU */
#define IEFWD_K_FFN2     4u   /* FFN down GEMM + bias + residual */
#define IEFWD_K_LN       5u   /* LayerNorm kernels (including the fused final LN + head) */
#define IEFWD_K_BWD_GEMM 6u   /* training: the backward pass's GEMMs (input and weight gradients) */
#define IEFWD_K_BWD      7u   /* training: the other backward kernels (LayerNorm, attention, sums, transposes) */
#define IEFWD_K_OPTIM    8u   /* training: the AdamW update and the transposed weight copies */
#define IEFWD_K_COUNT    9u

/* enable != 0: every later launch of class `kind` records the kernel's own
 * start and end timestamps into a pair of HIP events (hipExtLaunchKernel);
 * iefwd_kernel_time sums those kernel durations over completed batches.
 * enable = 0 stops timing; both calls reset the sums.  ESTATE while a batch is
 * in flight. */
int iefwd_time_kernel(iefwd_instance *inst, uint32_t kind, int enable);
int iefwd_kernel_time(iefwd_instance *inst, uint32_t kind, double *total_ms, uint64_t *launches);

/* ---- training (an SLO-insensitive training function, Sec. 3.4.1 and 5.2) ----------------
 * A training instance runs whole training steps of a post-LN encoder on the
 * same quota machinery as an inference instance: iefwd_set_quota* apply at
 * the next step, iefwd_last_batch_ms is the last step's device time and
 * iefwd_kernels_launched counts its kernels.  One step: forward (saving the
 * activations the backward needs), loss = mean over the B*S tokens of the
 * softmax cross-entropy of the token's n_out logits against its label,
 * backward of every parameter, one AdamW update (decoupled weight decay on the
 * weight matrices only, bias-corrected moments), all on the GPU.  The
 * optimiser keeps fp32 master weights and moments; the forward reads their
 * bf16 (matrices, biases) or fp32 (LayerNorm) copies.  Deterministic: a step's
 * results are a function of the config, the parameters, the inputs and the
 * step count, independent of the quota. */
typedef struct iefwd_train_params {
    uint32_t abi_version;   /* must be IEFWD_ABI_VERSION */
    uint32_t reserved0;
    float    lr;            /* learning rate (default 1e-4) */
    float    beta1, beta2;  /* moment decay rates (0.9, 0.999) */
    float    eps;           /* denominator offset (1e-8) */
    float    weight_decay;  /* decoupled weight decay of the weight matrices (0.01) */
    float    reserved1;
} iefwd_train_params;

/* Fills *tp with the defaults above. No status. */
void iefwd_train_params_init(iefwd_train_params *tp);

/* Creates a training instance: as iefwd_create (same weights for the same
 * config), plus the optimiser state (4 fp32 copies of the parameters) and the
 * activations of max_batch * max_seq tokens per layer.  Needs pre_ln = 0,
 * kv_cache = 0, 1 <= n_out <= 16 (classes), head dim 64 and max_seq <= 128;
 * EINVAL otherwise, EVERSION for a wrong tp->abi_version. */
int iefwd_train_create(const iefwd_config *cfg, const iefwd_train_params *tp, int device, iefwd_instance **out);

/* One training step, asynchronous like iefwd_submit: x fp32 [batch, seq,
 * d_model] and labels int32 [batch, seq] (class indices in [0, n_out); a
 * label outside that range counts as no class), both on the host (copied
 * before return) or both on the device (valid until the step completes).
 * batch * seq must be a multiple of 64.  ESTATE on an inference instance or
 * with a step or batch in flight.  After the step, iefwd_read_logits returns
 * the step's logits (computed before its update). */
int iefwd_train_step(iefwd_instance *inst, const float *x, const int32_t *labels, uint32_t batch, uint32_t seq,
                     int inputs_are_device);

/* Waits for the step in flight and writes its loss (before the update).
 * ESTATE if no step has run. */
int iefwd_train_loss(iefwd_instance *inst, float *loss);

/* Number of completed optimiser steps. */
int iefwd_train_steps(const iefwd_instance *inst, uint64_t *steps);

#define IEFWD_TRAIN_MASTER   0u   /* fp32 master weights */
#define IEFWD_TRAIN_GRAD     1u   /* gradients of the last step */
#define IEFWD_TRAIN_MOMENT1  2u   /* AdamW first moments */
#define IEFWD_TRAIN_MOMENT2  3u   /* AdamW second moments */

/* Copies one tensor of the optimiser state as fp32 in the logical layout of
 * iefwd_export_tensor (matrices [in, out]); slots as there (per layer 0..11;
 * layer = n_layers: 14 Wh, 15 bh).  n_floats must equal the tensor's size.
 * Waits for the step in flight. */
int iefwd_train_export(iefwd_instance *inst, uint32_t layer, uint32_t slot, uint32_t what, float *host_dst,
                       size_t n_floats);

/* ---- weights ------------------------------------------------------------------------ */

/* Copies a stored tensor to host memory in its logical layout.
 * Per-layer slots (layer < n_layers): 0 Wqkv bf16 [d, 3d], 1 bqkv bf16 [3d],
 * 2 Wo bf16 [d, d], 3 bo bf16 [d], 4 ln1 gamma f32 [d], 5 ln1 beta f32 [d],
 * 6 W1 bf16 [d, F], 7 b1 bf16 [F], 8 W2 bf16 [F, d], 9 b2 bf16 [d],
 * 10 ln2 gamma f32 [d], 11 ln2 beta f32 [d].
 * Global slots (layer == n_layers): 12 final-LN gamma f32 [d], 13 beta f32 [d],
 * 14 Wh bf16 [d, n_out], 15 bh bf16 [n_out] (only when n_out > 0).
 * Matrices are [in, out] row-major.  bytes must equal the tensor size. */
int iefwd_export_tensor(const iefwd_instance *inst, uint32_t layer, uint32_t slot,
                        void *host_dst, size_t bytes);

/* ---- errors --------------------------------------------------------------------------- */

/* Message for the last failed call on this thread ("" if none).  Valid until
 * the next iefwd_* call on this thread.  Never NULL. */
const char *iefwd_last_error(void);
/* Static name of a status code.  Never NULL. */
const char *iefwd_status_string(int status);

/* ---- quota controller ------------------------------------------------------------ */

/* The fast scale-up/down control of Sec. 3.4.1 (Alg. 2, IssueToken) with CUs as
 * tokens.  Pure host code: it neither reads nor changes any instance; the
 * caller reports each co-located instance's observations once per control
 * period, calls iefwd_ctl_issue, and applies the returned quota and first
 * mask bit with iefwd_set_quota_at.  Calls on one controller are serialised
 * by the caller.
 *
 * Per period, for every instance: R_current = kernels launched during the
 * period (RW keeps the last `window` of them), KLC = duration of its last
 * completed batch (T_current; T_min = the smallest reported).  SLO-sensitive
 * instances (evaluated first, in id order), dT = (T_current - T_min) / T_min,
 * or 0 in a period with no KLC reported:
 *   dT > eta_violation                 -> EMERGENCY,  MaxTokens * limit
 *   its RW sums to 0                   -> RECOVERY,   MaxTokens * request
 *   every other instance's RW is 0     -> RECOVERY,   min(R_last * eta_increase, MaxTokens)
 *   otherwise                          -> CONTENTION, MaxTokens * request
 * other instances, from the shared state:
 *   NONE (no SLO-sensitive instance)   -> MaxTokens * limit
 *   EMERGENCY                          -> min(MaxTokens * request, R_last) / (1 + dT_raiser)
 *   RECOVERY                           -> min(R_last * eta_increase, MaxTokens * limit)
 *   CONTENTION                         -> R_last
 * Only the instance that raised EMERGENCY can change the state.  Tokens become
 * quotas round(R / granule) * granule clamped to [min_quota, MaxTokens] and
 * fitted so that no two placements share a CU (a shared CU slows both, and an
 * instance moved onto CUs where another's batch is still in flight waits
 * behind it): SLO-sensitive quotas are scaled down (granule, >= min_quota)
 * until every other instance can keep min_quota, the others are scaled into
 * the CUs that remain.  SLO-sensitive instances take mask bits upward from 0,
 * the others downward from the top, each group in id order.  Overlap remains
 * only if the instances outnumber MaxTokens / min_quota.
 * Readings where the paper is silent: the eta defaults; dividing by the KLC
 * ratio 1 + dT rather than dT (dT < 1 would scale up); the SLO scale-up capped
 * at MaxTokens; T_min over the whole history; no KLC carried over from one
 * period to the next (a held-over KLC would keep an instance that went idle
 * after a violation in EMERGENCY, so it could never reach RECOVERY). */
typedef struct iefwd_ctl iefwd_ctl;

enum { IEFWD_CTL_NONE = 0, IEFWD_CTL_EMERGENCY = 1, IEFWD_CTL_RECOVERY = 2, IEFWD_CTL_CONTENTION = 3 };

typedef struct {
    uint32_t abi_version;    /* = IEFWD_ABI_VERSION */
    uint32_t max_tokens;     /* MaxTokens: CUs that can be issued (the device's CU count); >= 1 */
    uint32_t window;         /* RW length in control periods; >= 1 */
    uint32_t granule;        /* quotas are multiples of this many CUs; >= 1 */
    uint32_t min_quota;      /* smallest quota issued; 1 .. max_tokens */
    uint32_t flags;          /* 0 or IEFWD_CTL_TEMPORARY_YIELD (below) */
    double eta_violation;    /* relative KLC increase that raises EMERGENCY; >= 0 */
    double eta_increase;     /* multiplicative scale-up per period; >= 1 */
} iefwd_ctl_params;

/* flags: Sec. 3.4.1 calls the co-located instances' scale-down under EMERGENCY
 * temporary, while Alg. 2 keeps R_last in CONTENTION, so that without
 * this flag a yielded issue becomes R_last and is undone only through
 * RECOVERY (the SLO-sensitive instances idle for a whole window).  With it a
 * yielded issue leaves R_last, the plan held before the emergency, unchanged:
 * consecutive EMERGENCY periods do not compound the yield, and CONTENTION
 * afterwards restores the plan. */
#define IEFWD_CTL_TEMPORARY_YIELD 1u

/* Defaults: max_tokens 256, window 4, granule 8, min_quota 8, flags 0,
 * eta_violation 0.2, eta_increase 1.25. */
int iefwd_ctl_params_init(iefwd_ctl_params *p);

/* EINVAL on a field out of range, EVERSION on another ABI version. */
int iefwd_ctl_create(const iefwd_ctl_params *p, iefwd_ctl **out);
int iefwd_ctl_destroy(iefwd_ctl *ctl);   /* NULL accepted */

/* Adds an instance with <request, limit> as fractions of MaxTokens
 * (0 < request <= limit <= 1); *id = 0, 1, ... in order of addition. */
int iefwd_ctl_add(iefwd_ctl *ctl, double request, double limit, int slo_sensitive, uint32_t *id);

/* Observation of instance `id` for the current period: kernels launched during
 * it, and the KLC in milliseconds of the last batch it completed in the period
 * (<= 0 if none).  A later report in the same period replaces the earlier. */
int iefwd_ctl_report(iefwd_ctl *ctl, uint32_t id, uint64_t kernels, double klc_ms);

/* Ends the period.  Writes, for each of the n instances in id order, the
 * issued tokens (R_issue), the quota in CUs and the first mask bit of its
 * placement; any output pointer may be NULL.  EINVAL unless n equals the
 * number of instances. */
int iefwd_ctl_issue(iefwd_ctl *ctl, double *tokens, uint32_t *quotas, uint32_t *firsts, uint32_t n);

/* The shared state after the last issue (IEFWD_CTL_*). */
int iefwd_ctl_state(const iefwd_ctl *ctl, int32_t *state);

/* ---- per-kernel entry points (parity tests) ------------------------------------------
 * Each launches one kernel of the forward pass on `stream` (a hipStream_t, NULL
 * = the null stream of the current device) and returns without synchronising.
 * All pointers are device pointers; shapes are validated (EINVAL). */

/* GEMM epilogues */
#define IEFWD_EPI_BIAS_BF16       0u  /* out bf16 [M, N] = A W^T + b */
#define IEFWD_EPI_BIAS_GELU_BF16  1u  /* out bf16 [M, N] = GELU(A W^T + b) */
#define IEFWD_EPI_BIAS_RESID_F32  2u  /* out f32  [M, N] = resid + A W^T + b */

/* out = epilogue(A W^T + b): A bf16 [M, K] row-major (activations), W bf16
 * [N, K] row-major (the weight stored output-major), bias bf16 [N], resid f32
 * [M, N] (only for IEFWD_EPI_BIAS_RESID_F32, else may be NULL).  Accumulates
 * in fp32 with bf16 MFMA.  M >= 0, N % 64 == 0, K % 64 == 0. */
int iefwd_test_gemm(uint32_t epilogue, const void *a, const void *w, const void *bias,
                    const float *resid, void *out, uint32_t M, uint32_t N, uint32_t K,
                    void *stream);

/* Pure host function: how iefwd_test_gemm and the forward pass run an
 * M x N x K product on a stream with n_cu CUs; ln_residual != 0 for the
 * post-LN residual epilogue (the out-projection and FFN-down of a post-LN
 * model), whose tile choice skips the 128 x 192 tile.  k_order: the K summation order
 * of the weight shape (0 = sequential 64-wide K tiles, 1 = even and odd K
 * tiles summed separately, then added); tile_order: the order the chosen tile
 * sums in, always equal to k_order; tile_m x tile_n: the output tile (tokens x
 * features).  align: the width every tile must divide (d_model for the QKV
 * product, else N).  EINVAL unless 1 <= M <= 2^24, N and K are multiples of 64
 * in [64, 65536], align is a multiple of 64 dividing N and 1 <= n_cu <= 1024. */
int iefwd_test_gemm_plan(uint32_t M, uint32_t N, uint32_t K, uint32_t align, uint32_t n_cu, uint32_t ln_residual,
                         uint32_t *k_order, uint32_t *tile_order, uint32_t *tile_m, uint32_t *tile_n);

/* The decode-step product for M <= 16 activation rows: the same operands and
 * epilogues as iefwd_test_gemm, N % 16 == 0, K % 32 == 0.  Its K summation
 * order differs from iefwd_test_gemm's (bound by reading W once, not by the
 * matrix cores).  ln_z non-NULL: the activations are LayerNorm(z) instead of a
 * (a is then ignored): z f32 [M, K], ln_gamma / ln_beta f32 [K], row
 * statistics in fp32, the normalised rows rounded to bf16; needs K <= 4096
 * and M * K <= 16384 (EINVAL otherwise).  This is how a pre-LN block's LayerNorm is fused
 * into its QKV and FFN-up products during decode. */
int iefwd_test_gemm_skinny(uint32_t epilogue, const void *a, const void *w, const void *bias,
                           const float *resid, void *out, uint32_t M, uint32_t N, uint32_t K,
                           const float *ln_z, const float *ln_gamma, const float *ln_beta, float ln_eps,
                           void *stream);

/* The packed weight layout of the decode-step product (Sec. 3.4.1 footnote:
 * an inference iteration is one batch; a decode iteration reads every weight
 * once).  dst (N * K bf16, caller-owned, device) = W [N, K] rearranged for
 * `groups` K-groups (1, 2 or 4; N % (16 / groups) == 0, K % (32 * groups) ==
 * 0): 16-byte piece i of dst holds W[f][k .. k + 7] with
 *   i = (b * steps + s) * 64 + l,  steps = K / (32 groups),
 *   r = l % 16, c = l / 16, f = b * (16 / groups) + r % (16 / groups),
 *   k = (r / (16 / groups)) * (K / groups) + 32 s + 8 c,
 * so that each wave load instruction of the product reads 1 KB of
 * consecutive addresses.  Instances created with kv_cache = 1 keep such a copy
 * of their four matrices per layer. */
int iefwd_test_skinny_pack(const void *w, void *dst, uint32_t N, uint32_t K, uint32_t groups, void *stream);

/* iefwd_test_gemm_skinny on the packed copy (iefwd_test_skinny_pack) of W
 * instead of W itself; `groups` must be the K-group count the product uses
 * for (M, N, K) with or without the LayerNorm prologue
 * (iefwd_test_skinny_groups), else EINVAL.  Results equal
 * iefwd_test_gemm_skinny's bit for bit. */
int iefwd_test_gemm_skinny_packed(uint32_t epilogue, const void *a, const void *w_packed, uint32_t groups,
                                  const void *bias, const float *resid, void *out, uint32_t M, uint32_t N, uint32_t K,
                                  const float *ln_z, const float *ln_gamma, const float *ln_beta, float ln_eps,
                                  void *stream);

/* The K-group count (1, 2 or 4) of the decode-step product for M rows,
 * N % 16 == 0 and K % 32 == 0, with (ln != 0) or without the LayerNorm
 * prologue.  Host only. */
int iefwd_test_skinny_groups(uint32_t M, uint32_t N, uint32_t K, int ln, uint32_t *groups);

/* QKV projection with head scatter: A bf16 [batch*seq, d], W bf16 [3d, d],
 * bias bf16 [3d].  Writes Q and K as bf16 [batch, heads, seq, dh] and V
 * transposed as bf16 [batch, heads, dh, seq_pad], seq_pad = seq rounded up to
 * a multiple of 64 (entries past seq are left untouched). */
int iefwd_test_gemm_qkv(const void *a, const void *w, const void *bias, void *q, void *k,
                        void *vt, uint32_t batch, uint32_t seq, uint32_t d_model,
                        uint32_t n_heads, void *stream);

/* ctx bf16 [batch, seq, heads*dh] = softmax(Q K^T / sqrt(dh) [+ causal]) V per
 * (batch, head), from Q, K bf16 [batch, heads, seq, dh] and Vt bf16
 * [batch, heads, dh, seq_pad] (seq_pad = seq rounded up to a multiple of 64;
 * the padding may hold any bits).  dh in {64, 128}. */
int iefwd_test_attention(const void *q, const void *k, const void *vt, void *ctx,
                         uint32_t batch, uint32_t n_heads, uint32_t seq, uint32_t head_dim,
                         int causal, void *stream);

/* Row LayerNorm of z f32 [rows, d]: out_f32 (may be NULL) and out_bf16 (may be
 * NULL) get gamma * (z - mean) / sqrt(var + eps) + beta. */
int iefwd_test_layernorm(const float *z, const float *gamma, const float *beta,
                         float *out_f32, void *out_bf16, uint32_t rows, uint32_t d,
                         float eps, void *stream);

/* LayerNorm followed by the per-token head: logits f32 [rows, n_out] =
 * LN(z) Wh^T + bh with Wh bf16 [n_out, d] (output-major), bh bf16 [n_out]. */
int iefwd_test_ln_head(const float *z, const float *gamma, const float *beta,
                       const void *wh, const void *bh, float *logits, uint32_t rows,
                       uint32_t d, uint32_t n_out, float eps, void *stream);

/* Decode attention: one query per (batch, head), q bf16 [batch, heads, dh],
 * against keys 0 .. n_keys - 1 of K bf16 [batch, heads, k_rows, dh] and
 * V^T bf16 [batch, heads, dh, vt_stride] (columns >= n_keys may hold any
 * bits); ctx bf16 [batch, heads * dh].  dh in {64, 128}, 1 <= n_keys <= 8192,
 * k_rows >= n_keys, vt_stride >= n_keys and a multiple of 64,
 * batch * heads <= 65535.  The keys are split into chunks (64 keys up to 2048,
 * else 256) whose partial results a second kernel combines; the call
 * allocates that scratch and returns after the stream has drained. */
int iefwd_test_decode_attention(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch,
                                uint32_t n_heads, uint32_t n_keys, uint32_t head_dim, uint32_t k_rows,
                                uint32_t vt_stride, void *stream);

/* Allocation-free variant of iefwd_test_decode_attention, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Same arguments, kernels and
 * results (bit for bit); the chunks' partial results go to a fixed device
 * scratch of 8 MiB that the library holds on each GPU it runs on until the
 * process ends, instead of a per-call allocation.  Needs
 * batch * n_heads * chunks * (head_dim + 2) * 4 <= 8 MiB, chunks =
 * ceil(n_keys / 64) up to 2048 keys, else ceil(n_keys / 256) (EINVAL
 * otherwise).  Runs on the current device (stream must belong to it) and
 * returns without synchronising.  The call allocates nothing and frees
 * nothing.  Every call on one GPU uses the same scratch: calls that overlap
 * on one GPU (on different streams, or from different threads) race and
 * must be serialised by the caller. */
int iefwd_decode_attention_noalloc(const void *q, const void *k, const void *vt, void *ctx, uint32_t batch,
                                   uint32_t n_heads, uint32_t n_keys, uint32_t head_dim, uint32_t k_rows,
                                   uint32_t vt_stride, void *stream);

/* CU residency probe: launches n_groups workgroups of 64 threads on `stream`;
 * workgroup g writes out[2g] = XCC id, out[2g+1] = the hardware id register
 * (CU, SIMD, shader-array and shader-engine fields).  out: device uint32
 * [2 * n_groups]. */
int iefwd_test_cu_probe(void *stream, uint32_t n_groups, uint32_t *out);

#ifdef __cplusplus
}
#endif

#endif /* IEFWD_H */
