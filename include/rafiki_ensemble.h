/*
 * rafiki_ensemble.h -- C ABI of the MI355X (gfx950) ensemble-inference hot path.
 *
 * The paper's inference service deploys a list of trained models as one inference
 * job (Section 3: the SDK gets model instances -- a model name plus the names of its
 * parameters in the parameter server -- creates the inference job with them and
 * deploys it; workers then fetch the parameters).  Each scheduled batch of the
 * oldest b requests is served by the forward pass m.infer(q_{0:b}) of the models
 * selected by the binary vector v, v != 0 (Section 5.1, Algorithm "Inference";
 * Section 5.2 and Table 2), and the selected models' results are averaged
 * (Section 1).  This library maps those steps to:
 *
 *   rafiki_ensemble_create   job creation + deployment: parameters copied to HBM
 *   rafiki_ensemble_infer    one scheduled batch with one selection vector
 *   rafiki_ensemble_infer_vote     the same batch combined by majority vote (Section 5.2)
 *   rafiki_ensemble_model_logits   one model's raw logits (diagnostics, tests)
 *   rafiki_ensemble_destroy  teardown
 *
 * Conventions
 * - Every function returns an int status (RAFIKI_OK or a negative code) and never
 *   throws; rafiki_last_error() returns a thread-local message for the last failure
 *   on the calling thread.
 * - Host pointers: everything inside rafiki_model_desc / rafiki_layer (read during
 *   create only; the caller may free them on return).
 * - Device pointers: `batch`, `out_probs`, `out_labels`, `out_logits` are caller-owned,
 *   contiguous device buffers that must stay valid until `stream` has passed the
 *   enqueued work and must not alias each other.
 * - infer / model_logits only enqueue work on `stream` (a hipStream_t; 0 = the null
 *   stream) and return; kernel faults surface at the next synchronisation.
 * - A handle owns its device weights and a workspace sized for opts.max_batch, which
 *   every call shares: issue the calls on one stream, or make each call's stream wait
 *   for the previous call's work (an event); calls from several threads at once are
 *   not supported.
 * - Inputs are not checked on the device: token ids outside [0, vocab) read a zero
 *   embedding row (no error), and image values must be finite.
 * - Results are deterministic: the same inputs, mask and n give bitwise-identical
 *   outputs (sums are taken in a fixed order; the only atomics are maxima, which do
 *   not depend on order).
 */
#ifndef RAFIKI_ENSEMBLE_H
#define RAFIKI_ENSEMBLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
  RAFIKI_OK = 0,
  RAFIKI_ERR_INVALID = -1,      /* bad argument: null pointer, mask, n, malformed model */
  RAFIKI_ERR_UNSUPPORTED = -2,  /* valid but not implemented (e.g. a layer shape) */
  RAFIKI_ERR_NOMEM = -3,        /* device or host allocation failed */
  RAFIKI_ERR_HIP = -4           /* a HIP runtime call failed (e.g. no device) */
};

/* Compute precision of a handle.
 * RAFIKI_FP32: fp32 weights, activations and accumulation.
 * RAFIKI_BF16: weights rounded once (nearest, ties to even) to bfloat16, activations
 *   stored as bfloat16 between layers, fp32 accumulation, fp32 batch-norm fold and
 *   epilogue, fp32 logits, softmax and combine. */
enum { RAFIKI_FP32 = 0, RAFIKI_BF16 = 1 };

/* Request kinds. */
enum {
  RAFIKI_INPUT_IMAGE_NCHW_F32 = 0, /* batch = float [n, c, h, w] */
  RAFIKI_INPUT_TOKENS_I32 = 1      /* batch = int32 [n, h] token ids (h = sequence length) */
};

/* Layer operations.  A layer's output tensor id is its index in the model's layer
 * list; id -1 is the model input.  Layers must be topologically ordered. */
enum {
  RAFIKI_OP_CONV2D = 1,         /* cross-correlation, zero padding, floor output size;
                                   weight OIHW [c_out, c_in, kh, kw]; optional bias;
                                   optional inference BN (gamma, beta, mean, var, eps);
                                   optional residual tensor `input2` added before ReLU */
  RAFIKI_OP_MAXPOOL2D = 2,      /* kh x kw window, stride, pad (padding never wins) */
  RAFIKI_OP_GLOBAL_AVGPOOL = 3, /* mean over all spatial positions -> vector [c] */
  RAFIKI_OP_FC = 4,             /* z = W x + b; weight [c_out, c_in]; a spatial input
                                   [c, h, w] is flattened in (c, h, w) order */
  RAFIKI_OP_EMBEDDING = 5,      /* table [c_in = vocab, c_out = dim]; input must be -1 */
  RAFIKI_OP_CONV1D_MAXTIME = 6, /* valid conv1d over time, weight [c_out, c_in, kw],
                                   bias, ReLU, then max over time -> vector [c_out] */
  RAFIKI_OP_CONCAT = 7          /* vectors `input` then `input2`, joined along channels */
};

typedef struct rafiki_ensemble_s* rafiki_ensemble_t;

typedef struct {
  int op;
  int input, input2;            /* tensor ids; input2 = residual (CONV2D) / second operand
                                   (CONCAT), or -1 */
  int c_in, c_out;
  int kh, kw, stride, pad;
  int relu;                     /* nonzero: apply ReLU last (after the residual add) */
  const float* weight;          /* host fp32, canonical layout above; NULL for pools/concat */
  const float* bias;            /* host fp32 [c_out] or NULL */
  const float* bn_gamma;        /* host fp32 [c_out]; all four NULL = no batch-norm */
  const float* bn_beta;
  const float* bn_mean;
  const float* bn_var;
  float bn_eps;
} rafiki_layer;

typedef struct {
  int n_layers;
  const rafiki_layer* layers;   /* the last layer produces the logits [n_classes] */
  int n_classes;
} rafiki_model_desc;

typedef struct {
  int input_kind;               /* RAFIKI_INPUT_* */
  int c, h, w;                  /* image shape; for tokens h = sequence length, c = w = 1 */
  int vocab;                    /* token vocabulary size (tokens only) */
  int precision;                /* RAFIKI_FP32 or RAFIKI_BF16 */
  int max_batch;                /* largest n accepted by infer; the workspace is sized for it */
} rafiki_ensemble_opts;

/* Create an ensemble of `n_models` (1..32) models sharing the input shape and
 * n_classes.  Validates the layer lists, folds batch-norm into a per-channel fp32
 * scale and shift (computed in fp64), rounds weights to the compute precision,
 * packs them for the kernels, uploads them synchronously to the current device and
 * sizes the workspace for opts->max_batch.  In bf16, conv1d max-over-time layers that
 * read one sequence and whose outputs are joined only by concatenations (the TextCNN's
 * kernel widths) are packed as one GEMM whose max over time writes the concatenated
 * vector; every output value is that of its own layer's sum of products (environment
 * RAFIKI_FUSE_BRANCHES=0 at create keeps them apart).
 * Errors: RAFIKI_ERR_INVALID (null pointers, n_models out of range, mismatched
 * shapes or classes, malformed layers), RAFIKI_ERR_UNSUPPORTED, RAFIKI_ERR_NOMEM,
 * RAFIKI_ERR_HIP.  On error *out is set to NULL. */
int rafiki_ensemble_create(const rafiki_model_desc* models, int n_models,
                           const rafiki_ensemble_opts* opts, rafiki_ensemble_t* out);

/* Serve one batch: for every model m whose bit m is set in model_subset_mask (bit m =
 * model m in creation order), run its forward pass over the n requests in `batch`;
 * then out_probs[i, :] = mean over the selected models of softmax(logits_m[i, :]) and
 * out_labels[i] = lowest class index attaining the maximum of out_probs[i, :].
 * `batch` follows opts.input_kind; out_probs is fp32 [n, n_classes] row-major;
 * out_labels is int32 [n].  Requires 1 <= n <= max_batch, mask != 0 and no bit at
 * position >= n_models (else RAFIKI_ERR_INVALID).  Enqueue-only on `stream`, except
 * that the first call (infer or model_logits) with a given n blocks while it times
 * the candidate tile configurations of every layer inside forward passes on `stream`
 * (set the environment variable RAFIKI_AUTOTUNE=0 to use fixed defaults instead), and
 * the first infer of a (n, mask) with three or more models blocks while it times the
 * model schedules (see rafiki_ensemble_get_schedule).  Neither choice changes a
 * result: every tile candidate sums each output in the same order, and a schedule
 * only orders the same launches. */
int rafiki_ensemble_infer(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                          float* out_probs, int32_t* out_labels, void* stream);

/* Serve one batch like rafiki_ensemble_infer, but combine the selected models by
 * majority vote, the aggregation of the paper's ensemble experiment (Section 5.2):
 * each selected model votes for the lowest class index attaining the maximum of its
 * logits; out_labels[i] is the class with the most votes, and a tie between classes
 * goes to the class voted for by the lowest-numbered selected model (creation order is
 * the priority order: create the models sorted from the most to the least accurate to
 * resolve ties as the paper does).  out_votes is fp32 [n, n_classes] row-major: the
 * fraction of the selected models voting for each class (each row sums to 1).
 * Argument rules, errors and stream behaviour as rafiki_ensemble_infer; the result is
 * exact (integer votes) and deterministic. */
int rafiki_ensemble_infer_vote(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                               float* out_votes, int32_t* out_labels, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): serve one batch exactly like
 * rafiki_ensemble_infer (same arguments, rules, kernels and bitwise-identical
 * results), but the call's scratch -- the split-K partial sums of every selected
 * model's GEMMs and the keys of the fused max-over-time epilogues -- lives in a static
 * device array of the library (64 MiB per GPU, allocated when the library's code is
 * loaded on that GPU and held until the process ends) instead of the handle's
 * workspace.  It calls no hipMalloc / hipFree.  A call whose scratch exceeds 64 MiB
 * returns RAFIKI_ERR_UNSUPPORTED before enqueueing anything (the largest needs are
 * deep split-K layers at large n: use infer there).  The keys are cleared on `stream`
 * at the start of every call; the array otherwise keeps the last call's contents.
 * Every call on one GPU, from any handle, shares that GPU's array: calls whose work
 * overlaps on the device race (issue them on one stream, or order them with events).
 * Like infer, the first call with a new n (or a new (n, mask) with three or more
 * models) blocks while it tunes. */
int rafiki_ensemble_infer_noalloc(rafiki_ensemble_t h, const void* batch, int n, uint32_t model_subset_mask,
                                  float* out_probs, int32_t* out_labels, void* stream);

/* Run model `model` alone and write its fp32 logits [n, n_classes] to out_logits.
 * Same argument rules as infer.  Enqueue-only on `stream`. */
int rafiki_ensemble_model_logits(rafiki_ensemble_t h, int model, const void* batch, int n,
                                 float* out_logits, void* stream);

/* Number of models and classes of a handle (host-side query). */
int rafiki_ensemble_info(rafiki_ensemble_t h, int* n_models, int* n_classes, int* max_batch);

/* Diagnostics: per-launch timing.  Kernel classes of rafiki_trace_rec.kind: */
enum {
  RAFIKI_K_CONV_MFMA = 0,      /* bf16 implicit-GEMM conv / FC / conv1d on matrix cores */
  RAFIKI_K_SPLITK_REDUCE = 1,  /* ordered sum of split-K partials + epilogue */
  RAFIKI_K_CONV_F32 = 2,       /* fp32 direct conv / FC */
  RAFIKI_K_STAGE = 3,          /* NCHW fp32 -> NHWC input staging */
  RAFIKI_K_POOL = 4,           /* max-pool, global average pool, max over time */
  RAFIKI_K_EMBED = 5,          /* embedding gather */
  RAFIKI_K_CONCAT = 6,         /* vector concatenation */
  RAFIKI_K_COMBINE = 7,        /* softmax + ensemble mean + argmax */
  RAFIKI_K_VOTE = 8,           /* per-model argmax + majority vote */
  RAFIKI_K_FUSED_NET = 9       /* whole forward pass of small CNNs, one workgroup per image and model */
};
typedef struct {
  int kind;                     /* RAFIKI_K_* */
  int model, layer;             /* -1 for staging and combine */
  double flops;                 /* algorithmic FLOPs (2 x unpadded MACs) of the launch */
  double bytes;                 /* algorithmic bytes: each input, weight and output once */
  float ms;                     /* kernel execution time: elapsed time between the HIP
                                   events the launch records at the kernel's start and end
                                   (hipExtLaunchKernelGGL start/stop events) */
  int tile_cfg;                 /* bf16 GEMM launches (conv_mfma, splitk_reduce): the tile
                                   configuration used (rafiki_tile_config), or the number of
                                   configurations for the direct conv kernel; -1 otherwise */
  int splits;                   /* the same launches: K splits (1 = unsplit); 0 otherwise */
} rafiki_trace_rec;

/* Per-launch event timing of subsequent infer / model_logits calls on this handle:
 * enable = 0 off; 1 on, with the selected models run one after another on the
 * caller's stream (each kernel has the GPU to itself); 2 on, with the models on their
 * own streams in their kept schedule (kernels time their share of a concurrent step;
 * no schedule is timed while tracing).  Also discards unread records.  Tracing adds two
 * event records per launch; it does not change results.  Other values:
 * RAFIKI_ERR_INVALID. */
int rafiki_ensemble_trace(rafiki_ensemble_t h, int enable);

/* Set *count to the number of traced launches.  If cap >= *count, wait for them, copy
 * the records (in launch order) to `out` and discard them; otherwise copy nothing and
 * keep them (call again with a larger buffer).  Host-blocking. */
int rafiki_ensemble_trace_read(rafiki_ensemble_t h, rafiki_trace_rec* out, int cap, int* count);

/* Standalone kernels of the path, on caller-owned contiguous device buffers, enqueued on
 * `stream` (hipStream_t as void*; 0 = the null stream).  They are the kernels infer uses,
 * exposed for measurement and for callers that hold their own tensors (for example logits
 * of models that ran on other GPUs and were gathered, the model-sharded layout of the
 * paper's one-model-per-GPU deployment).  Argument errors return RAFIKI_ERR_INVALID
 * before any device call; nothing is allocated.
 *
 * Ensemble combine (Section 1; Section 5.2): logits fp32 [n_models][n][n_classes]; the
 * mean of the per-model softmax to out_probs fp32 [n][n_classes] and its first-index
 * argmax to out_labels int32 [n].  1 <= n_models <= 32, n >= 1, 1 <= n_classes <= 1024. */
int rafiki_combine_mean(const float* logits, int n_models, int n, int n_classes, float* out_probs,
                        int32_t* out_labels, void* stream);

/* Majority vote over the same logits (ties to the lowest model index's class; see
 * rafiki_ensemble_infer_vote): vote fractions to out_votes [n][n_classes], winners to
 * out_labels [n].  Same limits. */
int rafiki_combine_vote(const float* logits, int n_models, int n, int n_classes, float* out_votes,
                        int32_t* out_labels, void* stream);

/* Max-pool k x k, stride, padding pad on each side (padding cells never win: they are -inf),
 * over bf16 NHWC x [n][h][w][c] into y [n][ho][wo][c] with ho = (h + 2 pad - k) / stride + 1
 * (floor; likewise wo).  c a multiple of 8; k >= 1, stride >= 1, 0 <= pad < k; ho, wo >= 1. */
int rafiki_maxpool_nhwc_bf16(const void* x, void* y, int n, int h, int w, int c, int k, int stride, int pad,
                             void* stream);

/* Global average pool over bf16 NHWC x [n][h][w][c] into y [n][c] (fp32 sums in a fixed
 * order, one rounding to bf16).  c a multiple of 8. */
int rafiki_global_avgpool_nhwc_bf16(const void* x, void* y, int n, int h, int w, int c, void* stream);

/* Diagnostics: the device's own ceilings, against which the kernels are judged.
 * rafiki_probe_mfma_bf16: `blocks` workgroups of 4 wavefronts; each wavefront issues
 * iters x 8 independent v_mfma_f32_32x32x16_bf16 on register-resident operands
 * (32768 FLOP each; nothing is loaded in the loop) and writes one fp32 checksum to
 * out[block * 4 + wave] (device, >= blocks * 4 floats).
 * rafiki_probe_hbm_read: reads `bytes` (a multiple of 16) of device memory at x
 * (16-byte aligned) once with 16-byte streaming loads over `blocks` workgroups of
 * 256 threads and writes one checksum per wavefront to out (device, >= blocks * 4
 * words).  Both enqueue on `stream` only; time them with events. */
int rafiki_probe_mfma_bf16(int blocks, int iters, float* out, void* stream);
int rafiki_probe_hbm_read(const void* x, long long bytes, int blocks, unsigned* out, void* stream);

/* Diagnostics: the GEMM kernel's main loop with nothing loaded from memory, to separate
 * what its LDS fragment reads, LDS writes and barriers cost from what its loads cost.
 * Each of `blocks` workgroups runs `ktiles` K tiles of 64; per K tile every wavefront
 * reads its fragments from LDS and issues its 32x32x16 bf16 MFMAs (4 k-steps of
 * TM x TN MFMAs, 32768 FLOP each).  variant 0: 8 wavefronts of 64x128 outputs
 * (TM = 2, TN = 4; the 256x256 8-wavefront tile); 1: 4 wavefronts of 128x128 (4, 4);
 * 2: 4 wavefronts of 64x64 (2, 2); 3: 8 wavefronts of 64x32 (2, 1).  sync != 0: each
 * K tile also writes the tile's (BM + BN) x 64 bf16 into LDS and passes a workgroup
 * barrier.  One fp32 checksum per wavefront goes to out[block * 8 + wave] (device,
 * >= blocks * 8 floats).  Enqueues on `stream` only. */
int rafiki_probe_mainloop(int variant, int sync, int blocks, int ktiles, float* out, void* stream);

/* Diagnostics: tile configurations of the bf16 GEMM kernel.  Configuration `cfg`
 * (0 .. count - 1) computes output tiles of bm pixels x bn channels with `waves`
 * wavefronts, `stages` K tiles of bk channels in flight.  Every configuration sums each
 * output's K terms in the same order, so all of them give bitwise-identical results.
 * Returns RAFIKI_ERR_INVALID past the last configuration; null outputs are skipped. */
int rafiki_tile_config(int cfg, int* bm, int* bn, int* waves, int* stages, int* bk);

/* Diagnostics: make every subsequent unsplit bf16 GEMM launch of the handle use tile
 * configuration `cfg` wherever its channel tile suits the layer's output channels
 * (other layers keep their tuned choice); cfg = -1 restores the tuned choice.
 * cfg = RAFIKI_TILE_DIRECT runs every layer that the direct conv kernel takes with that
 * kernel (bf16, no residual, one launch per model; 3x3 stride 1 from 64 to 64 or 128
 * channels, optionally with the fused 2x2 max-pool, or with 64 output channels, ReLU
 * and no pool 3x3 stride 1 or 7x7 stride 2 over an image's 8 storage channels), which the tuner
 * otherwise times as one more candidate.  Results are unchanged; only speed differs. */
#define RAFIKI_TILE_DIRECT 1000
int rafiki_ensemble_force_tile(rafiki_ensemble_t h, int cfg);

/* Schedule of the selected models' forward passes for one (n, model_subset_mask).
 * The models are independent until the combine and run on their own streams.  With
 * three or more selected models, the first infer / infer_vote of a (n, mask) pair times
 * each candidate schedule on `stream` (best of four runs each, the candidates in turn;
 * it blocks the caller once) and keeps the fastest: solo = -1, all models concurrently; solo = m, model m
 * alone on one lane while the other selected models run one after another on a second
 * lane, longest estimated alone time first (ascending = 0) or shortest first
 * (ascending = 1).  A schedule only orders the same launches, so it never changes a
 * result.  Environment RAFIKI_SCHEDULE_TUNING=0 at create skips the timing (all
 * concurrent unless set).
 * get_schedule: the kept choice (`ascending` may be NULL); RAFIKI_ERR_INVALID if none
 * has been chosen yet.
 * set_schedule: sets it (solo = -1 or a model of the subset); synchronises the device
 * and drops any kept graphs. */
int rafiki_ensemble_get_schedule(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int* solo, int* ascending);
int rafiki_ensemble_set_schedule(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int solo, int ascending);

/* Tile policy of a kept schedule (Section 5.1: the selected models share the GPU).  The
 * tuner keeps, beside each layer's fastest tile alone, a lean choice for every unsplit
 * GEMM layer with an output map of at most 14 x 14 pixels: its fastest tile among those
 * of 8 waves, at least 128 x 128, K tiles of 64 and an LDS ring of at most 64 KB, which loads fewer
 * bytes per FLOP than the small tiles such layers prefer alone and leaves room on each
 * compute unit for the other models' workgroups.  The schedule timing of infer times
 * every candidate schedule with both policies (when their tiles differ) and keeps the
 * faster (environment RAFIKI_LEAN_TILES=0 at create: never tried).  Every tile gives
 * the same bits, so the policy never changes a result.
 * With a model alone on its lane there is a third policy: the lean tiles, and that
 * model's layers that would take the direct conv kernel on their fastest GEMM tile
 * instead (the direct kernel's persistent workgroups fill each compute unit's LDS and
 * leave no room for the other lane's workgroups).
 * get_schedule_tiles: the kept choice's policy (*lean = 0: the tiles fastest alone, 1:
 * lean tiles, 2: lean tiles and GEMM tiles for the solo model); RAFIKI_ERR_INVALID if no
 * schedule has been chosen yet.
 * set_schedule_tiles: sets the policy of the kept schedule (lean = 0, 1 or 2, where 2
 * acts as 1 without a solo model;
 * RAFIKI_ERR_INVALID if none is kept); synchronises the device and drops any kept
 * graphs.  set_schedule and set_schedule_pair reset it to 0. */
int rafiki_ensemble_get_schedule_tiles(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int* lean);
int rafiki_ensemble_set_schedule_tiles(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int lean);

/* Paired layers of two different models (Section 5.1: the selected models all run the
 * same batch).  At create, every two bf16 models with different layer lists whose ops
 * align for at least half of the shorter list (a longest common subsequence under equal
 * launch shapes: ResNet-50 within ResNet-101) are pairable.  A paired schedule runs such
 * a pair on one lane, each aligned pair of ops as one launch with a member per model and
 * the other ops alone in the merged order, while the other selected models run one after
 * another on a second lane.  Each member's outputs are those of its own launch, so the
 * schedule never changes a result.  The schedule timing of infer (above) also times
 * every pairable pair of the subset (with two selected models as well).
 * get_schedule_pair: the kept choice's pair, or *pa = *pb = -1 if it is not paired;
 * RAFIKI_ERR_INVALID if no schedule has been chosen yet.
 * set_schedule_pair: pa < pb, a pairable pair of the subset, or pa = -1 (all models
 * concurrent); synchronises the device and drops any kept graphs.
 * pairing: the number of aligned ops of models a < b (0: not pairable). */
int rafiki_ensemble_get_schedule_pair(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int* pa, int* pb);
int rafiki_ensemble_set_schedule_pair(rafiki_ensemble_t h, int n, uint32_t model_subset_mask, int pa, int pb);
int rafiki_ensemble_pairing(rafiki_ensemble_t h, int a, int b, int* aligned);

/* Graph replay of the forward passes (off by default; environment RAFIKI_GRAPHS=1 turns
 * it on at create).  Measured on MI355X it is no faster than the eager launches for one
 * model and slower for several, whose branches the replay did not overlap as well as
 * the per-model streams do.  Once a batch size n has been tuned, infer / infer_vote capture the
 * forward passes of (n, model_subset_mask) into a HIP graph on first use and replay it
 * on later calls: the staging of `batch` and the combine into the caller's buffers are
 * launched around the graph on `stream`, so results are those of the eager launches bit
 * for bit.  At most 64 (n, mask) graphs are kept per handle; further pairs run eagerly.
 * Token input is first copied (device to device, on `stream`) into a buffer of the
 * handle that the graph reads.  A capture that fails disables graphs for the handle and
 * the call runs eagerly.  Tracing (rafiki_ensemble_trace) always runs eagerly.
 * use_graphs synchronises the device and drops every kept graph; enable = 0 turns
 * replay off.  force_tile also drops them.  graph_stats reports the graphs kept, the
 * replays so far and the failed captures; any output pointer may be NULL. */
int rafiki_ensemble_use_graphs(rafiki_ensemble_t h, int enable);
int rafiki_ensemble_graph_stats(rafiki_ensemble_t h, int* n_graphs, long long* replays, long long* failures);

/* Synchronise the device, free everything the handle owns.  NULL is accepted. */
int rafiki_ensemble_destroy(rafiki_ensemble_t h);

/* Message of the last failure on this thread ("" if none). */
const char* rafiki_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RAFIKI_ENSEMBLE_H */
