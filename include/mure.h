/*
 * mure.h -- memoized DNN mutation testing on one AMD Instinct MI355X (gfx950).
 *
 * The library evaluates every mutant of a feed-forward classifier over a test
 * set, running each mutant only from its earliest mutated layer (mmi) onward
 * on activations of the original model cached in device memory, and reduces
 * the outputs to a kill matrix and a mutation score.  By the paper's
 * soundness theorem (Section 4.1, Theorem 1) this equals running every mutant
 * from the raw input ("vanilla" mutation testing).
 *
 * The calls follow the problem statement of Algorithm 1 (inputs: a model M,
 * a test set X and a mapping from mutant ids to mutants; output: every
 * mutant's outputs on X) and the measures of Section 5.2 (kill predicate,
 * killingLabels, mutation score):
 *
 *   mure_create -> mure_load_model -> mure_apply_mutants -> mure_run_original
 *     -> mure_run_mutants (any number of times) -> mure_destroy
 *
 * Conventions
 *   - Every call returns a mure_status; MURE_OK is 0.  No C++ exception crosses
 *     this interface.  On failure mure_last_error() describes the cause and
 *     the context is left as it was before the call (calls are atomic).
 *   - "host" pointers are ordinary CPU memory; "device" pointers are memory
 *     of the context's GPU (e.g. from hipMalloc or a torch CUDA tensor).
 *   - Tensors are NHWC, row-major.  A DENSE layer reads its input flattened in
 *     HWC order.  Weights: CONV2D [C_out][kh][kw][C_in], DENSE [C_out][C_in].
 *   - All device work is enqueued on the context's stream.  The library
 *     synchronises that stream before returning from a call that yields host
 *     results; device outputs are complete when the call returns.
 *   - One context per host thread; contexts are independent.
 */
#ifndef MURE_H
#define MURE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MURE_VERSION 6
#define MURE_N_KERNELS 9   /* kernel families in mure_stats */
/* Device scratch of mure_run_mutants_noalloc: a fixed array per GPU. */
#define MURE_NOALLOC_SCRATCH_BYTES (256u << 20)

typedef struct mure_ctx mure_ctx;

typedef enum {
  MURE_OK = 0,
  MURE_E_INVALID = -1,     /* bad argument: shapes, indices, operator, sizes */
  MURE_E_STATE = -2,       /* call out of order (e.g. run_mutants before run_original) */
  MURE_E_NOMEM = -3,       /* device or host allocation failed, or memory limit exceeded */
  MURE_E_DEVICE = -4,      /* a HIP runtime call failed; the message holds HIP's error string */
  MURE_E_UNSUPPORTED = -5  /* valid request this build does not implement */
} mure_status;

typedef enum { MURE_F32 = 0, MURE_BF16 = 1 } mure_dtype;

/* Neuron-level mutation operators (Section 3.1).  A neuron of a DENSE or
 * CONV2D layer is one output channel (Section 2.1: a conv layer's neurons are
 * its filters); its incoming weights are W[neuron][...] (fan_in values).
 *   GAUSS_FUZZ     W[i] <- round(W[i] + noise) (float32 addition, then the
 *                  model's weight dtype, round-to-nearest-even); bias kept.
 *   EFFECT_BLOCK   W[i] <- 0 and b[i] <- 0: the neuron's output is 0.
 *   ACT_INVERSE    W[i] <- -W[i] and b[i] <- -b[i]: the pre-activation is negated.
 *   NEURON_SWITCH  W[i] <-> W[partner] and b[i] <-> b[partner].
 *   WEIGHT_SHUFFLE W[i][k] <- W[i][perm[k]] for a permutation perm of the
 *                  neuron's fan_in incoming weights; bias kept.            */
typedef enum {
  MURE_OP_GAUSS_FUZZ = 0,
  MURE_OP_EFFECT_BLOCK = 1,
  MURE_OP_ACT_INVERSE = 2,
  MURE_OP_NEURON_SWITCH = 3,
  MURE_OP_WEIGHT_SHUFFLE = 4
} mure_op;

typedef enum {
  MURE_INPUT = 0,    /* the model input (must be node 0, and only node 0) */
  MURE_DENSE = 1,    /* y = x W^T + b, optional activation */
  MURE_CONV2D = 2,   /* cross-correlation, stride, zero padding, + b, optional activation,
                        optional 2x2 stride-2 max-pool (floor) */
  MURE_ADD = 3,      /* y = in[0] + s(in[1]) in float32, optional activation; shortcut 1
                        ("option A") subsamples in[1] by 2 in H and W and zero-pads
                        its channels, (C_out - C_in)/2 before and the rest after */
  MURE_GAP = 4,      /* global average pool to 1x1xC */
  MURE_FLATTEN = 5,  /* view as 1x1x(H*W*C) */
  MURE_DWCONV = 6,   /* depthwise convolution (MobileNetV2): output channel c filters
                        input channel c with its own kh x kw taps, stride, zero
                        padding, + b, optional activation; c_in = c_out = C;
                        weights [C][kh][kw] (fan_in = kh*kw) */
  MURE_EMBED = 7,    /* token embedding: reads a 1 x T x 1 node whose values are
                        token ids (integers in [0, c_in), as float32), writes
                        1 x T x c_out with out[t][d] = W[d][token_t]; weights
                        [c_out][c_in] (fan_in = c_in, the vocabulary); no bias */
  MURE_LSTM = 8      /* LSTM over the T steps of a 1 x T x c_in node (float32
                        models), h = c = 0 at the start; per step and unit j,
                        z_q = x_t . Wx_q[j] + h . Wh_q[j] + b_q[j] for the gates
                        q = input, forget, cell, output; i, f, o = sigmoid(z),
                        g = tanh(z_g), c = f*c + i*g, h = o*tanh(c).  Output
                        1 x T x c_out (seq = 1) or the last h, 1 x 1 x c_out.
                        Weights [c_out][4][c_in + c_out + 1]: unit j's row holds
                        per gate its input weights, recurrent weights and bias
                        (fan_in = 4*(c_in + c_out + 1)); the bias array is
                        ignored (pass zeros). */
} mure_kind;

/* One node of the model graph.  The array order is a topological order
 * (Section 4: tau); in[] lists the nodes this node reads, each with a smaller
 * index -- this is the dependence graph of Algorithm 2 given explicitly.
 * The last node is the output; its values are the float32 logits.
 * Fields that do not apply to a kind must be 0. */
typedef struct {
  int32_t kind;       /* mure_kind */
  int32_t n_in;       /* 0 for INPUT, 2 for ADD, 1 otherwise */
  int32_t in[2];
  int32_t c_in;       /* CONV2D/DWCONV: input channels; DENSE: H*W*C of its input;
                         ADD: channels of in[1]; GAP/FLATTEN: input channels */
  int32_t c_out;      /* output channels (DENSE: units) */
  int32_t kh, kw, stride, pad;   /* CONV2D/DWCONV only (DENSE: 1,1,1,0) */
  int32_t relu;       /* activation after the bias (or the sum): 0 none, 1 ReLU,
                         2 ReLU6 = min(max(x, 0), 6), in float32 */
  int32_t maxpool;    /* CONV2D: 0 or 2 */
  int32_t shortcut;   /* ADD: 0 identity, 1 option A */
  int32_t seq;        /* LSTM: 1 = output every step, 0 = only the last */
} mure_layer;

/* One mutation record: operator `op` applied to neuron `neuron` of node
 * `layer` of mutant `mutant`.  A mutant's records apply in array order. */
typedef struct {
  int32_t mutant;       /* 0 <= mutant < n_mutants */
  int32_t op;           /* mure_op */
  int32_t layer;        /* a DENSE, CONV2D, DWCONV, EMBED or LSTM node */
  int32_t neuron;       /* 0 <= neuron < c_out of that node */
  int32_t partner;      /* NEURON_SWITCH: the other neuron (!= neuron); else -1 */
  int32_t reserved;     /* 0 */
  const float* noise;   /* GAUSS_FUZZ: host, fan_in values in W[neuron] order; else NULL */
  int64_t noise_len;    /* GAUSS_FUZZ: = fan_in (c_in*kh*kw for CONV2D, kh*kw for DWCONV,
                           c_in for DENSE and EMBED, 4*(c_in + c_out + 1) for LSTM);
                           WEIGHT_SHUFFLE: = fan_in (length of perm) */
  const int32_t* perm;  /* WEIGHT_SHUFFLE: host, a permutation of 0..fan_in-1; else NULL */
} mure_record;

/* Mutation score (Section 5.2): MS = ms_num / ms_den with
 * ms_num = sum over mutants of |killingLabels(mutant)| and
 * ms_den = n_mutants * n_labels. */
typedef struct {
  int64_t ms_num, ms_den;
  double ms;
  int64_t killed_mutants;     /* mutants killed by at least one input */
  int64_t n_mutants, n_labels, n_inputs;
  int64_t nonfinite_logits;   /* logits that were NaN or infinite (expected 0) */
} mure_score;

/* Work and timing of the last run_original / run_mutants (for measurement).
 * MAC counts are per whole call (all inputs). */
typedef struct {
  int64_t n_groups;              /* distinct first-mutated layers (clusters) */
  int64_t n_identity_mutants;    /* mutants without records */
  int64_t macs_original;         /* one forward of the original over X */
  int64_t macs_vanilla;          /* every mutant from the raw input */
  int64_t macs_memoized;         /* Lemma 4 accounting: cost(P) once per cluster +
                                    every mutant from its mmi on (Algorithm 4) */
  int64_t macs_algorithmic;      /* touched channels at mmi (fuzz/inverse) +
                                    every layer after mmi, summed over mutants */
  int64_t macs_executed;         /* what run_mutants' kernels actually computed */
  int64_t cache_bytes;           /* prefix cache (memo table) size */
  int64_t workspace_bytes;       /* per-chunk activation buffers */
  int64_t launches;              /* kernel launches in the last run_mutants */
  double ms_apply, ms_run_original, ms_run_mutants;   /* device time, milliseconds */
  /* With option "kernel_timing" = 1: the CONV2D/DENSE (implicit-GEMM)
   * launches of the last run_mutants, timed one by one with HIP events on the
   * context's stream; MACs are algorithmic (as macs_algorithmic) and executed. */
  int64_t gemm_launches;
  double ms_gemm;
  int64_t gemm_macs_algorithmic, gemm_macs_executed;
  /* The same, split by kernel (MURE_N_KERNELS entries): [0] dense GEMM,
   * [1] vector-ALU convolution (few output channels), [2] LDS-resident
   * convolution, [3] im2col implicit GEMM with scalar gathers, [4] tiled bf16
   * implicit GEMM, [5] depthwise convolution, [6] embedding lookup, [7] LSTM
   * recursion, [8] bf16 3x3 convolution over LDS halo tiles. */
  int64_t kernel_launches[MURE_N_KERNELS];
  double kernel_ms[MURE_N_KERNELS];
  int64_t kernel_macs_algorithmic[MURE_N_KERNELS];
  /* Algorithmic HBM bytes of those launches: every input row read once (a
   * prefix-cache tensor once for all mutants), every output element written
   * once, every mutant's weights read once. */
  double kernel_bytes_algorithmic[MURE_N_KERNELS];
  /* Shapes the caller's buffers must match: classes of the loaded model,
   * inputs of the last run_original (0 before), registered mutants.
   * get_logits writes n_inputs * n_classes floats; run_mutants writes
   * n_mutants * ceil(n_inputs / 64) kill words. */
  int64_t n_classes, n_inputs, n_mutants;
  /* Side planes (one mutant's changed 8-channel group of the first mutated
   * node's output, over a chunk's inputs) built by the last run_mutants for
   * halo convolutions that read that output in channel groups (option
   * "group_reads"); 0 when every consumer read per-mutant copies. */
  int64_t group_planes;
  /* With option "kernel_timing" = 1: the part of ms_gemm spent computing the
   * clusters' first mutated nodes (the deltas of Section 3's memoized
   * execution), the rest being the suffix after them. */
  double ms_mmi;
} mure_stats;

/* Version of this interface (MURE_VERSION). */
int32_t mure_version(void);

/* Create a context on HIP device `device`, enqueueing on `hip_stream` (a
 * hipStream_t; NULL = the device's null stream).  device = -1 creates a
 * planning-only context: load_model and apply_mutants validate and plan, but
 * nothing touches a GPU and run_original/run_mutants/get_logits return
 * MURE_E_UNSUPPORTED.  *out receives the context, owned by the caller until
 * mure_destroy. */
mure_status mure_create(mure_ctx** out, int32_t device, void* hip_stream);

/* Load the model (Section 4: the DAG (V, E, Phi, I, O)): n_layers
 * descriptors in topological order, input shape in_hwc = {H, W, C}, weight
 * dtype, and per node a host pointer to its weights (`weights[i]`, in dtype:
 * float32 or bfloat16 bit patterns as uint16) and float32 bias (`biases[i]`);
 * NULL for nodes without parameters.  The library copies everything (to
 * device memory); the caller keeps ownership of its arrays.  Resets any
 * mutants and cache.  Errors: MURE_E_INVALID for inconsistent shapes, a
 * non-topological order, or a missing/unused parameter array. */
mure_status mure_load_model(mure_ctx* ctx, const mure_layer* layers, int32_t n_layers,
                            const int32_t in_hwc[3], int32_t dtype,
                            const void* const* weights, const float* const* biases);

/* Register n_mutants mutants given by n_records records (host array).  For
 * each mutant the library derives its mutated layers mu(M'), its earliest
 * mutated layer mmi = min mu(M') and its memoization boundary
 * K = { p < mmi : some node >= mmi reads p } (Algorithm 1; Section 4), groups
 * mutants by mmi (the clusters of Algorithm 1), and materialises each mutated
 * layer of each mutant as a copy-on-write copy of the original parameters
 * with the records applied.  A mutant without records is an identity mutant:
 * never killed.  Noise arrays are copied.  Replaces earlier mutants and
 * invalidates the prefix cache (run_original must run again).
 * Errors: MURE_E_INVALID (mutant/layer/neuron/partner out of range, a layer
 * without neurons, unknown op, noise length != fan_in); nothing is applied. */
mure_status mure_apply_mutants(mure_ctx* ctx, int32_t n_mutants,
                               const mure_record* records, int64_t n_records);

/* Run the original model once over the inputs (device, [n][H][W][C] in the
 * model dtype) and fill the prefix cache: the activations of every node in
 * the union of the mutants' boundaries K (the memo table of Algorithm 1 and
 * Algorithm 3's probe points), of each cluster's first mutated layer, and the
 * original's float32 logits.  Derives label(x): `labels` (host, n values in
 * [0, classes)) or, if NULL, the original's prediction (argmax, lowest index
 * on ties), and the label set L.  `inputs_dev` is only read during the call.
 * Errors: MURE_E_STATE before load_model/apply_mutants; MURE_E_INVALID for
 * n < 1 or a label out of range. */
mure_status mure_run_original(mure_ctx* ctx, const void* inputs_dev, int64_t n_inputs,
                              const int32_t* labels);

/* Run every mutant's suffix over every input and classify each (mutant,
 * input) pair: kill(mutant, x) holds when argmax of the original's logits at
 * x equals label(x) and argmax of the mutant's logits differs from label(x)
 * (Section 5.2).  Outputs (each may be NULL):
 *   kill_bits_dev     device uint64 [n_mutants][ceil(n/64)]; the bit for
 *                     (m, x) is bit (x & 63) of word m*ceil(n/64) + (x >> 6);
 *                     padding bits are 0;
 *   kills_host        host int64 [n_mutants]: inputs killing each mutant;
 *   score             host: the mutation score and counts.
 * Deterministic: repeated calls give identical bits.
 * Errors: MURE_E_STATE unless run_original ran after the last apply_mutants. */
mure_status mure_run_mutants(mure_ctx* ctx, uint64_t* kill_bits_dev, int64_t* kills_host,
                             mure_score* score);

/* mure_run_mutants for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same kernels, outputs and errors, but the call allocates
 * nothing.  Its chunk activation workspace and the per-mutant kill counts and
 * label masks live in one file-scope device array of
 * MURE_NOALLOC_SCRATCH_BYTES per GPU, set up by mure_create and held until
 * the process ends; chunks of inputs and mutants are sized to fit it.
 * Differences from mure_run_mutants:
 *   - kill_bits_dev is required (the caller's output buffer);
 *   - per-launch timing (option "kernel_timing") is skipped;
 *   - every call on one GPU shares that GPU's array, so calls that overlap
 *     on one GPU (contexts on different host threads or streams) race:
 *     serialise them.
 * Errors: as mure_run_mutants; MURE_E_INVALID for kill_bits_dev == NULL;
 * MURE_E_NOMEM, before any device work, when the smallest chunk of some
 * cluster (one mutant x min(64, n) inputs) or the counters need more than
 * MURE_NOALLOC_SCRATCH_BYTES. */
mure_status mure_run_mutants_noalloc(mure_ctx* ctx, uint64_t* kill_bits_dev, int64_t* kills_host,
                                     mure_score* score);

/* Logits of one mutant (or of the original for mutant_id = -1) over all
 * inputs: device float32 [n][classes].  Runs that mutant's suffix alone with
 * the same kernels as run_mutants (for checking; not the fast path).
 * Errors: MURE_E_STATE before run_original; MURE_E_INVALID for a bad id. */
mure_status mure_get_logits(mure_ctx* ctx, int32_t mutant_id, float* out_dev);

/* Plan of one mutant (host outputs, any may be NULL): its mmi (-1 for an
 * identity mutant), its group index, and its boundary K (up to max_k node
 * indices, ascending; *n_k receives |K|).  Works on planning-only contexts. */
mure_status mure_mutant_plan(const mure_ctx* ctx, int32_t mutant_id, int32_t* mmi,
                             int32_t* group, int32_t* k_nodes, int32_t max_k, int32_t* n_k);

/* Work/timing counters of the most recent calls (host output). */
mure_status mure_get_stats(const mure_ctx* ctx, mure_stats* out);

/* Tuning and testing knobs (name, integer value).  Known names:
 *   "max_workspace_mb"  cap on per-chunk activation buffers (default 65536)
 *   "max_device_mb"     cap on the device memory of the model, the mutants'
 *                       copy-on-write layers and the prefix cache (0 = none,
 *                       the default): apply_mutants and run_original refuse a
 *                       plan above it with MURE_E_NOMEM and change nothing
 *   "chunk_inputs"      inputs per chunk, multiple of 64 (0 = automatic)
 *   "fused_paths"       1 (default) fuse a residual block's ADD into its second
 *                       convolution and the kill into the output layer where
 *                       the graph allows; 0 run them as kernels of their own
 *                       (the same results, bit for bit)
 *   "vanilla"           1: no memoization -- every mutant runs from the first
 *                       layer after the input (exhaustive mutation testing, the
 *                       baseline the paper compares against); takes effect at
 *                       the next apply_mutants.  0 (default) memoized
 *   "conv_tile"         block shape of the tiled bf16 convolution: 0 automatic,
 *                       1 = 128 output pixels per block, 2 = 256
 *   "group_reads"       1 (default): where every consumer of a cluster's first
 *                       mutated node is a bf16 halo convolution (or an
 *                       identity-shortcut ADD fused into one), the consumers
 *                       read that output in 8-channel groups: the cached
 *                       groups for all mutants, only each mutant's changed
 *                       groups copied.  0: a full copy per mutant (the same
 *                       results, bit for bit).  Not used by
 *                       mure_run_mutants_noalloc.
 *   "kernel_timing"     1: time each implicit-GEMM launch of run_mutants (see
 *                       mure_stats); 0 (default) off
 * Errors: MURE_E_INVALID for an unknown name or value. */
mure_status mure_set_option(mure_ctx* ctx, const char* name, int64_t value);

/* Message describing the last failure on ctx (or of mure_create when ctx is
 * NULL: a thread-local message).  Never NULL; valid until the next call. */
const char* mure_last_error(const mure_ctx* ctx);

/* Release the context and everything it owns.  NULL is ignored. */
void mure_destroy(mure_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* MURE_H */
