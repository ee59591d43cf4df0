/*
 * gevo.h -- C-ABI of libgevo: population-batched fitness evaluation on one
 * AMD Instinct MI355X (gfx950).
 *
 * The method is GEVO-ML (Liou, Forrest, Wu; arXiv 2310.10211).  Its run time is
 * dominated by fitness evaluation (section 4.3): every individual of the
 * evolving population is either retrained on the dataset, recording training
 * time and model error (training workload), or run over the dataset as a
 * pretrained model, recording inference time and error (prediction workload).
 * The two objectives are time and error (section 4.3).  The paper's training
 * model is a two-layer fully-connected net trained by mini-batch SGD whose
 * output gradient is prediction minus label, reduced over the batch, scaled by
 * 1/batch, multiplied by the learning rate and subtracted from weights and
 * biases (section 6.2).  Its discovered mutations act like a changed learning
 * rate (section 6.2) and like pruned parameters (abstract, section 2), so an
 * individual here is the original model with its own learning rate and its own
 * Bernoulli weight-pruning mask.
 *
 * Conventions for every entry point
 *  - Device memory belongs to the caller: datasets, the workspace and the HIP
 *    stream are passed in; the library never allocates or frees device memory.
 *    Host arrays passed in or out belong to the caller.
 *  - Arguments are validated on the host before any HIP call; a bad argument
 *    returns an error code and launches nothing.
 *  - Work is enqueued asynchronously on the handle's stream.  Device faults are
 *    sticky and are reported by the next synchronising call (gevo_pop_scores,
 *    gevo_pop_export) as GEVO_E_HIP.
 *  - A handle is not thread-safe; distinct handles are independent.
 *
 * Numerics
 *  - Weights of layer l are d_{l-1} x d_l ("in x out") in every host-visible
 *    (canonical) array; the device layout is private.
 *  - GEVO_F32: fp32 operands, fp32 accumulation.  GEVO_BF16: bf16 GEMM operands
 *    (input rows, weights rounded from the fp32 master each step, hidden
 *    activations after ReLU, gradients), fp32 accumulation, fp32 master
 *    weights, fp32 logits/softmax/loss/bias gradients/update.  Rounding to bf16
 *    is round-to-nearest-even.
 *  - Random draws use Philox4x32-10 (Salmon et al., SC'11) with key = (seed low
 *    32 bits, seed high 32 bits) and counter (c0, c1, c2, c3) = (block, layer
 *    index l-1, variant or epoch, stream); stream 1 learning rate, 2 density,
 *    3 mask, 4 initial weights, 5 weight noise, 6 data order.  A uniform u24 is
 *    the top 24 bits of a word.  Weight (k -> n) of layer l has element index
 *    e = n * d_{l-1} + k.  Learning rate: exp(ln lo + u (ln hi - ln lo)) in
 *    fp64, rounded to fp32 (block 0, word 0).  Density: list[v mod n] or
 *    lo + u (hi - lo).  Mask: keep <=> u24 < round_half_away(rho 2^24) (block
 *    e/4, word e%4).  Xavier init, shared by all variants (the original model):
 *    (2u - 1) * fl32(sqrt(6 / (d_{l-1} + d_l))) (block e/4, word e%4, variant
 *    field 0).  Weight noise: eps = sqrt(-2 ln u1) cos(2 pi u2) with
 *    u1 = (u24 + 1) 2^-24 and u2 = u24 2^-24 from words 2(e%2), 2(e%2)+1 of block
 *    e/2.  Data order of epoch e: Fisher-Yates from the last index down, swap
 *    index j = (r * (i + 1)) >> 32 with r word i%4 of block i/4 (variant field =
 *    epoch, layer field 0); one order shared by all variants.
 *  - Masked weights are exactly +0.0 and stay so (the update is a select).
 */
#ifndef GEVO_H
#define GEVO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GEVO_ABI_VERSION 1u
#define GEVO_MAX_LAYERS 3u      /* supported depth of the net (hidden layers + output) */
#define GEVO_MAX_CLASSES 32u    /* d_L */
#define GEVO_MAX_BATCH 256u
#define GEVO_MAX_WIDTH 8192u    /* any d_l */

typedef enum {
  GEVO_OK = 0,
  GEVO_E_ARG = -1,          /* NULL pointer, zero size, bad enum */
  GEVO_E_SHAPE = -2,        /* inconsistent dimensions / sizes */
  GEVO_E_WORKSPACE = -3,    /* workspace too small or misaligned (256 B) */
  GEVO_E_ORDER = -4,        /* call out of sequence (epoch order, predict before init) */
  GEVO_E_HIP = -5,          /* a HIP runtime call failed (sticky device error) */
  GEVO_E_UNSUPPORTED = -6   /* valid but beyond this build's limits */
} gevo_status;

typedef enum { GEVO_F32 = 0, GEVO_BF16 = 1 } gevo_dtype;
typedef enum { GEVO_INIT_XAVIER = 0, GEVO_INIT_BASE_NOISE = 1 } gevo_init;

/*
 * Population description.  n_layers = L (1..GEVO_MAX_LAYERS); dims[0..L] are
 * the layer widths d_0 (input) .. d_L (classes).  Learning rates are
 * log-uniform in [lr_lo, lr_hi) (lr_lo == lr_hi: fixed).  Densities come from
 * dens_list (host array, cycled by variant index) if n_dens_list > 0, else
 * uniform in [dens_lo, dens_hi].  init = GEVO_INIT_BASE_NOISE multiplies each
 * weight of the base model by (1 + noise_rel_std * eps); the base model is
 * base_params (host array, canonical layout: per layer W_l in x out then b_l)
 * or, if NULL, the seeded Xavier model.  n_train may be 0 (prediction only).
 */
typedef struct {
  uint32_t abi_version;               /* must be GEVO_ABI_VERSION */
  uint32_t n_layers;
  uint32_t dims[GEVO_MAX_LAYERS + 1];
  uint32_t P;                         /* variants, >= 1 */
  uint32_t batch;                     /* B, 1..GEVO_MAX_BATCH */
  gevo_dtype dtype;
  uint64_t seed;
  float lr_lo, lr_hi;
  float dens_lo, dens_hi;
  const float* dens_list;
  uint32_t n_dens_list;
  gevo_init init;
  const float* base_params;
  float noise_rel_std;
  int64_t n_train;                    /* rows of the training split (0 allowed) */
  int64_t n_test;                     /* rows of the test split (>= 1) */
} gevo_pop_config;

typedef struct gevo_pop gevo_pop;     /* opaque handle */

/* Bytes of device workspace gevo_pop_init needs for cfg (always a multiple of 256). */
gevo_status gevo_pop_workspace_bytes(const gevo_pop_config* cfg, size_t* bytes);

/*
 * Create a population (section 4: copies of the original model carrying random
 * edits; here a per-variant learning rate and pruning mask).  d_ws: device
 * workspace of at least gevo_pop_workspace_bytes bytes, 256-byte aligned, owned
 * by the caller and untouched by it while the handle lives.  Datasets: device
 * arrays, row-major float32 [n][d_0] features and int32 labels in
 * [0, d_L); they must outlive the handle (train pointers may be NULL when
 * n_train == 0).  hip_stream: a hipStream_t (NULL = default stream).
 * Enqueues mask generation, weight init and dataset conversion.
 */
gevo_status gevo_pop_init(const gevo_pop_config* cfg, void* d_ws, size_t ws_bytes,
                          const float* d_train_x, const int32_t* d_train_y,
                          const float* d_test_x, const int32_t* d_test_y,
                          void* hip_stream, gevo_pop** out);

/*
 * Training workload of section 4.3 / mini-batch SGD of section 6.2: one epoch
 * over the training split in the epoch's data order, batches of B rows (the
 * short last batch is kept and scaled by fl32(1/b)).  Epochs must be called as
 * 0, 1, 2, ... (GEVO_E_ORDER otherwise).  Per variant the epoch's mean
 * cross-entropy (taken before each step's update) and the wall time of the
 * call (HIP events) are recorded for gevo_pop_scores.
 * With GEVO_RESIDENT=1 in the environment when gevo_pop_init runs, two-layer
 * bf16 nets of 784 (or 769..800) inputs, 256 hidden units, at most 16 classes
 * and a batch of 97..128 rows train in the resident kernel (a pair of
 * workgroups per variant, cooperative launch; slower than the default on
 * gfx950).  That path synchronises the stream at the end of the call and
 * returns GEVO_E_HIP if a workgroup gave up waiting for its partner.
 */
gevo_status gevo_pop_train_epoch(gevo_pop* pop, uint32_t epoch);

/*
 * Steps [step_begin, step_end) of epoch `epoch`; a sequence of such calls
 * covering 0..T-1 in order is bit-identical to gevo_pop_train_epoch.  The
 * first call of an epoch must start at step 0, later calls where the previous
 * one ended.
 */
gevo_status gevo_pop_train_steps(gevo_pop* pop, uint32_t epoch, uint32_t step_begin, uint32_t step_end);

/* Number of SGD steps per epoch, ceil(n_train / B). */
gevo_status gevo_pop_steps_per_epoch(const gevo_pop* pop, uint32_t* steps);

/*
 * Prediction workload of section 4.3 (and the held-out check of the fittest
 * individual): forward pass of every variant over the test split; records
 * the mean cross-entropy and the accuracy (argmax, lowest index on ties, a
 * NaN logit counts as a miss) per variant, and the call's wall time.
 */
gevo_status gevo_pop_predict(gevo_pop* pop);

/*
 * For callers that cannot allocate device memory or create objects during
 * the call (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): gevo_pop_predict, computing the same scores bit
 * for bit, whose scratch (per-chunk activations, bf16 weight copies, partial
 * sums) is a static device array of GEVO_NOALLOC_SCRATCH_BYTES instead of
 * part of the workspace.  Every GPU the library runs on holds one such array
 * from the first gevo_pop_init on it until the process ends.  Variants are
 * processed in groups that fit the array; the call allocates nothing and
 * creates no event (kernel-level profiling is not recorded for it).  All
 * calls on one GPU share its array: calls that overlap on one GPU (other
 * streams, other threads) race and must not be made.  GEVO_E_UNSUPPORTED
 * when the scratch of a single variant exceeds the array (e.g. hidden layers
 * of 8192 x 8192 bf16 weights); GEVO_E_HIP for a runtime error.
 */
#define GEVO_NOALLOC_SCRATCH_BYTES (64ull << 20)
gevo_status gevo_pop_predict_noalloc(gevo_pop* pop);

/*
 * Fitness of every variant (section 4.3: error and time).  Synchronises the
 * stream.  Host arrays of P entries, any may be NULL: mean training CE of the
 * last trained epoch (NaN if never trained), training accuracy of that epoch,
 * mean test CE and test accuracy in [0,1] of the last predict (NaN before),
 * and time_s = variant v's share of the wall time of the last
 * train/predict call: the call's time times v's share of the device time of
 * its workgroups (each kernel's workgroups belong to one variant and add their
 * clock-counter time to that variant's total), so the time_s sum to the
 * call's time.  Workgroups of unit tiles that GEVO_EDIT_WIDTH removes whole
 * are skipped in training, so narrowed variants get a smaller share.  The
 * small kernels that serve every variant at once (batch gathers, reductions)
 * count toward no variant, so their time is split in the same shares.
 */
gevo_status gevo_pop_scores(gevo_pop* pop, float* train_loss, float* train_acc, float* test_loss,
                            float* test_acc, float* time_s);

/* Wall time in seconds of the last train_epoch / train_steps / predict call. */
gevo_status gevo_pop_last_time(gevo_pop* pop, double* seconds);

/*
 * Variant v's state in canonical layout (synchronises the stream):
 * params_out (host float, per layer W_l in x out then b_l; may be NULL),
 * mask_out (host uint8 0/1 per weight, same order as the weights; may be NULL),
 * lr_out, density_out (may be NULL).
 */
gevo_status gevo_pop_export(gevo_pop* pop, uint32_t v, float* params_out, uint8_t* mask_out,
                            float* lr_out, float* density_out);

/* Overwrite variant v's parameters from a host array in canonical layout
 * (masked weights are forced to +0).  Synchronous. */
gevo_status gevo_pop_import(gevo_pop* pop, uint32_t v, const float* params);

/* Labels of the current epoch in the order the steps consume them (n_train
 * entries; synchronises).  Exposes the data order for exactness checks. */
gevo_status gevo_pop_epoch_labels(gevo_pop* pop, int32_t* labels_out, int64_t n);

/* Host-side data order of epoch `epoch` over n rows (definition above). */
gevo_status gevo_epoch_permutation(uint64_t seed, uint32_t epoch, uint32_t n, uint32_t* out);

/*
 * Search step (paper section 4).  GEVO-ML evolves individuals that are lists
 * of edits to the original program (patch representation, section 4.2):
 * each initial individual gets three random mutations (section 4), crossover
 * is one-point messy crossover (section 4.2), and selection keeps the best 16
 * unchanged and fills the rest by tournament selection among NSGA-II ranked
 * individuals (section 4.4).  Here an edit is one of the two effects the
 * paper attributes to its evolved edits: a changed learning rate (section 6.2)
 * or pruned weights (abstract).
 *
 * Every random choice is a Philox4x32-10 draw (key = seed as above), word w of
 * Philox((c0, c1, c2, stream)):
 *   tournament j of generation g:       (j, g, 0, 7), words 0 and 1 pick the two
 *                                       contestants (multiply-shift onto [0, n))
 *   crossover of children 2i, 2i+1:     (0, g, 2i, 8) word 0 decides (u24 < cxpb),
 *                                       word 1 the cut; (1 + t/4, g, 2i, 8) word
 *                                       t%4 the Fisher-Yates draw for position t
 *   mutation of child i, generation g:  (0, g, i, 9) word 0 decides (u24 < mutpb);
 *                                       the edit from words 1 and 2 of (1, g, i, 9)
 *   edit j of initial individual i:     words 1 and 2 of (j, 0, i, 9)
 * where u24 = (word >> 8) * 2^-24.  A drawn edit is structural when word 1's
 * u24 < struct_p: bias removal of layer 1 + (word 0 onto [0, L)) when word 3's
 * u24 < 1/2 or the net has no hidden layer, otherwise width 1 + (word 2 onto
 * [0, d_l)) of hidden layer l = 1 + (word 0 onto [0, L-1)).  Otherwise it is a
 * learning-rate factor exp(ln(1/2) + u ln 4) (u from word 2, binary64, rounded
 * to binary32) when word 1's u24 < struct_p + (1 - struct_p)/2, else pruning
 * at density rho = rho_lo + u (1 - rho_lo), threshold round-half-even(rho 2^24).
 * struct_p = 0 draws no structural edit (dims may then be null).
 */
typedef enum {
  GEVO_EDIT_LR = 0,        /* value = bits of a binary32 learning-rate factor */
  GEVO_EDIT_PRUNE = 1,     /* id = mask draw id, value = keep threshold (<= 2^24) */
  GEVO_EDIT_WIDTH = 2,     /* id = hidden layer l (1 .. L-1), value = units kept (>= 1) */
  GEVO_EDIT_BIAS_OFF = 3,  /* id = layer l (1 .. L): its biases are removed */
  GEVO_EDIT_LAYER_OFF = 4  /* id = hidden layer l (1 .. L-1): the layer is removed */
} gevo_edit_kind;
typedef struct {
  uint32_t kind;    /* gevo_edit_kind */
  uint32_t id;
  uint32_t value;
} gevo_edit;

/* NSGA-II ranking (Deb et al., IEEE TEC 2002) of n points with m objectives,
 * all minimised, objs row-major [n][m], no NaN.  rank[i] = front index (0 =
 * non-dominated; a dominates b when no objective is larger and one is
 * smaller); crowding[i] = sum over objectives k of (f_k of the next point -
 * f_k of the previous point) / (max - min of f_k) over i's front, neighbours
 * ordered by f_k then by index, the first and last point of every objective
 * getting +infinity, terms added in objective order in binary64.  Host
 * arrays; GEVO_E_ARG for a null pointer, m == 0 or a NaN objective. */
gevo_status gevo_nsga2_rank(uint32_t n, uint32_t m, const double* objs, uint32_t* rank, double* crowding);

/* Selection of generation gen (section 4.4): out[0 .. n_elite) are the
 * n_elite best points by the crowded comparison (lower rank, then larger
 * crowding, then lower index), best first; out[n_elite .. n_select) are
 * binary-tournament winners under the same comparison (draws above).  Host
 * arrays; GEVO_E_ARG unless n_elite <= n_select, n_elite <= n and n > 0 (when
 * n_select > 0). */
gevo_status gevo_nsga2_select(uint32_t n, const uint32_t* rank, const double* crowding, uint32_t n_elite,
                              uint32_t n_select, uint64_t seed, uint32_t gen, uint32_t* out);

/* Initial population (section 4): individual i gets n_mut drawn edits, edit j
 * with id id_base + n_mut i + j, written to out[n_mut i + j] (host array of
 * n * n_mut edits).  dims[n_layers + 1]: the net's widths (for structural
 * edits).  GEVO_E_ARG for a null pointer, rho_lo or struct_p outside [0, 1]. */
gevo_status gevo_genomes_initial(uint32_t n, uint32_t n_mut, uint64_t seed, double rho_lo, uint32_t id_base,
                                 double struct_p, uint32_t n_layers, const uint32_t* dims, gevo_edit* out);

/* Children of generation gen >= 1 from n parents (the tournament winners);
 * parent i's edits are edits[offsets[i] .. offsets[i+1]).  Pairs (2i, 2i+1)
 * are recombined with probability cxpb by one-point messy crossover:
 * concatenate both lists, shuffle (Fisher-Yates from the last position), cut
 * at a drawn point in [0, length], each child keeping at most max_edits; an
 * odd last parent is copied.  Then child i gets one drawn edit with id
 * id_base + i, with probability mutpb, when it holds fewer than max_edits
 * (structural with probability struct_p, see above).  Writes
 * out_offsets[n + 1] and the edits (host arrays); GEVO_E_ARG for bad offsets,
 * gen == 0, probabilities outside [0, 1] or out_capacity below offsets[n] + n. */
gevo_status gevo_genomes_breed(uint32_t n, const uint32_t* offsets, const gevo_edit* edits, uint64_t seed,
                               uint32_t gen, double cxpb, double mutpb, double rho_lo, uint32_t id_base,
                               uint32_t max_edits, double struct_p, uint32_t n_layers, const uint32_t* dims,
                               uint32_t* out_offsets, gevo_edit* out_edits, size_t out_capacity);

/* Rebuild the population from genomes, variant v from edits[offsets[v] ..
 * offsets[v+1]) (host arrays, offsets[P] entries after the first).  Learning
 * rate: lr_base times the GEVO_EDIT_LR factors in order, each product rounded
 * to binary32.  Mask: a weight is kept when every GEVO_EDIT_PRUNE edit keeps
 * it, edit (id, threshold) keeping weight (layer l, index e = n d_{l-1} + k)
 * when the top 24 bits of the mask draw of initialisation, taken with id in
 * place of the variant index, are below the threshold (one edit (v, T_v)
 * reproduces variant v of gevo_pop_init).  Structural edits (removing the
 * bias term, section 6.1; shrinking a tensor, the repair of section 4.1):
 * GEVO_EDIT_WIDTH keeps the first `value` units of hidden layer `id` (several
 * on one layer: the smallest), removing every weight into and out of the
 * other units and their biases; GEVO_EDIT_BIAS_OFF removes the biases of
 * layer `id`.  Removed biases are +0 and stay +0 in training; a variant whose
 * units are removed computes exactly what the narrower network computes.
 * GEVO_EDIT_LAYER_OFF removes hidden layer `id` (section 6.1 removes a layer;
 * section 4.1 repairs the shapes): the layer takes its identity form, unit n
 * passing kept input n on (weight 1 at k == n < min(kept inputs, kept
 * units)), units beyond the kept inputs holding the value 1 (no weights,
 * bias 1), every other weight and bias +0, the mask marking the ones; its
 * pruning edits and bias removal do not apply, and it trains with learning
 * rate 0 (so it stays the identity while its gradients are finite).  On
 * non-negative inputs (ReLU outputs, or non-negative data for layer 1) the
 * layer passes its input on exactly.
 * Weights are the initial weights of gevo_pop_init under the new mask,
 * biases as initialised; the next training epoch is epoch 0 again.  Writes
 * lr_out[P] and density_out[P] when not null: the product of the pruning
 * edits' keep fractions threshold / 2^24 in order, times the fraction of
 * weights the structural edits keep (sum over layers that are not removed of
 * kept inputs times kept units over sum of d_{l-1} d_l), in binary64.  At most 64 pruning edits
 * per variant.  Synchronous; GEVO_E_ARG for bad offsets, kinds, layers,
 * widths of 0, thresholds above 2^24, a non-finite or non-positive learning
 * rate or too many pruning edits, GEVO_E_ORDER during an epoch. */
gevo_status gevo_pop_set_genomes(gevo_pop* pop, float lr_base, const uint32_t* offsets, const gevo_edit* edits,
                                 float* lr_out, double* density_out);

/* Per-element output-gradient scale (section 6.2: the mutation that improved
 * 2fcNet replaced the scalar 1/32 multiplying the output gradient by a tensor
 * of the gradient's shape, mostly ones).  scale is a host array [P][batch][C]
 * (C = classes): from the next training step on, row i of every batch of
 * variant v has G_L[i][c] = (p - onehot(y))[i][c] * scale[v][i][c] in
 * binary32, in place of (p - onehot(y)) * fl(1/b_t); rows past a short last
 * batch are not used.  scale == NULL restores the scalar.  Synchronous;
 * GEVO_E_ARG for a non-finite entry, GEVO_E_ORDER during an epoch. */
gevo_status gevo_pop_set_grad_scale(gevo_pop* pop, const float* scale);

/* Self-check of the binary32 -> bfloat16 rounding that the bf16 kernels use
 * for every operand they round (weights from the master, activations,
 * gradients; round-to-nearest-even, see Numerics).  The kernels convert with
 * gfx950's packed conversion instruction.  This call converts every binary32
 * encoding twice, paired two ways as the instruction's two operands, compares
 * each result with a bit-level round-to-nearest-even (NaN -> quiet NaN) and
 * writes the number of differing results per pairing to the caller's device
 * array d_counts[2] (8-byte aligned): both are 0 when the kernels round
 * exactly.  Zeroes d_counts first; runs on `hip_stream` and synchronises it.
 * GEVO_E_ARG for a null or misaligned pointer, GEVO_E_HIP for a runtime
 * error. */
gevo_status gevo_check_bf16_rounding(void* hip_stream, uint64_t* d_counts);

/*
 * Kernel-level timing for evidence (fitness time of section 4.3 broken down
 * by kernel).  With profiling enabled, every kernel enqueued by this handle
 * carries a HIP event pair recorded by its own dispatch on the handle's
 * stream; gevo_pop_kernel_stats synchronises and returns, per kind, the summed
 * kernel time in ms and the launch count since the handle was created.
 */
typedef enum {
  GEVO_KERNEL_INIT = 0,          /* population init (masks, weights) */
  GEVO_KERNEL_GATHER = 1,        /* per-epoch gather of the data order, transpose */
  GEVO_KERNEL_LAYER_TRAIN = 2,   /* hidden layer: weight gradient, masked SGD, next forward */
  GEVO_KERNEL_LAYER_FWD = 3,     /* hidden layer forward only (epoch start, prediction) */
  GEVO_KERNEL_OUT_TRAIN = 4,     /* output layer: loss, gradients, update */
  GEVO_KERNEL_OUT_PREDICT = 5,   /* output layer: loss and accuracy on the test split */
  GEVO_KERNEL_BWD = 6,           /* hidden backward GEMM */
  GEVO_KERNEL_AUX = 7,           /* zeroing, reductions */
  GEVO_KERNEL_FUSED_TRAIN = 8,   /* two-layer nets: whole SGD steps, one workgroup per variant */
  GEVO_KERNEL_WEIGHT_COPY = 9,   /* bf16 weight copies read by the prediction GEMM */
  GEVO_KERNEL_FWD_OUT = 10,      /* prediction: last hidden layer GEMM with the output layer fused */
  GEVO_KERNEL_KINDS = 11
} gevo_kernel_kind;

gevo_status gevo_pop_set_profiling(gevo_pop* pop, int enable);
gevo_status gevo_pop_kernel_stats(gevo_pop* pop, int kind, double* total_ms, uint64_t* launches);

/* Release the handle (does not free the caller's device memory). */
void gevo_pop_destroy(gevo_pop* pop);

const char* gevo_status_str(gevo_status s);

/* ------------------------------------------------------------------------
 * Convolutional prediction workload (section 4.3: the prediction workload
 * runs a model over a dataset and records its error; Table 1 lists
 * MobileNet, a depthwise-separable convolutional net).  P variants of a
 * CIFAR-shaped, MobileNet-like net are evaluated over a test set:
 *   stem   3x3 convolution (stride 1, zero padding 1) C -> stem_channels,
 *          bias, ReLU
 *   block  3x3 depthwise convolution (stride 1 or 2, zero padding 1), bias,
 *          ReLU; then 1x1 pointwise convolution -> block_channels[i], bias,
 *          ReLU
 *   head   global average pooling, fully connected -> classes, softmax
 *          cross-entropy and argmax (lowest index on ties)
 * Variant v is the caller's base model with every weight multiplied by
 * fl(1 + fl(noise_rel_std * eps)) (eps standard normal, Box-Muller) and kept
 * with probability rho_v ~ U[dens_lo, dens_hi] (a pruning edit, section
 * 4.2); biases are the base's.  bf16 operands and activations, fp32
 * accumulation and master weights.
 *
 * Canonical parameter layout (base_params, gevo_cnn_export): the tensors in
 * order stem, (depthwise i, pointwise i) for each block, head; each as a
 * K x N row-major matrix followed by its N biases:
 *   stem        K = 9 C, row (3 dy + dx) C + c, N = stem_channels
 *   depthwise   K = 9, row 3 dy + dx, N = the block's input channels
 *   pointwise   K = input channels, N = block_channels[i]
 *   head        K = last block_channels, N = classes
 * Images are fp32 [n][height][width][channels] (NHWC), labels int32 in
 * [0, classes).
 * ------------------------------------------------------------------------ */
#define GEVO_CNN_MAX_BLOCKS 4u

typedef struct {
  uint32_t abi_version;               /* must be GEVO_ABI_VERSION */
  uint32_t P;                         /* variants, 1..65535 */
  uint32_t height, width, channels;   /* input images; channels 1..4, (height + 2) (width + 2) channels
                                         <= 28672 */
  uint32_t stem_channels;             /* multiple of 32, <= 512 */
  uint32_t n_blocks;                  /* 1..GEVO_CNN_MAX_BLOCKS */
  uint32_t block_stride[GEVO_CNN_MAX_BLOCKS];    /* 1 or 2 */
  uint32_t block_channels[GEVO_CNN_MAX_BLOCKS];  /* multiples of 128, <= 1024 */
  uint32_t classes;                   /* 2..32 */
  uint64_t seed;                      /* counter-based draws of densities, masks, noise */
  float dens_lo, dens_hi;             /* 0 <= lo <= hi <= 1 */
  float noise_rel_std;                /* >= 0 */
} gevo_cnn_config;

typedef struct gevo_cnn gevo_cnn;     /* opaque handle */

/* Number of floats of the canonical parameter vector.  GEVO_E_UNSUPPORTED
 * for shapes outside the limits above or whose pointwise layers would see a
 * row count (64 images x pixels) that is not a multiple of 256. */
gevo_status gevo_cnn_param_count(const gevo_cnn_config* cfg, size_t* count);

/* Device workspace for n_test test images (caller-owned, 256-byte aligned). */
gevo_status gevo_cnn_workspace_bytes(const gevo_cnn_config* cfg, int64_t n_test, size_t* bytes);

/* Builds the population on the device.  base_params: host array of
 * gevo_cnn_param_count floats (read during the call).  d_test_x, d_test_y:
 * device arrays that must outlive the handle.  Synchronous; labels outside
 * [0, classes) give GEVO_E_SHAPE.  The library allocates no device memory. */
gevo_status gevo_cnn_init(const gevo_cnn_config* cfg, void* d_ws, size_t ws_bytes, const float* base_params,
                          const float* d_test_x, const int32_t* d_test_y, int64_t n_test, void* hip_stream,
                          gevo_cnn** out);

/* Runs every variant over the test set (asynchronous on the stream). */
gevo_status gevo_cnn_predict(gevo_cnn* h);

/* Mean test CE and accuracy per variant (host arrays of P, any may be NULL)
 * and time_s = wall time of the last predict divided by P.  Synchronises;
 * GEVO_E_ORDER before the first predict. */
gevo_status gevo_cnn_scores(gevo_cnn* h, float* test_loss, float* test_acc, float* time_s);

/* Structural edit: variant v loses block layer `layer` (its index in the
 * canonical tensor order: 2 i + 1 the depthwise layer of block i, 2 i + 2
 * its pointwise layer).  Section 6.1 removes a convolution layer of
 * MobileNet; section 4.1 repairs the shapes that an edit breaks by
 * shrinking or padding tensors.  The removed layer passes its input on,
 * repaired to the shape the next layer reads: a depthwise layer of stride 2
 * keeps the pixels (2 yo, 2 xo); a pointwise layer keeps its first
 * block_channels[i] channels or appends channels of value 1 (the value
 * section 4.1 pads with).  The variant's master of that layer is
 * overwritten by the layer's identity form (the depthwise centre tap 1, or
 * ones on the pointwise diagonal; every other weight +0; every bias +0
 * except 1 for appended channels; the mask marks the ones), which computes
 * exactly that on the layer's non-negative (ReLU) inputs, so later predict
 * calls see the edit and gevo_cnn_export returns that form.  The edit
 * cannot be undone short of a new gevo_cnn_init.  Asynchronous on the
 * handle's stream; allocates nothing.  GEVO_E_ARG for v >= P or a layer
 * past the head, GEVO_E_UNSUPPORTED for the stem (0) and the head
 * (2 n_blocks + 1). */
gevo_status gevo_cnn_remove_layer(gevo_cnn* h, uint32_t v, uint32_t layer);

/* Variant v's parameters (canonical layout), mask (uint8 0/1 over the
 * weights, same order) and density rho_v (the draw of gevo_cnn_init; not
 * updated by gevo_cnn_remove_layer); any output may be NULL. */
gevo_status gevo_cnn_export(gevo_cnn* h, uint32_t v, float* params_out, uint8_t* mask_out, float* density_out);

/* Kernel-level timing, as for gevo_pop_set_profiling: with profiling enabled
 * every kernel that gevo_cnn_predict enqueues carries a HIP event pair
 * recorded by its own dispatch on the handle's stream; gevo_cnn_kernel_stats
 * synchronises and returns, per kind, the summed kernel time in ms and the
 * launch count since the handle was created.  GEVO_E_ARG for a null handle
 * or a kind outside the enum. */
typedef enum {
  GEVO_CNN_KERNEL_STEM = 0,        /* 3x3 stem convolution */
  GEVO_CNN_KERNEL_DEPTHWISE = 1,   /* 3x3 depthwise convolutions */
  GEVO_CNN_KERNEL_POINTWISE = 2,   /* 1x1 pointwise convolutions (per-variant GEMMs) */
  GEVO_CNN_KERNEL_POOL = 3,        /* global average pooling */
  GEVO_CNN_KERNEL_HEAD = 4,        /* fully connected head, loss and argmax */
  GEVO_CNN_KERNEL_REDUCE = 5,      /* per-variant sums of the chunks' partial scores */
  GEVO_CNN_KERNEL_POINTWISE_DEPTHWISE = 6,   /* a pointwise layer fused with the next depthwise layer */
  GEVO_CNN_KERNEL_KINDS = 7
} gevo_cnn_kernel_kind;

gevo_status gevo_cnn_set_profiling(gevo_cnn* h, int enable);
gevo_status gevo_cnn_kernel_stats(gevo_cnn* h, int kind, double* total_ms, uint64_t* launches);

void gevo_cnn_destroy(gevo_cnn* h);

#ifdef __cplusplus
}
#endif

#endif /* GEVO_H */
