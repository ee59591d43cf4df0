/*
 * gevo_oracle.c -- CPU oracle for population-batched fitness evaluation
 * (GEVO-ML, arXiv 2310.10211).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, deliberately naive
 * CPU implementation of what the GPU path computes.  Only the test-suite, the
 * smoke check and the CPU-baseline leg of the benchmark may build, load or call
 * it.  It shares no code, header, table or helper with the HIP library; the two
 * implement the same published definitions independently.
 *
 * What is modelled (paper, section 4.3 "Fitness Evaluation" and section 6.2):
 * each individual of the population is evaluated by retraining its model on the
 * dataset (training workload) or by running it over the dataset (prediction
 * workload), and is scored by error and time.  The paper's training model is a
 * net of two fully-connected layers trained by mini-batch SGD, where the output
 * gradient is the difference between prediction and label, reduced over the
 * batch, scaled by 1/batch (1/32 in the paper), multiplied by the learning rate
 * and subtracted from weights and biases (section 6.2).  Its key mutations act
 * like a changed learning rate (section 6.2) and like pruning of non-essential
 * parameters (abstract; section 2 on GEVO's SGD result), so a variant here is
 * (learning rate, pruning mask) applied to a copy of the original model
 * (section 4: the initial population consists of mutated copies of the
 * original program).
 *
 * Precision modes:
 *   OR_F64  -- everything in binary64; no rounding anywhere (for pins).
 *   OR_F32  -- binary32 storage and binary32 elementwise ops; every dot product
 *              is accumulated exactly enough in binary64 and rounded once.
 *   OR_BF16 -- as OR_F32, plus round-to-nearest-even to bfloat16 of every GEMM
 *              operand: the input rows, the weights (taken from the fp32
 *              master each step), each hidden activation after ReLU and each
 *              gradient before it is used as a GEMM operand.  Logits, softmax,
 *              loss, bias gradients, weight gradients and the master update
 *              stay binary32.
 * Elementwise binary32 operations are evaluated in binary64 and rounded to
 * binary32; for +, -, *, / and sqrt this gives the correctly rounded binary32
 * result because 53 >= 2*24+2.  Build with -ffp-contract=off.
 *
 * Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), written here from that paper.
 * Counter words (c0, c1, c2, c3) = (block index, layer, variant or epoch,
 * stream id); key = (seed low 32 bits, seed high 32 bits).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F64 0
#define OR_F32 1
#define OR_BF16 2

#define OR_STREAM_LR 1u
#define OR_STREAM_DENS 2u
#define OR_STREAM_MASK 3u
#define OR_STREAM_INIT 4u
#define OR_STREAM_NOISE 5u
#define OR_STREAM_PERM 6u

#define OR_MAX_LAYERS 7
#define OR_PI 3.14159265358979323846

/* ------------------------------------------------------------------------ */
/* Philox4x32-10, per the SC'11 paper: ten rounds of two 32x32->64 bit        */
/* multiplications whose high halves are xored with the other counter words   */
/* and the round key; the key is bumped by the Weyl constants between rounds. */
/* ------------------------------------------------------------------------ */
void or_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)x0;
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)x2;
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    x0 = hi1 ^ x1 ^ k0;
    x1 = lo1;
    x2 = hi0 ^ x3 ^ k1;
    x3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

static uint32_t draw_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2,
                          uint32_t stream, uint32_t word) {
  uint32_t ctr[4] = {c0, c1, c2, stream};
  uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
  uint32_t out[4];
  or_philox4x32_10(ctr, key, out);
  return out[word];
}

/* 24-bit uniform on [0,1): top 24 bits of a word, times 2^-24 (exact). */
static double u24_of(uint32_t r) { return (double)(r >> 8) * (1.0 / 16777216.0); }

/* ------------------------------------------------------------------------ */
/* Rounding helpers                                                          */
/* ------------------------------------------------------------------------ */
static double f32(double x) { return (double)(float)x; }

/* IEEE round-to-nearest-even from binary32 to bfloat16, by bit arithmetic. */
float or_bf16_round(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) {      /* NaN stays a (quiet) NaN */
    u = (u | 0x00400000u) & 0xffff0000u;
  } else {
    uint32_t lsb = (u >> 16) & 1u;
    u = (u + 0x7fffu + lsb) & 0xffff0000u;
  }
  memcpy(&f, &u, 4);
  return f;
}

/* rounding of a stored working value */
static double rw(int mode, double x) { return mode == OR_F64 ? x : f32(x); }
/* rounding of a GEMM operand */
static double rop(int mode, double x) {
  if (mode == OR_F64) return x;
  if (mode == OR_F32) return f32(x);
  return (double)or_bf16_round((float)x);
}

/* ------------------------------------------------------------------------ */
/* Parameter layout (canonical): for each layer l = 1..L, W_l row-major as    */
/* d_{l-1} x d_l ("in x out"), followed by b_l (d_l entries).                 */
/* ------------------------------------------------------------------------ */
size_t or_param_count(int L, const uint32_t* dims) {
  size_t n = 0;
  for (int l = 1; l <= L; ++l) n += (size_t)dims[l - 1] * dims[l] + dims[l];
  return n;
}
size_t or_weight_count(int L, const uint32_t* dims) {
  size_t n = 0;
  for (int l = 1; l <= L; ++l) n += (size_t)dims[l - 1] * dims[l];
  return n;
}
static size_t w_off(const uint32_t* dims, int l) { /* offset of W_l in params */
  size_t n = 0;
  for (int j = 1; j < l; ++j) n += (size_t)dims[j - 1] * dims[j] + dims[j];
  return n;
}
static size_t m_off(const uint32_t* dims, int l) { /* offset of mask of W_l */
  size_t n = 0;
  for (int j = 1; j < l; ++j) n += (size_t)dims[j - 1] * dims[j];
  return n;
}

/* ------------------------------------------------------------------------ */
/* Population generation (section 4: initial population = copies of the     */
/* original model with random edits; the edits' effects are modelled as a    */
/* per-variant learning rate and a per-variant Bernoulli pruning mask).      */
/* ------------------------------------------------------------------------ */
int or_variant_hparams(uint64_t seed, uint32_t v, float lr_lo, float lr_hi,
                       float dens_lo, float dens_hi, const float* dens_list,
                       uint32_t n_dens_list, float* lr, float* dens, uint32_t* thresh) {
  if (lr_lo == lr_hi) {
    *lr = lr_lo;
  } else {
    double u = u24_of(draw_word(seed, 0, 0, v, OR_STREAM_LR, 0));
    double a = log((double)lr_lo), b = log((double)lr_hi);
    *lr = (float)exp(a + u * (b - a));           /* log-uniform in [lo, hi) */
  }
  float rho;
  if (n_dens_list > 0) {
    rho = dens_list[v % n_dens_list];
  } else {
    double u = u24_of(draw_word(seed, 0, 0, v, OR_STREAM_DENS, 0));
    rho = (float)((double)dens_lo + u * ((double)dens_hi - (double)dens_lo));
  }
  *dens = rho;
  double t = (double)rho * 16777216.0;            /* keep <=> u24 < round(rho 2^24) */
  if (t < 0.0) t = 0.0;
  if (t > 16777216.0) t = 16777216.0;
  *thresh = (uint32_t)llround(t);
  return 0;
}

/*
 * Weight (k -> n) of layer l (k < d_{l-1}, n < d_l) has element index
 * e = n * d_{l-1} + k for every draw that concerns it.
 * init_kind 0: Xavier-uniform, identical for every variant (the original
 *              model), biases zero, then the mask is applied.
 * init_kind 1: base model (given in canonical layout, or Xavier from the seed
 *              when base == NULL) times (1 + noise_std * eps), eps ~ N(0,1) by
 *              Box-Muller, then the mask; biases are copied unperturbed.
 * Masked weights are exactly +0.
 */
/* One weight tensor of variant v, viewed as din x dout with layer index li
 * (the third Philox counter word), as section 4 builds the initial
 * population: mask bit keep <=> u24 < thresh; W = Xavier draw (init_kind 0)
 * or base * fl(1 + fl(std * eps)) (init_kind 1, eps by Box-Muller); W = +0
 * where the mask drops it; biases 0 or the base's.  W is [din][dout]
 * row-major, bias [dout], M [din][dout]; base_w/base_b may be NULL. */
int or_tensor_init(uint64_t seed, uint32_t v, uint32_t li, uint32_t din, uint32_t dout, uint32_t thresh,
                   int init_kind, const double* base_w, const double* base_b, float noise_std, double* W,
                   double* bias, uint8_t* M) {
  float a = (float)sqrt(6.0 / ((double)din + (double)dout));
  for (uint32_t k = 0; k < din; ++k) {
    for (uint32_t n = 0; n < dout; ++n) {
      uint64_t e = (uint64_t)n * din + k;
      uint32_t rm = draw_word(seed, (uint32_t)(e >> 2), li, v, OR_STREAM_MASK, (uint32_t)(e & 3));
      int keep = (rm >> 8) < thresh;
      double w;
      if (init_kind == 1 && base_w != NULL) {
        w = base_w[(size_t)k * dout + n];
      } else {
        uint32_t ri = draw_word(seed, (uint32_t)(e >> 2), li, 0, OR_STREAM_INIT, (uint32_t)(e & 3));
        double t = 2.0 * u24_of(ri) - 1.0;      /* exact in binary32 */
        w = f32(t * (double)a);
      }
      if (init_kind == 1) {
        uint32_t c0 = (uint32_t)(e >> 1), w0 = (uint32_t)((e & 1) * 2);
        uint32_t ra = draw_word(seed, c0, li, v, OR_STREAM_NOISE, w0);
        uint32_t rb = draw_word(seed, c0, li, v, OR_STREAM_NOISE, w0 + 1);
        double u1 = (double)((ra >> 8) + 1u) * (1.0 / 16777216.0);  /* (0,1] */
        double u2 = u24_of(rb);
        double eps = sqrt(-2.0 * log(u1)) * cos(2.0 * OR_PI * u2);
        double s = f32(1.0 + f32((double)noise_std * f32(eps)));
        w = f32(w * s);
      }
      W[(size_t)k * dout + n] = keep ? w : 0.0;
      M[(size_t)k * dout + n] = (uint8_t)keep;
    }
  }
  for (uint32_t n = 0; n < dout; ++n) bias[n] = (init_kind == 1 && base_b != NULL) ? base_b[n] : 0.0;
  return 0;
}

int or_variant_init(uint64_t seed, uint32_t v, int L, const uint32_t* dims,
                    uint32_t thresh, int init_kind, const double* base, float noise_std,
                    double* params, uint8_t* mask) {
  if (L < 1 || L > OR_MAX_LAYERS) return -1;
  for (int l = 1; l <= L; ++l) {
    uint32_t din = dims[l - 1], dout = dims[l];
    double* W = params + w_off(dims, l);
    const double* bw = base ? base + w_off(dims, l) : NULL;
    or_tensor_init(seed, v, (uint32_t)(l - 1), din, dout, thresh, init_kind, bw, bw ? bw + (size_t)din * dout : NULL,
                   noise_std, W, W + (size_t)din * dout, mask + m_off(dims, l));
  }
  return 0;
}

/* Mask of an individual whose pruning edits are (edit_id[i], thresh[i]),
 * i < n_edits.  An edit keeps weight (layer l, flat index e = n*din + k) when
 * the top 24 bits of its mask draw, taken with the edit id where the initial
 * population uses the variant index, fall below its threshold; a weight is
 * kept when every edit keeps it (the edits of an individual apply in sequence
 * to the original program, section 4.2; their effect is pruning, abstract).
 * No edit keeps everything.  A single edit (v, T_v) gives the initial mask of
 * variant v (or_variant_init). */
int or_genome_mask(uint64_t seed, int L, const uint32_t* dims, uint32_t n_edits, const uint32_t* edit_id,
                   const uint32_t* thresh, uint8_t* mask) {
  if (L < 1 || L > OR_MAX_LAYERS) return -1;
  for (int l = 1; l <= L; ++l) {
    uint32_t din = dims[l - 1], dout = dims[l];
    uint8_t* M = mask + m_off(dims, l);
    for (uint32_t k = 0; k < din; ++k) {
      for (uint32_t n = 0; n < dout; ++n) {
        uint64_t e = (uint64_t)n * din + k;
        int keep = 1;
        for (uint32_t i = 0; i < n_edits; ++i) {
          uint32_t rm = draw_word(seed, (uint32_t)(e >> 2), (uint32_t)(l - 1), edit_id[i], OR_STREAM_MASK,
                                  (uint32_t)(e & 3));
          if ((rm >> 8) >= thresh[i]) keep = 0;
        }
        M[(size_t)k * dout + n] = (uint8_t)keep;
      }
    }
  }
  return 0;
}

/* Structural edits of an individual: layer l keeps its first width[l] units
 * (width[0] = d0 and width[L] = dL: inputs and classes are never removed) and
 * its bias unless bias_keep[l-1] is 0 (removing the bias term, section 6.1;
 * shrinking a tensor, the repair of section 4.1).  Clears the weights into
 * and out of removed units in the weight mask (canonical order) and writes
 * the bias mask (bmask, over all biases, 1 = trained).  A network whose
 * removed units have no weights and no bias computes exactly what the
 * narrower network computes. */
int or_structure_masks(int L, const uint32_t* dims, const uint32_t* width, const uint8_t* bias_keep,
                       uint8_t* mask, uint8_t* bmask) {
  if (L < 1 || L > OR_MAX_LAYERS) return -1;
  size_t bo = 0;
  for (int l = 1; l <= L; ++l) {
    uint32_t din = dims[l - 1], dout = dims[l];
    uint8_t* M = mask + m_off(dims, l);
    for (uint32_t k = 0; k < din; ++k)
      for (uint32_t n = 0; n < dout; ++n)
        if (k >= width[l - 1] || n >= width[l]) M[(size_t)k * dout + n] = 0;
    for (uint32_t n = 0; n < dout; ++n) bmask[bo + n] = (uint8_t)(n < width[l] && bias_keep[l - 1]);
    bo += dout;
  }
  return 0;
}

/* Per-epoch data order, shared by all variants: Fisher-Yates from the end,
 * swap index j = floor(r * (i+1) / 2^32) with r a 32-bit Philox word
 * (multiply-shift, no rejection). */
void or_permutation(uint64_t seed, uint32_t epoch, uint32_t n, uint32_t* perm) {
  for (uint32_t i = 0; i < n; ++i) perm[i] = i;
  for (uint32_t i = n; i-- > 1;) {
    uint32_t r = draw_word(seed, i >> 2, 0, epoch, OR_STREAM_PERM, i & 3);
    uint32_t j = (uint32_t)(((uint64_t)r * (uint64_t)(i + 1)) >> 32);
    uint32_t tmp = perm[i]; perm[i] = perm[j]; perm[j] = tmp;
  }
}

/* ------------------------------------------------------------------------ */
/* Forward, loss and backward on one mini-batch of b rows.                    */
/* ------------------------------------------------------------------------ */
typedef struct {
  int L;
  const uint32_t* dims;
  double* act[OR_MAX_LAYERS + 1];   /* act[0] = operand-rounded input rows; act[l] = hidden l */
  double* logits;                   /* b x dL */
  double* G;                        /* scratch: gradient of the current layer output */
  double* Gprev;
  double* wop;                      /* scratch: operand-rounded weights */
} work_t;

static int argmax_correct(const double* z, uint32_t C, int32_t y) {
  uint32_t best = 0;
  double bz = z[0];
  int nan = isnan(z[0]);
  for (uint32_t c = 1; c < C; ++c) {
    if (isnan(z[c])) nan = 1;
    else if (z[c] > bz) { best = c; bz = z[c]; }   /* strict: lowest index wins ties */
  }
  return !nan && (int32_t)best == y;
}

/* forward of rows act[0] (b x d0) through all layers; fills act[1..L-1], logits */
static void forward(int mode, work_t* w, const double* params, uint32_t b) {
  int L = w->L;
  const uint32_t* d = w->dims;
  for (int l = 1; l <= L; ++l) {
    uint32_t din = d[l - 1], dout = d[l];
    const double* W = params + w_off(d, l);
    const double* bias = W + (size_t)din * dout;
    for (size_t i = 0; i < (size_t)din * dout; ++i) w->wop[i] = rop(mode, W[i]);
    const double* A = w->act[l - 1];
    double* out = (l < L) ? w->act[l] : w->logits;
    for (uint32_t i = 0; i < b; ++i) {
      for (uint32_t n = 0; n < dout; ++n) {
        double acc = 0.0;
        for (uint32_t k = 0; k < din; ++k) acc += A[(size_t)i * din + k] * w->wop[(size_t)k * dout + n];
        double z = rw(mode, rw(mode, acc) + bias[n]);           /* Z_l = A_{l-1} W_l + b_l */
        if (l < L) out[(size_t)i * dout + n] = rop(mode, z > 0.0 ? z : 0.0);  /* ReLU */
        else out[(size_t)i * dout + n] = z;
      }
    }
  }
}

/* Softmax cross-entropy of one logit row; optionally the gradient
 * (p - onehot(y)) * scale, or (p - onehot(y))[c] * srow[c] when a row of a
 * gradient-scale tensor is given (the 2fcNet mutation replaces the scalar
 * 1/32 by a tensor of the gradient's shape, section 6.2).
 * Returns CE = log sum exp(z - m) + m - z_y. */
static double softmax_ce(int mode, const double* z, uint32_t C, int32_t y, double scale,
                         const float* srow, double* g, double* probs) {
  double m = z[0];
  for (uint32_t c = 1; c < C; ++c) if (z[c] > m) m = z[c];
  double s = 0.0;
  double e[256];
  for (uint32_t c = 0; c < C; ++c) { e[c] = rw(mode, exp(rw(mode, z[c] - m))); s = rw(mode, s + e[c]); }
  double lse = rw(mode, rw(mode, log(s)) + m);
  double ce = rw(mode, lse - z[y]);
  for (uint32_t c = 0; c < C; ++c) {
    double p = rw(mode, e[c] / s);
    if (probs) probs[c] = p;
    if (g) g[c] = rw(mode, rw(mode, p - (c == (uint32_t)y ? 1.0 : 0.0)) * (srow ? (double)srow[c] : scale));
  }
  return ce;
}

/*
 * Gradients of the batch loss sum_i CE_i * scale with respect to all parameters
 * (section 6.2: output gradient = prediction - label, reduced over the batch and
 * multiplied by 1/batch).  grads has the canonical parameter layout.
 * ReLU'(z) is taken as [stored activation > 0], so ReLU'(0) = 0.
 */
static void backward(int mode, work_t* w, const double* params, const int32_t* y, uint32_t b,
                     double scale, const float* gscale, double* grads, double* ce_sum, uint64_t* correct,
                     double* probs) {
  int L = w->L;
  const uint32_t* d = w->dims;
  uint32_t C = d[L];
  double* G = w->G;                 /* b x d_l, working precision (unrounded) */
  for (uint32_t i = 0; i < b; ++i) {
    const double* z = w->logits + (size_t)i * C;
    double ce = softmax_ce(mode, z, C, y[i], scale, gscale ? gscale + (size_t)i * C : NULL, G + (size_t)i * C,
                           probs ? probs + (size_t)i * C : NULL);
    if (ce_sum) *ce_sum += ce;
    if (correct) *correct += (uint64_t)argmax_correct(z, C, y[i]);
  }
  for (int l = L; l >= 1; --l) {
    uint32_t din = d[l - 1], dout = d[l];
    const double* W = params + w_off(d, l);
    double* dW = grads + w_off(d, l);
    double* db = dW + (size_t)din * dout;
    const double* A = w->act[l - 1];
    /* bias gradient: output layer from the working-precision gradient,
       hidden layers from the operand-rounded (stored) gradient */
    double* Gop = w->Gprev;         /* reuse as operand-rounded copy */
    for (size_t i = 0; i < (size_t)b * dout; ++i) Gop[i] = rop(mode, G[i]);
    for (uint32_t n = 0; n < dout; ++n) {
      double acc = 0.0;
      for (uint32_t i = 0; i < b; ++i) acc += (l == L ? G : Gop)[(size_t)i * dout + n];
      db[n] = rw(mode, acc);
    }
    for (uint32_t k = 0; k < din; ++k)
      for (uint32_t n = 0; n < dout; ++n) {
        double acc = 0.0;
        for (uint32_t i = 0; i < b; ++i) acc += A[(size_t)i * din + k] * Gop[(size_t)i * dout + n];
        dW[(size_t)k * dout + n] = rw(mode, acc);                /* dW_l = A^T G_l */
      }
    if (l > 1) {
      /* G_{l-1} = (G_l W_l^T) * [A_{l-1} > 0], using the pre-update weights */
      for (size_t i = 0; i < (size_t)din * dout; ++i) w->wop[i] = rop(mode, W[i]);
      double* Gn = (double*)malloc(sizeof(double) * (size_t)b * din);
      for (uint32_t i = 0; i < b; ++i)
        for (uint32_t k = 0; k < din; ++k) {
          double acc = 0.0;
          for (uint32_t n = 0; n < dout; ++n) acc += Gop[(size_t)i * dout + n] * w->wop[(size_t)k * dout + n];
          double g = A[(size_t)i * din + k] > 0.0 ? rw(mode, acc) : 0.0;
          Gn[(size_t)i * din + k] = g;
        }
      memcpy(G, Gn, sizeof(double) * (size_t)b * din);
      free(Gn);
    }
  }
}

static int work_alloc(work_t* w, int L, const uint32_t* dims, uint32_t b) {
  memset(w, 0, sizeof(*w));
  w->L = L;
  w->dims = dims;
  uint32_t dmax = 0;
  size_t wmax = 0;
  for (int l = 0; l <= L; ++l) if (dims[l] > dmax) dmax = dims[l];
  for (int l = 1; l <= L; ++l) if ((size_t)dims[l - 1] * dims[l] > wmax) wmax = (size_t)dims[l - 1] * dims[l];
  for (int l = 0; l < L; ++l) {
    w->act[l] = (double*)malloc(sizeof(double) * (size_t)b * dims[l] + 8);
    if (!w->act[l]) return -1;
  }
  w->logits = (double*)malloc(sizeof(double) * (size_t)b * dims[L] + 8);
  w->G = (double*)malloc(sizeof(double) * (size_t)b * dmax + 8);
  w->Gprev = (double*)malloc(sizeof(double) * (size_t)b * dmax + 8);
  w->wop = (double*)malloc(sizeof(double) * wmax + 8);
  if (!w->logits || !w->G || !w->Gprev || !w->wop) return -1;
  return 0;
}
static void work_free(work_t* w) {
  for (int l = 0; l < w->L; ++l) free(w->act[l]);
  free(w->logits); free(w->G); free(w->Gprev); free(w->wop);
}

static int check_dims(int L, const uint32_t* dims) {
  if (L < 1 || L > OR_MAX_LAYERS) return -1;
  for (int l = 0; l <= L; ++l) if (dims[l] == 0) return -2;
  if (dims[L] > 256) return -2;
  return 0;
}

/*
 * Loss and gradients of one batch (rows already gathered; b x d0 binary32
 * inputs).  scale <= 0 selects the default fl(1/b); a gradient-scale tensor
 * gscale (b x dL binary32, nullable) replaces the scalar.  Used by the pins
 * (finite differences, hand-computed example).  probs (b x dL) optional.
 */
int or_batch_grad(int mode, int L, const uint32_t* dims, const double* params,
                  const float* X, const int32_t* y, uint32_t b, double scale, const float* gscale,
                  double* grads, double* ce_sum, double* logits_out, double* probs_out) {
  if (check_dims(L, dims)) return -1;
  if (b == 0) return -2;
  work_t w;
  if (work_alloc(&w, L, dims, b)) { work_free(&w); return -3; }
  for (size_t i = 0; i < (size_t)b * dims[0]; ++i) w.act[0][i] = rop(mode, (double)X[i]);
  if (scale <= 0.0) scale = (mode == OR_F64) ? 1.0 / (double)b : f32(1.0 / (double)b);
  forward(mode, &w, params, b);
  if (logits_out) memcpy(logits_out, w.logits, sizeof(double) * (size_t)b * dims[L]);
  double ce = 0.0;
  backward(mode, &w, params, y, b, scale, gscale, grads, &ce, NULL, probs_out);
  if (ce_sum) *ce_sum = ce;
  work_free(&w);
  return 0;
}

/*
 * Steps [t0, t1) of one epoch of mini-batch SGD for one variant.
 * Step t uses rows perm[t*B .. min(n, (t+1)*B)); the short last batch is kept
 * and scaled by fl(1/b_t), or, when the gradient-scale tensor gscale (batch x
 * dL binary32) is given, row i of every batch by its row i (section 6.2's
 * mutation).  Update (section 6.2: the mean gradient times the
 * learning rate is subtracted from weights and biases):
 *   W <- mask ? fl(W - fl(lr * dW)) : +0,   b <- bmask ? fl(b - fl(lr * db)) : +0
 * (bmask over all biases, nullable: every bias is trained).  A layer l with
 * bit l-1 of `frozen` set (a removed layer, sections 6.1 and 4.1: replaced by
 * the identity map) takes the update with learning rate 0.
 * The loss of step t is taken before its update; ce_sum and correct accumulate.
 */
int or_train_steps(int mode, int L, const uint32_t* dims, double* params, const uint8_t* mask,
                   const uint8_t* bmask, uint32_t frozen, float lr, const float* X, const int32_t* y, uint32_t n,
                   const uint32_t* perm, uint32_t batch, uint32_t t0, uint32_t t1, const float* gscale,
                   double* ce_sum, uint64_t* correct) {
  if (check_dims(L, dims)) return -1;
  if (batch == 0) return -2;
  uint32_t T = (n + batch - 1) / batch;
  if (t1 > T || t0 > t1) return -3;
  work_t w;
  if (work_alloc(&w, L, dims, batch)) { work_free(&w); return -4; }
  size_t np = or_param_count(L, dims);
  double* grads = (double*)malloc(sizeof(double) * np);
  int32_t* yb = (int32_t*)malloc(sizeof(int32_t) * batch);
  if (!grads || !yb) { free(grads); free(yb); work_free(&w); return -4; }
  uint32_t d0 = dims[0];
  for (uint32_t t = t0; t < t1; ++t) {
    uint32_t r0 = t * batch;
    uint32_t b = (n - r0 < batch) ? n - r0 : batch;
    for (uint32_t i = 0; i < b; ++i) {
      uint32_t src = perm[r0 + i];
      for (uint32_t k = 0; k < d0; ++k) w.act[0][(size_t)i * d0 + k] = rop(mode, (double)X[(size_t)src * d0 + k]);
      yb[i] = y[src];
    }
    double scale = (mode == OR_F64) ? 1.0 / (double)b : f32(1.0 / (double)b);
    forward(mode, &w, params, b);
    backward(mode, &w, params, yb, b, scale, gscale, grads, ce_sum, correct, NULL);
    size_t bo = 0;
    for (int l = 1; l <= L; ++l) {
      const double lrd = ((frozen >> (l - 1)) & 1u) ? 0.0 : (double)lr;
      uint32_t din = dims[l - 1], dout = dims[l];
      double* W = params + w_off(dims, l);
      double* dW = grads + w_off(dims, l);
      const uint8_t* M = mask + m_off(dims, l);
      for (size_t i = 0; i < (size_t)din * dout; ++i)
        W[i] = M[i] ? rw(mode, W[i] - rw(mode, lrd * dW[i])) : 0.0;
      double* bias = W + (size_t)din * dout;
      double* db = dW + (size_t)din * dout;
      for (uint32_t j = 0; j < dout; ++j)
        bias[j] = (!bmask || bmask[bo + j]) ? rw(mode, bias[j] - rw(mode, lrd * db[j])) : 0.0;
      bo += dout;
    }
  }
  free(grads); free(yb);
  work_free(&w);
  return 0;
}

/* elementwise bfloat16 rounding of an array (test helper) */
void or_bf16_round_array(const float* x, float* out, size_t n) {
  for (size_t i = 0; i < n; ++i) out[i] = or_bf16_round(x[i]);
}

/* Prediction workload (section 4.3): forward over n rows in order; sums the
 * cross-entropy (binary64) and counts argmax hits (lowest index on ties, any
 * NaN logit counts as a miss). */
int or_predict(int mode, int L, const uint32_t* dims, const double* params,
               const float* X, const int32_t* y, uint32_t n, double* ce_sum, uint64_t* correct) {
  if (check_dims(L, dims)) return -1;
  const uint32_t chunk = 256;
  work_t w;
  if (work_alloc(&w, L, dims, chunk)) { work_free(&w); return -4; }
  uint32_t d0 = dims[0], C = dims[L];
  for (uint32_t r0 = 0; r0 < n; r0 += chunk) {
    uint32_t b = (n - r0 < chunk) ? n - r0 : chunk;
    for (size_t i = 0; i < (size_t)b * d0; ++i) w.act[0][i] = rop(mode, (double)X[(size_t)r0 * d0 + i]);
    forward(mode, &w, params, b);
    for (uint32_t i = 0; i < b; ++i) {
      const double* z = w.logits + (size_t)i * C;
      if (ce_sum) *ce_sum += softmax_ce(mode, z, C, y[r0 + i], 1.0, NULL, NULL, NULL);
      if (correct) *correct += (uint64_t)argmax_correct(z, C, y[r0 + i]);
    }
  }
  work_free(&w);
  return 0;
}
