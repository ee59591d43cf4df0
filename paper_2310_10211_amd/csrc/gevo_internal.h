// Internal declarations shared by the host runtime (gevo_capi.hip) and the
// kernels (gevo_kernels.hip) of libgevo.  Not part of the C-ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace gevo {

// Tiling constants every launcher checks its shapes against.
constexpr int kTile = 32;          // MFMA output tile edge; all padded dims are multiples
constexpr int kThreads = 256;      // 4 wave64 per workgroup
constexpr int kPassRows = 256;     // forward rows per pass of the layer kernel
constexpr int kOutRows = 256;      // rows per workgroup of the output kernel (predict)
constexpr int kPredictChunk = 2048;  // test rows per predict chunk
constexpr size_t kLdsBudget = 120 * 1024;  // dynamic LDS of the output kernel (one workgroup per variant)
constexpr size_t kLayerLds = 76 * 1024;   // dynamic LDS per hidden-layer workgroup (two fit in 160 KiB)

// Philox stream ids (counter word 3)
constexpr uint32_t kStreamLr = 1, kStreamDens = 2, kStreamMask = 3, kStreamInit = 4,
                   kStreamNoise = 5, kStreamPerm = 6, kStreamSelect = 7, kStreamCross = 8,
                   kStreamMut = 9;
constexpr uint32_t kMaxGenomePrunes = 64;   // pruning edits per variant held on the device

inline int round_up(int x, int m) { return (x + m - 1) / m * m; }

// ---------------------------------------------------------------- kernels args
// Storage type S is float (fp32 path) or uint16_t holding bfloat16 bits.

struct InitArgs {
  int P, l_index, K, N, Kp, Np;  // layer shape (true and padded)
  uint64_t seed;
  int init_kind;                 // 0 Xavier, 1 base * (1 + std * eps)
  float xavier_a;                // fl32(sqrt(6/(K+N)))
  float noise_std;
  const float* base_w;           // optional base weights, device, [Np][Kp] padded (layer slice)
  const float* base_b;           // optional base biases, device, [Np]
  const uint32_t* thresh;        // [P] mask thresholds
  // optional genomes: variant v keeps a weight only when each of its pruning
  // edits i in [prune_off[v], prune_off[v+1]) keeps it, drawing with
  // prune_id[i] where the initial population draws with v, against prune_th[i]
  const uint32_t* prune_off;     // [P+1] (null: one edit per variant, (v, thresh[v]))
  const uint32_t* prune_id;
  const uint32_t* prune_th;
  // optional structural edits: variant v keeps inputs k < width_in[v], units
  // n < width_out[v] and, when bias_keep[v], their biases (null: everything)
  const uint32_t* width_in;      // [P]
  const uint32_t* width_out;     // [P]
  const uint32_t* bias_keep;     // [P]
  // optional removed layers: variant v with ident[v] != 0 gets the identity
  // form (W[k][k] = 1 for k < min(width_in, width_out), bias 1 for units
  // width_in <= n < width_out, everything else +0; the mask marks the ones)
  const uint32_t* ident;         // [P]
  float* Wm;                     // [P][Kp/32][Np][32] (k-blocked)
  float* bias;                   // [P][Np]
  uint32_t* mask;                // [P][Np][Kp/32] row words
};

template <typename S>
struct LayerArgs {
  int Kp, Np;                    // padded input / output width of the layer
  int KB;                        // input columns per LDS block (set by the launcher)
  int Bp;                        // padded batch rows of the update
  float* Wm;                     // [P][Kp/32][Np][32] fp32 master (k-blocked)
  float* bias;                   // [P][Np]
  const uint32_t* mask;          // [P][Np][Kp/32] row words: bit k%32 of word [n][k/32]
  const uint32_t* bmask;         // [P][Np/32]: bit n%32 of word n/32 = bias n is trained
  const float* lr;               // [P]
  int do_update;
  const S* Gcols; size_t g_vs;   // [v][Np][Bp] gradient at this layer's output
  const S* Acols; size_t ac_vs;  // [v][Kp][Bp] input activations (vs = 0: shared by all variants)
  int do_forward;
  int R;                         // forward rows (multiple of kTile)
  const S* Arows; size_t ar_vs;  // [v][R][Kp] forward input rows
  S* Orows; size_t or_vs;        // [v][R][Np] relu output rows
  S* Ocols; size_t oc_vs;        // [v][Np][R] relu output, transposed (nullable)
  S* Wt;                         // [v][Kp][Np] operand copy of W, transposed (nullable)
  // bf16 streaming kernel only: the master as a register image and its mask
  // words block-major (see launch_w1_image / launch_mask_block_major)
  float* Wimg;                   // [P][Kp/32][Np/32][4][64][4]
  const uint32_t* mblk;          // [P][Kp/32][Np]
  // structural edits: variant v keeps units n < wout[v] of this layer (null:
  // all); a workgroup whose units are all removed does nothing (their
  // weights and biases are +0 and stay +0; the caller keeps their activation
  // and operand-copy slots at zero)
  const uint32_t* wout;
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
};

// bf16 forward of a hidden layer over prediction rows (no update)
struct FwdGemmArgs {
  const uint16_t* A; size_t a_vs;   // [v][R][Kp] input rows (a_vs = 0: shared by all variants)
  const float* Wm;                  // [P][Kp/32][Np][32] fp32 master (k-blocked)
  const float* bias;                // [P][Np]
  uint16_t* O; size_t o_vs;         // [v][R][Np] relu output rows
  int Kp, Np, R, P;
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
};

// bf16 prediction GEMM of a hidden layer (gevo_predict.hip): per variant
// O = bf16(relu(A W + b)) over R rows, W the bf16 operand copy; with WL set,
// the layer (Np == 256) is the last hidden one and its tile also runs the
// output layer, writing per-tile loss sums and hit counts instead of O
struct PredGemmArgs {
  const uint16_t* A; size_t a_vs;   // [v][R][Kp] input rows (a_vs = 0: shared by all variants)
  const uint16_t* W;                // [P][Np][Kp] bf16 weights
  const float* bias;                // [P][Np]
  uint16_t* O; size_t o_vs;         // [v][R][Np] relu output rows (unused with WL)
  int Kp, Np, R, P;
  const float* WL;                  // output layer master [P][Np/32][32][32] (k-blocked), or null
  const float* bL;                  // [P][32]
  int C;                            // classes
  const int32_t* labels;            // [R] labels of the chunk's rows, < 0 for padding rows
  int chunk0, n_chunks_total;       // partial sums at [v][chunk0 + row tile]
  double* part_ce;
  unsigned int* part_correct;
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
};

template <typename S>
struct OutArgs {
  int Kp;                        // padded width of the last hidden layer (input of the output layer)
  int C;                         // classes (<= 32); padded output width is 32
  int Bp;                        // padded batch rows (training)
  float* Wm;                     // [P][Kp/32][32][32] (k-blocked)
  float* bias;                   // [P][32]
  const uint32_t* mask;          // [P][32][Kp/32] row words
  const uint32_t* bmask;         // [P]: bit c = bias of class c is trained
  const float* lr;               // [P]
  int train;                     // 1: loss + backward + update on one batch; 0: predict chunk
  const S* Arows; size_t ar_vs;  // [v][rows][Kp]
  const S* Acols; size_t ac_vs;  // [v][Kp][Bp] (training)
  const int32_t* labels;         // [rows]; < 0 marks a padding row
  int rows;                      // rows covered by the grid (training: Bp)
  float scale;                   // fl32(1/b_t)
  const float* gscale;           // [P][Bp][32] per-element output-gradient scale (nullable: scale)
  double* ce_acc;                // [P] training accumulators
  unsigned long long* correct_acc;
  int chunk0;                    // predict: index of the first 256-row chunk
  int n_chunks_total;            // predict: stride of the partial arrays
  double* part_ce;               // [P][n_chunks_total]
  unsigned int* part_correct;
  S* Gcols; size_t gc_vs;        // [v][Kp][Bp] gradient of the last hidden layer (training)
  S* Grows; size_t gr_vs;        // [v][Bp][Kp] same, row-major (nullable)
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
  // training, between the two passes: G rows [P][Bp][32] and, per 32-row
  // tile, the sums of G by class [P][Bp/32][32], of CE [P][Bp/32] and hits
  S* ogrd;
  float* opdb;
  double* opce;
  unsigned int* opcorr;
};

template <typename S>
struct BwdArgs {
  int Kp, Np, Bp;                // layer l: input width Kp, output width Np
  const S* Wt;                   // [v][Kp][Np] pre-update operand weights, transposed
  const S* Grows; size_t gr_vs;  // [v][Bp][Np] gradient at layer l output
  const S* Acols; size_t ac_vs;  // [v][Kp][Bp] activations of layer l-1 (for ReLU')
  S* Gcols; size_t gc_vs;        // [v][Kp][Bp] gradient at layer l-1 output
  S* Grows_out; size_t go_vs;    // [v][Bp][Kp] (nullable)
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
};

// Fused per-variant training of a two-layer net (bf16 operands), one
// workgroup per variant over steps [t0, t1) of an epoch.
struct Fused2Args {
  int Kp, Hp, C, B, Bp, T;       // input width, hidden width (128|256), classes, batch, padded batch, steps/epoch
  int64_t n;                     // training rows
  int t0, t1;
  const uint16_t* xrows;         // [T][Kp/32][Bp][32] bf16 bits (block-major rows)
  const uint16_t* xcols;         // [T][Kp][Bp]
  const int32_t* labels;         // [T][Bp]
  float* W1; float* b1; const uint32_t* m1;   // register image (see launch_w1_image), [P][Hp], [P][Kp/32][Hp]
  float* W2; float* b2; const uint32_t* m2;   // [P][Hp/32][32][32], [P][32], [P][32][Hp/32]
  const uint32_t* bm1; const uint32_t* bm2;   // bias masks [P][Hp/32], [P] (bit = bias trained)
  const float* lr;               // [P] learning rate of W1, b1 (0 for a removed hidden layer)
  const float* lr2;              // [P] learning rate of W2, b2
  double* ce_acc;
  unsigned long long* correct_acc;
  const float* gscale;           // [P][Bp][32] per-element output-gradient scale (nullable: fl32(1/b_t))
  unsigned long long* vtime;      // [P] per-variant device time in clock ticks (nullable)
};

// Resident training of two-layer nets (gevo_resident.hip): a pair of
// workgroups per variant, exchanging their halves' logits once per step.
constexpr int kResXW = 2048;             // exchange words per half and step parity
constexpr int kResMaxPairs = 128;        // pairs per launch (variants beyond run in later rounds)
struct Res2Args {
  Fused2Args f;                          // X copies in the resident layout (perm32 within each block)
  unsigned long long* xbuf;              // [kResMaxPairs][2 halves][2 parities][kResXW], zero before the launch
  unsigned int* err;                     // set to 1 when a half gave up waiting for its partner
  int P;
};

// Position of element x (0..31) of a 32-element block in the resident X
// copies: the middle two groups of four of each 16 are swapped (an involution).
__host__ __device__ inline int perm32(int x) {
  const int a = (x >> 2) & 3;
  return (x & ~12) | ((((a & 1) << 1) | (a >> 1)) << 2);
}

struct GatherArgs {
  const float* X;                // [n][d0] caller's rows
  const int32_t* y;              // [n]
  const uint32_t* perm;          // [n] (nullable: identity)
  int64_t n;
  int d0, Kp, B, Bp, T;          // T = steps (row blocks)
  int blocked;                   // rows block-major, [T][Kp/32][Bp][32], instead of [T][Bp][Kp]
  int res_order;                 // (blocked only) element k of a block at position perm32(k)
  void* rows;                    // [T][Bp][Kp] S
  int32_t* labels;               // [T][Bp]
};

struct TransposeArgs {
  const void* src;               // [T][Bp][Kp] S, or [T][Kp/32][Bp][32] when blocked
  void* dst;                     // [T][Kp][Bp] S
  int Kp, Bp, T;
  int blocked;
  int res_order;                 // source positions perm32(k); destination rows keep k and put row b of
                                 // each 32 at column position perm32(b)
};

// ---------------------------------------------------------------- launchers
// Each returns hipSuccess or the launch error.  Shapes are validated by the
// caller (gevo_capi.hip) before these are reached.  A non-null event pair is
// recorded by the dispatch itself around the kernel (kernel-level timing).
struct LaunchEv {
  hipEvent_t start = nullptr, stop = nullptr;
};
hipError_t launch_init(const InitArgs& a, hipStream_t s, const LaunchEv& ev);
template <typename S> hipError_t launch_layer(const LayerArgs<S>& a, int P, hipStream_t s, const LaunchEv& ev);
template <typename S> hipError_t launch_out(const OutArgs<S>& a, int P, hipStream_t s, const LaunchEv& ev);
template <typename S> hipError_t launch_bwd(const BwdArgs<S>& a, int P, hipStream_t s, const LaunchEv& ev);
template <typename S> hipError_t launch_gather(const GatherArgs& a, hipStream_t s, const LaunchEv& ev);
template <typename S> hipError_t launch_transpose(const TransposeArgs& a, hipStream_t s, const LaunchEv& ev);
hipError_t launch_zero_bytes(void* p, size_t bytes, hipStream_t s, const LaunchEv& ev);
hipError_t launch_fused2(const Fused2Args& a, int P, hipStream_t s, const LaunchEv& ev);
// W1 master of a two-layer net: k-blocked layout <-> the fused kernel's register image
hipError_t launch_w1_image(const float* src, float* dst, int P, int Kp, int Hp, bool to_image, hipStream_t s,
                           const LaunchEv& ev);
// W1 mask row words [P][Hp][Kp/32] -> block-major words [P][Kp/32][Hp]
hipError_t launch_mask_block_major(const uint32_t* src, uint32_t* dst, int P, int Kp, int Hp, hipStream_t s,
                                   const LaunchEv& ev);
hipError_t launch_bf16_check(unsigned long long* counts, hipStream_t s);   // counts zeroed by the caller
bool fwd_gemm_supported(int Kp, int Np, int R);   // Kp % 32, Np % 128, R % 256
hipError_t launch_fwd_gemm(const FwdGemmArgs& a, hipStream_t s, const LaunchEv& ev);
bool pred_gemm_supported(int Kp, int Np, int R);  // Kp % 32, Np % 256, R % 256
hipError_t launch_pred_gemm(const PredGemmArgs& a, hipStream_t s, const LaunchEv& ev);
// k-blocked fp32 master [P][Kp/32][Np][32] -> bf16 [P][Np][Kp] (Np % 256 == 0)
hipError_t launch_wt_bf16(const float* Wm, uint16_t* Wb, int P, int Kp, int Np, hipStream_t s, const LaunchEv& ev);
// bf16 hidden layer over one training batch (update and/or forward of the
// next batch) streaming the fp32 master once; shapes outside these use k_layer
bool stream_layer_supported(int Kp, int Np, int Bp, int R);
// bf16 backward GEMM of a hidden layer (per variant, LDS-tiled); other shapes use k_bwd
bool bwd_gemm_supported(int Kp, int Np, int Bp);
hipError_t launch_bwd_gemm(const BwdArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev);
hipError_t launch_stream_layer(const LayerArgs<uint16_t>& a, int P, hipStream_t s, const LaunchEv& ev);
size_t fused2_lds_bytes(int hp, int bp);     // 0 when the shape has no fused instantiation
bool res2_supported(int Kp, int Hp, int Bp, int C);   // Kp 800, Hp 256, Bp 128, C <= 16
int res2_max_pairs();                        // co-resident pairs on the current device (0: no cooperative launch)
hipError_t launch_res2(const Res2Args& a, int pairs, hipStream_t s, const LaunchEv& ev);
hipError_t launch_reduce_partials(const double* part_ce, const unsigned int* part_corr, int P, int n_chunks,
                                  double* ce_out, unsigned long long* corr_out, hipStream_t s, const LaunchEv& ev);

// Philox4x32-10 on the host (the library's own draws: learning rates,
// densities, data order).
void philox4x32_10_host(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

}  // namespace gevo
