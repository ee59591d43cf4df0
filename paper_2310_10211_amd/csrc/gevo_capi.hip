// Host runtime and C-ABI of libgevo (declared in include/gevo.h): validates
// configurations, lays out the caller's workspace, draws the per-variant
// hyper-parameters and the per-epoch data order, and enqueues the kernels of
// gevo_kernels.hip on the caller's stream.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <new>
#include <type_traits>
#include <vector>

#include "gevo.h"
#include "gevo_internal.h"

using namespace gevo;

namespace {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct LayerLay {
  int K = 0, N = 0, Kp = 0, Np = 0;
  size_t Wm = 0, bias = 0, mask = 0, Wt = 0, base_w = 0, base_b = 0;
  size_t bmask = 0;                                // [P][Np/32] bias-trained bits
  size_t win = 0, wout = 0, bkeep = 0;             // [P] structural edits (gevo_pop_set_genomes)
  size_t ident = 0;                                // [P] removed layer: identity form (gevo_pop_set_genomes)
  size_t arows[2] = {0, 0}, acols[2] = {0, 0};   // training activations (hidden layers)
  size_t gcols = 0, grows = 0;                     // gradient at this layer's output (hidden)
  size_t prows = 0;                                // predict activations
  bool pred = false;                               // bf16 hidden layer predicted by k_pred_gemm
  size_t wbf = 0;                                  // its bf16 weight copy [P][Np][Kp]
  bool streamed = false;                           // bf16 hidden layer trained by the streaming kernel
  size_t wimg = 0, mblk = 0;                       // its master as a register image, block-major mask words
};

struct Layout {
  int L = 0, P = 0, B = 0, Bp = 0, T = 0;
  bool fused = false;                              // two-layer bf16 nets train in the fused per-variant kernel
  bool resident = false;                           // ... or, for the shapes it covers, in the resident kernel
  bool images = false;                             // some layer trains on a register-image copy of its master
  int64_t n_train = 0, n_test = 0;
  int n_test_pad = 0, n_chunks_test = 0;
  size_t elt = 4;
  LayerLay lay[GEVO_MAX_LAYERS];
  size_t prune_off = 0, prune_id = 0, prune_th = 0;   // genome pruning edits (gevo_pop_set_genomes)
  size_t gscale = 0;                               // [P][Bp][32] output-gradient scales (gevo_pop_set_grad_scale)
  size_t ogrd = 0, opdb = 0, opce = 0, opcorr = 0; // training output layer, between its two passes
  size_t lrh = 0;                                  // [L][P] learning rate of each layer (0: a removed layer)
  size_t lr = 0, thresh = 0, train_ce = 0, train_corr = 0, test_ce = 0, test_corr = 0, part_ce = 0,
         part_corr = 0, xrows = 0, xcols = 0, yep = 0, xte = 0, yte = 0, perm = 0;
  size_t w1img = 0, m1blk = 0;                    // fused training: W1 register image, block-major W1 mask
  size_t xbuf = 0, rerr = 0;                       // resident training: pair exchange words, error word
  size_t vtime = 0;                                // [P] device clock ticks of each variant's waves, last call
  size_t total = 0;
};

// GEVO_RESIDENT=1 in the environment trains the two-layer nets the resident
// kernel covers in that kernel instead of the streaming fused kernel (it is
// correct but slower on gfx950: its register-resident masters leave too few
// registers for the rest of the step, which spills to scratch).
bool resident_requested() {
  const char* e = getenv("GEVO_RESIDENT");
  return e && e[0] && e[0] != '0';
}

gevo_status validate(const gevo_pop_config* c) {
  if (!c) return GEVO_E_ARG;
  if (c->abi_version != GEVO_ABI_VERSION) return GEVO_E_ARG;
  if (c->n_layers < 1 || c->n_layers > GEVO_MAX_LAYERS) return c->n_layers < 1 ? GEVO_E_ARG : GEVO_E_UNSUPPORTED;
  if (c->dtype != GEVO_F32 && c->dtype != GEVO_BF16) return GEVO_E_ARG;
  if (c->init != GEVO_INIT_XAVIER && c->init != GEVO_INIT_BASE_NOISE) return GEVO_E_ARG;
  if (c->P < 1 || c->batch < 1) return GEVO_E_ARG;
  if (c->batch > GEVO_MAX_BATCH) return GEVO_E_UNSUPPORTED;
  for (uint32_t l = 0; l <= c->n_layers; ++l) {
    if (c->dims[l] < 1) return GEVO_E_SHAPE;
    if (c->dims[l] > GEVO_MAX_WIDTH) return GEVO_E_UNSUPPORTED;
  }
  if (c->dims[c->n_layers] > GEVO_MAX_CLASSES) return GEVO_E_UNSUPPORTED;
  if (c->n_train < 0 || c->n_test < 1) return GEVO_E_SHAPE;
  if (c->n_train > 2000000000LL || c->n_test > 2000000000LL) return GEVO_E_UNSUPPORTED;
  if (!(c->lr_lo >= 0.0f) || !(c->lr_hi >= c->lr_lo) || !isfinite(c->lr_hi)) return GEVO_E_ARG;
  if (c->lr_lo < c->lr_hi && !(c->lr_lo > 0.0f)) return GEVO_E_ARG;
  if (c->n_dens_list > 0) {
    if (!c->dens_list) return GEVO_E_ARG;
    for (uint32_t i = 0; i < c->n_dens_list; ++i)
      if (!(c->dens_list[i] >= 0.0f && c->dens_list[i] <= 1.0f)) return GEVO_E_ARG;
  } else if (!(c->dens_lo >= 0.0f && c->dens_hi >= c->dens_lo && c->dens_hi <= 1.0f)) {
    return GEVO_E_ARG;
  }
  if (!isfinite(c->noise_rel_std)) return GEVO_E_ARG;
  return GEVO_OK;
}

// dynamic LDS of the output kernel: operand copy of W_L plus, in training, the gradient rows
size_t out_lds(int Kp, int Bp, size_t elt, int pad) {
  return (size_t)32 * (Kp + pad) * elt + (size_t)Bp * (32 + pad) * elt + (size_t)8 * 32 * 36 * 4;
}

gevo_status make_layout(const gevo_pop_config* c, Layout* o) {
  gevo_status st = validate(c);
  if (st != GEVO_OK) return st;
  Layout& y = *o;
  y = Layout();
  y.L = (int)c->n_layers;
  y.P = (int)c->P;
  y.B = (int)c->batch;
  y.Bp = round_up(y.B, kTile);
  y.n_train = c->n_train;
  y.n_test = c->n_test;
  y.T = (int)((c->n_train + y.B - 1) / y.B);
  y.n_test_pad = round_up((int)c->n_test, kOutRows);
  y.n_chunks_test = y.n_test_pad / kOutRows;
  y.elt = c->dtype == GEVO_BF16 ? 2 : 4;
  const int pad = c->dtype == GEVO_BF16 ? 8 : 1;
  for (int l = 1; l <= y.L; ++l) {
    LayerLay& q = y.lay[l - 1];
    q.K = (int)c->dims[l - 1];
    q.N = (int)c->dims[l];
    q.Kp = round_up(q.K, kTile);
    q.Np = (l == y.L) ? kTile : round_up(q.N, kTile);
  }
  if (out_lds(y.lay[y.L - 1].Kp, y.Bp, y.elt, pad) > kLdsBudget) return GEVO_E_UNSUPPORTED;
  y.fused = y.L == 2 && c->dtype == GEVO_BF16 && fused2_lds_bytes(y.lay[0].Np, y.Bp) > 0;
  y.resident = y.fused && res2_supported(y.lay[0].Kp, y.lay[0].Np, y.Bp, (int)c->dims[2]) && resident_requested();
  for (int l = 0; l + 1 < y.L; ++l) {
    LayerLay& q = y.lay[l];
    q.pred = c->dtype == GEVO_BF16 && pred_gemm_supported(q.Kp, q.Np, kOutRows);
    q.streamed = c->dtype == GEVO_BF16 && !y.fused && stream_layer_supported(q.Kp, q.Np, y.Bp, y.Bp);
    y.images = y.images || q.streamed;
  }
  y.images = y.images || y.fused;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  const size_t P = (size_t)y.P, Bp = (size_t)y.Bp, e = y.elt;
  for (int l = 0; l < y.L; ++l) {
    LayerLay& q = y.lay[l];
    const size_t Kp = q.Kp, Np = q.Np;
    q.Wm = take(P * Np * Kp * 4);
    q.bias = take(P * Np * 4);
    q.mask = take(P * Np * (Kp / 32) * 4);
    q.bmask = take(P * (Np / 32) * 4);
    q.win = take(P * 4);
    q.wout = take(P * 4);
    q.bkeep = take(P * 4);
    q.ident = take(P * 4);
    q.base_w = take(Np * Kp * 4);
    q.base_b = take(Np * 4);
    if (l >= 1 && l < y.L - 1) q.Wt = take(P * Kp * Np * e);         // hidden layer >= 2
    if (l < y.L - 1) {                                                // hidden layer: activations
      for (int bsel = 0; bsel < 2; ++bsel) {
        q.arows[bsel] = take(P * Bp * Np * e);
        q.acols[bsel] = take(P * Np * Bp * e);
      }
      q.gcols = take(P * Np * Bp * e);
      if (l >= 1) q.grows = take(P * Bp * Np * e);
      q.prows = take(P * (size_t)kPredictChunk * Np * e);
    }
    if (q.pred) q.wbf = take(P * Np * Kp * 2);
    if (q.streamed) {
      q.wimg = take(P * Np * Kp * 4);
      q.mblk = take(P * Np * (Kp / 32) * 4);
    }
  }
  y.lr = take(P * 4);
  y.lrh = take((size_t)y.L * P * 4);
  y.thresh = take(P * 4);
  y.prune_off = take((P + 1) * 4);
  y.gscale = take(P * Bp * 32 * 4);
  if (y.n_train > 0) {
    y.ogrd = take(P * Bp * 32 * e);
    y.opdb = take(P * (Bp / 32) * 32 * 4);
    y.opce = take(P * (Bp / 32) * 8);
    y.opcorr = take(P * (Bp / 32) * 4);
  }
  y.prune_id = take(P * (size_t)kMaxGenomePrunes * 4);
  y.prune_th = take(P * (size_t)kMaxGenomePrunes * 4);
  y.vtime = take(P * 8);
  y.train_ce = take(P * 8);
  y.train_corr = take(P * 8);
  y.test_ce = take(P * 8);
  y.test_corr = take(P * 8);
  y.part_ce = take(P * (size_t)y.n_chunks_test * 8);
  y.part_corr = take(P * (size_t)y.n_chunks_test * 4);
  const size_t Kp1 = (size_t)y.lay[0].Kp;
  const size_t T = (size_t)(y.T > 0 ? y.T : 1);
  y.xrows = take(T * Bp * Kp1 * e);
  y.xcols = take(T * Kp1 * Bp * e);
  y.yep = take(T * Bp * 4);
  y.xte = take((size_t)y.n_test_pad * Kp1 * e);
  y.yte = take((size_t)y.n_test_pad * 4);
  y.perm = take((size_t)(y.n_train > 0 ? y.n_train : 1) * 4);
  if (y.fused) {
    const size_t Np1 = (size_t)y.lay[0].Np;
    y.w1img = take(P * Np1 * Kp1 * 4);
    y.m1blk = take(P * Np1 * (Kp1 / 32) * 4);
  }
  if (y.resident) {
    y.xbuf = take((size_t)kResMaxPairs * 2 * 2 * kResXW * 8);
    y.rerr = take(4);
  }
  y.total = off;
  return GEVO_OK;
}

uint32_t draw_word(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t stream, uint32_t word) {
  const uint32_t ctr[4] = {c0, c1, c2, stream};
  const uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
  uint32_t out[4];
  philox4x32_10_host(ctr, key, out);
  return out[word];
}

void fisher_yates(uint64_t seed, uint32_t epoch, uint32_t n, uint32_t* out) {
  for (uint32_t i = 0; i < n; ++i) out[i] = i;
  for (uint32_t i = n; i-- > 1;) {
    const uint32_t r = draw_word(seed, i >> 2, 0, epoch, kStreamPerm, i & 3);
    const uint32_t j = (uint32_t)(((uint64_t)r * (uint64_t)(i + 1)) >> 32);
    const uint32_t t = out[i];
    out[i] = out[j];
    out[j] = t;
  }
}

}  // namespace

namespace gevo {
void philox4x32_10_host(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
  for (int i = 0; i < 10; ++i) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c0, p1 = (uint64_t)0xCD9E8D57u * c2;
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0, n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
    c1 = (uint32_t)p1;
    c3 = (uint32_t)p0;
    c0 = n0;
    c2 = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}
}  // namespace gevo

struct gevo_pop {
  gevo_pop_config cfg{};
  std::vector<float> dens_list;
  Layout y;
  char* ws = nullptr;
  hipStream_t stream = nullptr;
  const float* trX = nullptr;
  const int32_t* trY = nullptr;
  const float* teX = nullptr;
  const int32_t* teY = nullptr;
  std::vector<float> lr, dens;
  std::vector<uint32_t> thresh;
  int expected_epoch = 0;   // next epoch that may be started
  int open_epoch = -1;      // epoch in progress (-1: none)
  int last_epoch = -1;      // epoch whose loss the accumulators hold
  uint32_t next_step = 0;
  int64_t rows_done = 0;
  std::vector<uint32_t> perm_host[2];
  hipEvent_t perm_ev[2] = {nullptr, nullptr};
  bool perm_ev_used[2] = {false, false};
  hipEvent_t ev0 = nullptr, ev1 = nullptr;
  bool timing_pending = false;
  double last_s = 0.0;
  bool predicted = false;
  bool has_base = false;    // initial weights come from the caller's base model
  bool gscale_on = false;   // output gradients scaled per element (gevo_pop_set_grad_scale)
  bool ragged = false;      // some variant's hidden layer is narrowed (GEVO_EDIT_WIDTH): skip removed unit tiles
  // fused training keeps W1 in its own register image: which copy is current
  bool img_valid = false;   // the image (and the block-major mask) match the k-blocked master
  bool blk_stale = false;   // training has advanced the image past the k-blocked master
  bool wbf_valid = false;   // the bf16 weight copies of the prediction GEMM match the masters
  // kernel-level timing (gevo_pop_set_profiling)
  bool prof_on = false;
  struct ProfRec { int kind; hipEvent_t a, b; };
  std::vector<ProfRec> prof_pending;
  std::vector<hipEvent_t> ev_free, ev_all;
  double prof_ms[GEVO_KERNEL_KINDS] = {0};
  uint64_t prof_n[GEVO_KERNEL_KINDS] = {0};
};

namespace {

template <typename T>
T* at(gevo_pop* p, size_t off) { return reinterpret_cast<T*>(p->ws + off); }

constexpr size_t kProfBatch = 4096;   // launches between resolutions of pending timings

hipEvent_t take_event(gevo_pop* p) {
  if (!p->ev_free.empty()) {
    hipEvent_t e = p->ev_free.back();
    p->ev_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  p->ev_all.push_back(e);
  return e;
}

hipError_t prof_resolve(gevo_pop* p) {
  if (p->prof_pending.empty()) return hipSuccess;
  hipError_t err = hipStreamSynchronize(p->stream);
  if (err != hipSuccess) return err;
  for (const auto& r : p->prof_pending) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      p->prof_ms[r.kind] += (double)ms;
      p->prof_n[r.kind] += 1;
    }
    p->ev_free.push_back(r.a);
    p->ev_free.push_back(r.b);
  }
  p->prof_pending.clear();
  return hipSuccess;
}

// events recorded by the dispatch of the next launch of this kind (none when profiling is off)
LaunchEv prof(gevo_pop* p, int kind) {
  LaunchEv ev;
  if (!p->prof_on) return ev;
  if (p->prof_pending.size() >= kProfBatch && prof_resolve(p) != hipSuccess) return ev;
  ev.start = take_event(p);
  ev.stop = take_event(p);
  if (!ev.start || !ev.stop) {
    if (ev.start) p->ev_free.push_back(ev.start);
    if (ev.stop) p->ev_free.push_back(ev.stop);
    return LaunchEv{};
  }
  p->prof_pending.push_back({kind, ev.start, ev.stop});
  return ev;
}

#define HIP_TRY(x)                              \
  do {                                          \
    if ((x) != hipSuccess) return GEVO_E_HIP;   \
  } while (0)

// forward of hidden layer l over the R rows of a training batch (layer 0
// reads arows0; deeper layers the previous layer's activations of buffer
// outsel), writing the activations of buffer outsel in both orientations
template <typename S>
gevo_status forward_layer(gevo_pop* p, int l, const S* arows0, size_t ar0_vs, int R, int outsel) {
  const Layout& y = p->y;
  const LayerLay& q = y.lay[l];
  LayerArgs<S> a{};
  a.Kp = q.Kp; a.Np = q.Np; a.Bp = y.Bp;
  a.Wm = at<float>(p, q.Wm); a.bias = at<float>(p, q.bias); a.mask = at<uint32_t>(p, q.mask); a.bmask = at<uint32_t>(p, q.bmask);
  a.lr = at<float>(p, y.lr);
  a.do_update = 0;
  a.do_forward = 1;
  a.R = R;
  if (l == 0) { a.Arows = arows0; a.ar_vs = ar0_vs; }
  else { a.Arows = at<S>(p, y.lay[l - 1].arows[outsel]); a.ar_vs = (size_t)y.Bp * y.lay[l - 1].Np; }
  a.Orows = at<S>(p, q.arows[outsel]); a.or_vs = (size_t)y.Bp * q.Np;
  a.Ocols = at<S>(p, q.acols[outsel]); a.oc_vs = (size_t)q.Np * y.Bp;
  if (q.Wt) a.Wt = at<S>(p, q.Wt);
  a.vtime = at<unsigned long long>(p, y.vtime);
  if (p->ragged) a.wout = at<uint32_t>(p, q.wout);
  if (a.Kp % kTile || a.Np % kTile || a.R % kTile || a.R <= 0) return GEVO_E_SHAPE;
  if constexpr (std::is_same<S, uint16_t>::value) {
    if (q.streamed) {
      a.Wimg = at<float>(p, q.wimg); a.mblk = at<uint32_t>(p, q.mblk);
      HIP_TRY(launch_stream_layer(a, y.P, p->stream, prof(p, GEVO_KERNEL_LAYER_FWD)));
      return GEVO_OK;
    }
  }
  HIP_TRY(launch_layer<S>(a, y.P, p->stream, prof(p, GEVO_KERNEL_LAYER_FWD)));
  return GEVO_OK;
}

template <typename S>
gevo_status forward_hidden(gevo_pop* p, const S* arows0, size_t ar0_vs, int R, int outsel) {
  for (int l = 0; l < p->y.L - 1; ++l) {
    gevo_status st = forward_layer<S>(p, l, arows0, ar0_vs, R, outsel);
    if (st != GEVO_OK) return st;
  }
  return GEVO_OK;
}

template <typename S>
gevo_status begin_epoch(gevo_pop* p, int e) {
  const Layout& y = p->y;
  const int slot = e & 1;
  if (p->perm_ev_used[slot]) HIP_TRY(hipEventSynchronize(p->perm_ev[slot]));
  std::vector<uint32_t>& ph = p->perm_host[slot];
  ph.resize((size_t)y.n_train);
  fisher_yates(p->cfg.seed, (uint32_t)e, (uint32_t)y.n_train, ph.data());
  HIP_TRY(hipMemcpyAsync(at<uint32_t>(p, y.perm), ph.data(), ph.size() * 4, hipMemcpyHostToDevice, p->stream));
  HIP_TRY(hipEventRecord(p->perm_ev[slot], p->stream));
  p->perm_ev_used[slot] = true;
  GatherArgs g{};
  g.X = p->trX; g.y = p->trY; g.perm = at<uint32_t>(p, y.perm); g.n = y.n_train;
  g.d0 = y.lay[0].K; g.Kp = y.lay[0].Kp; g.B = y.B; g.Bp = y.Bp; g.T = y.T;
  g.rows = p->ws + y.xrows; g.labels = at<int32_t>(p, y.yep);
  g.blocked = y.fused;                             // the fused kernel reads rows one column block at a time
  g.res_order = y.resident;
  HIP_TRY(launch_gather<S>(g, p->stream, prof(p, GEVO_KERNEL_GATHER)));
  TransposeArgs tr{};
  tr.src = p->ws + y.xrows; tr.dst = p->ws + y.xcols; tr.Kp = y.lay[0].Kp; tr.Bp = y.Bp; tr.T = y.T;
  tr.blocked = y.fused;
  tr.res_order = y.resident;
  HIP_TRY(launch_transpose<S>(tr, p->stream, prof(p, GEVO_KERNEL_GATHER)));
  HIP_TRY(launch_zero_bytes(p->ws + y.train_ce, (size_t)y.P * 8, p->stream, prof(p, GEVO_KERNEL_AUX)));
  HIP_TRY(launch_zero_bytes(p->ws + y.train_corr, (size_t)y.P * 8, p->stream, prof(p, GEVO_KERNEL_AUX)));
  // forward of step 0 for the hidden layers (the fused kernel does its own)
  if (y.L > 1 && !y.fused) {
    gevo_status st = forward_hidden<S>(p, at<S>(p, y.xrows), 0, y.Bp, 0);
    if (st != GEVO_OK) return st;
  }
  p->rows_done = 0;
  return GEVO_OK;
}

template <typename S>
gevo_status train_step(gevo_pop* p, int t) {
  const Layout& y = p->y;
  const int L = y.L;
  const int buf = t & 1, nb = buf ^ 1;
  const int64_t r0 = (int64_t)t * y.B;
  const int bt = (int)((y.n_train - r0) < y.B ? (y.n_train - r0) : y.B);
  const size_t e = y.elt;
  const size_t xstep_r = (size_t)y.Bp * y.lay[0].Kp, xstep_c = xstep_r;
  const S* xrows_t = reinterpret_cast<const S*>(p->ws + y.xrows) + (size_t)t * xstep_r;
  const S* xcols_t = reinterpret_cast<const S*>(p->ws + y.xcols) + (size_t)t * xstep_c;
  (void)e;
  // output layer: loss, gradient, W_L update, gradient of the last hidden layer
  {
    const LayerLay& q = y.lay[L - 1];
    OutArgs<S> a{};
    a.Kp = q.Kp; a.C = q.N; a.Bp = y.Bp;
    a.Wm = at<float>(p, q.Wm); a.bias = at<float>(p, q.bias); a.mask = at<uint32_t>(p, q.mask); a.bmask = at<uint32_t>(p, q.bmask);
    a.lr = at<float>(p, y.lr);
    a.train = 1;
    if (L == 1) {
      a.Arows = xrows_t; a.ar_vs = 0; a.Acols = xcols_t; a.ac_vs = 0;
    } else {
      const LayerLay& h = y.lay[L - 2];
      a.Arows = at<S>(p, h.arows[buf]); a.ar_vs = (size_t)y.Bp * h.Np;
      a.Acols = at<S>(p, h.acols[buf]); a.ac_vs = (size_t)h.Np * y.Bp;
      a.Gcols = at<S>(p, h.gcols); a.gc_vs = (size_t)h.Np * y.Bp;
      if (h.grows) { a.Grows = at<S>(p, h.grows); a.gr_vs = (size_t)y.Bp * h.Np; }
    }
    a.labels = at<int32_t>(p, y.yep) + (size_t)t * y.Bp;
    a.rows = y.Bp;
    a.scale = (float)(1.0 / (double)bt);
    a.gscale = p->gscale_on ? at<float>(p, y.gscale) : nullptr;
    a.ce_acc = at<double>(p, y.train_ce);
    a.correct_acc = at<unsigned long long>(p, y.train_corr);
    a.vtime = at<unsigned long long>(p, y.vtime);
    a.ogrd = at<S>(p, y.ogrd);
    a.opdb = at<float>(p, y.opdb);
    a.opce = at<double>(p, y.opce);
    a.opcorr = at<unsigned int>(p, y.opcorr);
    if (a.Kp % kTile || a.Bp % kTile) return GEVO_E_SHAPE;
    HIP_TRY(launch_out<S>(a, y.P, p->stream, prof(p, GEVO_KERNEL_OUT_TRAIN)));
  }
  // hidden backward GEMMs, top down (pre-update weights)
  for (int l = L - 2; l >= 1; --l) {          // layer index l (0-based) has a hidden layer below
    const LayerLay& q = y.lay[l];
    const LayerLay& h = y.lay[l - 1];
    BwdArgs<S> a{};
    a.Kp = q.Kp; a.Np = q.Np; a.Bp = y.Bp;
    a.Wt = at<S>(p, q.Wt);
    a.Grows = at<S>(p, q.grows); a.gr_vs = (size_t)y.Bp * q.Np;
    a.Acols = at<S>(p, h.acols[buf]); a.ac_vs = (size_t)h.Np * y.Bp;
    a.Gcols = at<S>(p, h.gcols); a.gc_vs = (size_t)h.Np * y.Bp;
    if (h.grows) { a.Grows_out = at<S>(p, h.grows); a.go_vs = (size_t)y.Bp * h.Np; }
    a.vtime = at<unsigned long long>(p, y.vtime);
    if (a.Kp % kTile || a.Np % kTile || a.Bp % kTile || a.Kp != h.Np) return GEVO_E_SHAPE;
    if constexpr (std::is_same<S, uint16_t>::value) {
      if (bwd_gemm_supported(a.Kp, a.Np, a.Bp)) {
        HIP_TRY(launch_bwd_gemm(a, y.P, p->stream, prof(p, GEVO_KERNEL_BWD)));
        continue;
      }
    }
    HIP_TRY(launch_bwd<S>(a, y.P, p->stream, prof(p, GEVO_KERNEL_BWD)));
  }
  // hidden layers bottom up: update, then the forward of step t+1
  const bool fwd = t + 1 < y.T;
  for (int l = 0; l < L - 1; ++l) {
    const LayerLay& q = y.lay[l];
    LayerArgs<S> a{};
    a.Kp = q.Kp; a.Np = q.Np; a.Bp = y.Bp;
    a.Wm = at<float>(p, q.Wm); a.bias = at<float>(p, q.bias); a.mask = at<uint32_t>(p, q.mask); a.bmask = at<uint32_t>(p, q.bmask);
    a.lr = at<float>(p, y.lrh) + (size_t)l * y.P;   // 0 for the variants that removed this layer
    a.do_update = 1;
    a.Gcols = at<S>(p, q.gcols); a.g_vs = (size_t)q.Np * y.Bp;
    if (l == 0) { a.Acols = xcols_t; a.ac_vs = 0; }
    else { a.Acols = at<S>(p, y.lay[l - 1].acols[buf]); a.ac_vs = (size_t)y.lay[l - 1].Np * y.Bp; }
    a.do_forward = fwd ? 1 : 0;
    a.R = y.Bp;
    if (fwd) {
      if (l == 0) { a.Arows = xrows_t + xstep_r; a.ar_vs = 0; }
      else { a.Arows = at<S>(p, y.lay[l - 1].arows[nb]); a.ar_vs = (size_t)y.Bp * y.lay[l - 1].Np; }
      a.Orows = at<S>(p, q.arows[nb]); a.or_vs = (size_t)y.Bp * q.Np;
      a.Ocols = at<S>(p, q.acols[nb]); a.oc_vs = (size_t)q.Np * y.Bp;
    }
    if (q.Wt) a.Wt = at<S>(p, q.Wt);
    a.vtime = at<unsigned long long>(p, y.vtime);
    if (p->ragged) a.wout = at<uint32_t>(p, q.wout);
    if (a.Kp % kTile || a.Np % kTile || a.Bp % kTile || a.Bp > kPassRows) return GEVO_E_SHAPE;
    if constexpr (std::is_same<S, uint16_t>::value) {
      if (q.streamed) {
        a.Wimg = at<float>(p, q.wimg); a.mblk = at<uint32_t>(p, q.mblk);
        HIP_TRY(launch_stream_layer(a, y.P, p->stream, prof(p, GEVO_KERNEL_LAYER_TRAIN)));
        continue;
      }
    }
    HIP_TRY(launch_layer<S>(a, y.P, p->stream, prof(p, GEVO_KERNEL_LAYER_TRAIN)));
  }
  p->rows_done += bt;
  return GEVO_OK;
}

// The fused training kernel and the streaming hidden-layer kernel read and
// write register-image copies of their masters (with block-major mask words);
// every other consumer reads the k-blocked master.  These bring the copy that
// is about to be read up to date.
gevo_status sync_images(gevo_pop* p) {
  const Layout& y = p->y;
  if (!y.images || p->img_valid) return GEVO_OK;
  if (y.fused) {
    const LayerLay& q = y.lay[0];
    HIP_TRY(launch_w1_image(at<float>(p, q.Wm), at<float>(p, y.w1img), y.P, q.Kp, q.Np, true, p->stream,
                            prof(p, GEVO_KERNEL_AUX)));
    HIP_TRY(launch_mask_block_major(at<uint32_t>(p, q.mask), at<uint32_t>(p, y.m1blk), y.P, q.Kp, q.Np, p->stream,
                                    prof(p, GEVO_KERNEL_AUX)));
  }
  for (int l = 0; l + 1 < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    if (!q.streamed) continue;
    HIP_TRY(launch_w1_image(at<float>(p, q.Wm), at<float>(p, q.wimg), y.P, q.Kp, q.Np, true, p->stream,
                            prof(p, GEVO_KERNEL_AUX)));
    HIP_TRY(launch_mask_block_major(at<uint32_t>(p, q.mask), at<uint32_t>(p, q.mblk), y.P, q.Kp, q.Np, p->stream,
                                    prof(p, GEVO_KERNEL_AUX)));
  }
  p->img_valid = true;
  return GEVO_OK;
}

gevo_status sync_masters(gevo_pop* p, bool profile = true) {
  const Layout& y = p->y;
  if (!y.images || !p->blk_stale) return GEVO_OK;
  if (y.fused) {
    const LayerLay& q = y.lay[0];
    HIP_TRY(launch_w1_image(at<float>(p, y.w1img), at<float>(p, q.Wm), y.P, q.Kp, q.Np, false, p->stream,
                            profile ? prof(p, GEVO_KERNEL_AUX) : LaunchEv{}));
  }
  for (int l = 0; l + 1 < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    if (!q.streamed) continue;
    HIP_TRY(launch_w1_image(at<float>(p, q.wimg), at<float>(p, q.Wm), y.P, q.Kp, q.Np, false, p->stream,
                            profile ? prof(p, GEVO_KERNEL_AUX) : LaunchEv{}));
  }
  p->blk_stale = false;
  return GEVO_OK;
}

template <typename S>
gevo_status do_train_steps(gevo_pop* p, uint32_t epoch, uint32_t s0, uint32_t s1) {
  const Layout& y = p->y;
  if (y.n_train == 0 || y.T == 0) return GEVO_E_ORDER;
  if (s0 > s1 || s1 > (uint32_t)y.T) return GEVO_E_ARG;
  bool begin = false;
  if (p->open_epoch < 0) {
    if (s0 != 0 || (int)epoch != p->expected_epoch) return GEVO_E_ORDER;
    begin = true;
  } else if ((int)epoch != p->open_epoch || s0 != p->next_step) {
    return GEVO_E_ORDER;
  }
  HIP_TRY(hipEventRecord(p->ev0, p->stream));
  p->wbf_valid = false;                             // the masters move on
  HIP_TRY(launch_zero_bytes(p->ws + y.vtime, (size_t)y.P * 8, p->stream, LaunchEv{}));
  {
    gevo_status sti = sync_images(p);               // before the first forward of an epoch
    if (sti != GEVO_OK) return sti;
  }
  if (begin) {
    gevo_status st = begin_epoch<S>(p, (int)epoch);
    if (st != GEVO_OK) return st;
    p->open_epoch = (int)epoch;
    p->last_epoch = (int)epoch;
    p->next_step = 0;
  }
  if (y.fused && s1 > s0) {
    Fused2Args f{};
    const LayerLay& q1 = y.lay[0];
    const LayerLay& q2 = y.lay[1];
    f.Kp = q1.Kp; f.Hp = q1.Np; f.C = q2.N; f.B = y.B; f.Bp = y.Bp; f.T = y.T;
    f.n = y.n_train; f.t0 = (int)s0; f.t1 = (int)s1;
    f.xrows = at<uint16_t>(p, y.xrows); f.xcols = at<uint16_t>(p, y.xcols); f.labels = at<int32_t>(p, y.yep);
    f.W1 = at<float>(p, y.w1img); f.b1 = at<float>(p, q1.bias); f.m1 = at<uint32_t>(p, y.m1blk);
    f.W2 = at<float>(p, q2.Wm); f.b2 = at<float>(p, q2.bias); f.m2 = at<uint32_t>(p, q2.mask);
    f.bm1 = at<uint32_t>(p, q1.bmask); f.bm2 = at<uint32_t>(p, q2.bmask);
    f.lr = at<float>(p, y.lrh);                   // hidden layer (0 where removed)
    f.lr2 = at<float>(p, y.lrh) + y.P;            // output layer
    f.gscale = p->gscale_on ? at<float>(p, y.gscale) : nullptr;
    f.ce_acc = at<double>(p, y.train_ce);
    f.correct_acc = at<unsigned long long>(p, y.train_corr);
    f.vtime = at<unsigned long long>(p, y.vtime);
    if (q2.Kp != q1.Np || q1.Kp % kTile || fused2_lds_bytes(f.Hp, f.Bp) == 0) return GEVO_E_SHAPE;
    if (y.resident) {
      const int maxp = res2_max_pairs();
      if (maxp < 1) return GEVO_E_UNSUPPORTED;
      Res2Args ra{};
      ra.f = f;
      ra.xbuf = at<unsigned long long>(p, y.xbuf);
      ra.err = at<unsigned int>(p, y.rerr);
      ra.P = y.P;
      const int pairs = y.P < maxp ? y.P : maxp;
      HIP_TRY(launch_zero_bytes(p->ws + y.xbuf, (size_t)pairs * 2 * 2 * kResXW * 8 + 0, p->stream, LaunchEv{}));
      HIP_TRY(launch_zero_bytes(p->ws + y.rerr, 4, p->stream, LaunchEv{}));
      HIP_TRY(launch_res2(ra, pairs, p->stream, prof(p, GEVO_KERNEL_FUSED_TRAIN)));
      uint32_t err = 0;
      HIP_TRY(hipMemcpyAsync(&err, p->ws + y.rerr, 4, hipMemcpyDeviceToHost, p->stream));
      HIP_TRY(hipStreamSynchronize(p->stream));
      if (err) return GEVO_E_HIP;                 // a half of a pair stopped waiting for its partner
    } else {
      HIP_TRY(launch_fused2(f, y.P, p->stream, prof(p, GEVO_KERNEL_FUSED_TRAIN)));
    }
    p->blk_stale = true;
    for (uint32_t t = s0; t < s1; ++t) {
      const int64_t r0 = (int64_t)t * y.B;
      p->rows_done += (y.n_train - r0) < y.B ? (y.n_train - r0) : y.B;
    }
  } else {
    for (uint32_t t = s0; t < s1; ++t) {
      gevo_status st = train_step<S>(p, (int)t);
      if (st != GEVO_OK) return st;
    }
    if (y.images && (begin || s1 > s0)) p->blk_stale = true;   // streamed layers moved on in their images
  }
  p->next_step = s1;
  if (s1 == (uint32_t)y.T) {
    p->open_epoch = -1;
    p->expected_epoch = (int)epoch + 1;
  }
  HIP_TRY(hipEventRecord(p->ev1, p->stream));
  p->timing_pending = true;
  return GEVO_OK;
}

// Scratch and variant range of one prediction pass: variants [v0, v0 + G);
// per hidden layer the chunk activations act[l] ([G][kPredictChunk][Np]
// operands) and the bf16 weight copy wbf[l] ([G][Np][Kp], null when the layer
// does not run on the prediction GEMM); the partial sums [G][n_chunks_test].
// gevo_pop_predict takes them from the workspace, gevo_pop_predict_noalloc
// from the library's static scratch, one group of variants at a time.
struct PredictBufs {
  int v0 = 0, G = 0;
  void* act[GEVO_MAX_LAYERS] = {};
  uint16_t* wbf[GEVO_MAX_LAYERS] = {};
  bool convert = true;             // write the bf16 weight copies first
  double* part_ce = nullptr;
  unsigned int* part_corr = nullptr;
  bool profile = true;             // per-kernel timing events (they may be created on first use)
};

LaunchEv pev(gevo_pop* p, const PredictBufs& b, int kind) { return b.profile ? prof(p, kind) : LaunchEv{}; }

// forward of hidden layer l of variants [v0, v0 + G) over R prediction rows
template <typename S>
gevo_status predict_layer(gevo_pop* p, const PredictBufs& b, int l, const S* arows, size_t ar_vs, int R) {
  const Layout& y = p->y;
  const LayerLay& q = y.lay[l];
  const size_t v0 = (size_t)b.v0;
  LayerArgs<S> a{};
  a.Kp = q.Kp; a.Np = q.Np; a.Bp = y.Bp;
  a.Wm = at<float>(p, q.Wm) + v0 * q.Np * q.Kp; a.bias = at<float>(p, q.bias) + v0 * q.Np;
  a.mask = at<uint32_t>(p, q.mask) + v0 * q.Np * (q.Kp / 32); a.bmask = at<uint32_t>(p, q.bmask) + v0 * (q.Np / 32);
  a.lr = at<float>(p, y.lr) + v0;
  a.do_update = 0;
  a.do_forward = 1;
  a.R = R;
  a.Arows = arows; a.ar_vs = ar_vs;
  a.Orows = static_cast<S*>(b.act[l]); a.or_vs = (size_t)kPredictChunk * q.Np;
  a.vtime = at<unsigned long long>(p, y.vtime) + v0;
  if (a.Kp % kTile || a.Np % kTile || a.R % kTile || a.R <= 0) return GEVO_E_SHAPE;
  if constexpr (std::is_same<S, uint16_t>::value) {
    if (b.wbf[l] && pred_gemm_supported(q.Kp, q.Np, R)) {
      PredGemmArgs g{};
      g.A = arows; g.a_vs = ar_vs; g.W = b.wbf[l]; g.bias = a.bias; g.O = a.Orows; g.o_vs = a.or_vs;
      g.Kp = q.Kp; g.Np = q.Np; g.R = R; g.P = b.G;
      g.vtime = a.vtime;
      HIP_TRY(launch_pred_gemm(g, p->stream, pev(p, b, GEVO_KERNEL_LAYER_FWD)));
      return GEVO_OK;
    }
    if (fwd_gemm_supported(a.Kp, a.Np, a.R)) {                 // plain per-variant GEMM, fp32 weights
      FwdGemmArgs g{};
      g.A = arows; g.a_vs = ar_vs; g.Wm = a.Wm; g.bias = a.bias; g.O = a.Orows; g.o_vs = a.or_vs;
      g.Kp = a.Kp; g.Np = a.Np; g.R = a.R; g.P = b.G;
      g.vtime = a.vtime;
      HIP_TRY(launch_fwd_gemm(g, p->stream, pev(p, b, GEVO_KERNEL_LAYER_FWD)));
      return GEVO_OK;
    }
  }
  HIP_TRY(launch_layer<S>(a, b.G, p->stream, pev(p, b, GEVO_KERNEL_LAYER_FWD)));
  return GEVO_OK;
}

// One pass over the test split for variants [v0, v0 + G): hidden layers per
// chunk (a last hidden layer of exactly one 256-unit tile on the prediction
// GEMM also runs the output layer), the output layer otherwise, then the
// per-variant sums of the chunks' partial sums into test_ce / test_corr.
template <typename S>
gevo_status predict_pass(gevo_pop* p, const PredictBufs& b) {
  const Layout& y = p->y;
  const size_t v0 = (size_t)b.v0;
  if constexpr (std::is_same<S, uint16_t>::value) {
    if (b.convert)
      for (int l = 0; l + 1 < y.L; ++l) {
        const LayerLay& q = y.lay[l];
        if (b.wbf[l])
          HIP_TRY(launch_wt_bf16(at<float>(p, q.Wm) + v0 * q.Np * q.Kp, b.wbf[l], b.G, q.Kp, q.Np, p->stream,
                                 pev(p, b, GEVO_KERNEL_WEIGHT_COPY)));
      }
  }
  const LayerLay& o = y.lay[y.L - 1];
  const size_t Kp1 = (size_t)y.lay[0].Kp;
  for (int c0 = 0; c0 < y.n_test_pad; c0 += kPredictChunk) {
    const int R = (y.n_test_pad - c0) < kPredictChunk ? (y.n_test_pad - c0) : kPredictChunk;
    const S* xr = reinterpret_cast<const S*>(p->ws + y.xte) + (size_t)c0 * Kp1;
    bool fused = false;
    for (int l = 0; l < y.L - 1; ++l) {
      const LayerLay& q = y.lay[l];
      const S* ain = l == 0 ? xr : static_cast<const S*>(b.act[l - 1]);
      const size_t a_vs = l == 0 ? 0 : (size_t)kPredictChunk * y.lay[l - 1].Np;
      if constexpr (std::is_same<S, uint16_t>::value) {
        if (b.wbf[l] && l == y.L - 2 && q.Np == 256 && o.Kp == 256 && pred_gemm_supported(q.Kp, q.Np, R)) {
          PredGemmArgs g{};                                      // last hidden layer, one tile wide
          g.A = ain; g.a_vs = a_vs; g.W = b.wbf[l]; g.bias = at<float>(p, q.bias) + v0 * q.Np;
          g.Kp = q.Kp; g.Np = q.Np; g.R = R; g.P = b.G;
          g.WL = at<float>(p, o.Wm) + v0 * 32 * o.Kp; g.bL = at<float>(p, o.bias) + v0 * 32; g.C = o.N;
          g.labels = at<int32_t>(p, y.yte) + c0;
          g.chunk0 = c0 / kOutRows; g.n_chunks_total = y.n_chunks_test;
          g.part_ce = b.part_ce; g.part_correct = b.part_corr;
          g.vtime = at<unsigned long long>(p, y.vtime) + v0;
          HIP_TRY(launch_pred_gemm(g, p->stream, pev(p, b, GEVO_KERNEL_FWD_OUT)));
          fused = true;
          continue;
        }
      }
      gevo_status st = predict_layer<S>(p, b, l, ain, a_vs, R);
      if (st != GEVO_OK) return st;
    }
    if (fused) continue;
    OutArgs<S> a{};
    a.Kp = o.Kp; a.C = o.N; a.Bp = y.Bp;
    a.Wm = at<float>(p, o.Wm) + v0 * 32 * o.Kp; a.bias = at<float>(p, o.bias) + v0 * 32;
    a.mask = at<uint32_t>(p, o.mask) + v0 * 32 * (o.Kp / 32); a.bmask = at<uint32_t>(p, o.bmask) + v0;
    a.lr = at<float>(p, y.lr) + v0;
    a.train = 0;
    if (y.L == 1) { a.Arows = xr; a.ar_vs = 0; }
    else { a.Arows = static_cast<const S*>(b.act[y.L - 2]); a.ar_vs = (size_t)kPredictChunk * y.lay[y.L - 2].Np; }
    a.labels = at<int32_t>(p, y.yte) + c0;
    a.rows = R;
    a.chunk0 = c0 / kOutRows;
    a.n_chunks_total = y.n_chunks_test;
    a.part_ce = b.part_ce;
    a.part_correct = b.part_corr;
    a.vtime = at<unsigned long long>(p, y.vtime) + v0;
    if (a.Kp % kTile || R % kOutRows) return GEVO_E_SHAPE;
    HIP_TRY(launch_out<S>(a, b.G, p->stream, pev(p, b, GEVO_KERNEL_OUT_PREDICT)));
  }
  HIP_TRY(launch_reduce_partials(b.part_ce, b.part_corr, b.G, y.n_chunks_test, at<double>(p, y.test_ce) + v0,
                                 at<unsigned long long>(p, y.test_corr) + v0, p->stream,
                                 pev(p, b, GEVO_KERNEL_AUX)));
  return GEVO_OK;
}

template <typename S>
gevo_status do_predict(gevo_pop* p) {
  const Layout& y = p->y;
  HIP_TRY(hipEventRecord(p->ev0, p->stream));
  HIP_TRY(launch_zero_bytes(p->ws + y.vtime, (size_t)y.P * 8, p->stream, LaunchEv{}));
  gevo_status stb = sync_masters(p);
  if (stb != GEVO_OK) return stb;
  PredictBufs b;
  b.v0 = 0;
  b.G = y.P;
  bool any_copy = false;
  for (int l = 0; l + 1 < y.L; ++l) {
    b.act[l] = p->ws + y.lay[l].prows;
    if (y.lay[l].pred) {
      b.wbf[l] = at<uint16_t>(p, y.lay[l].wbf);
      any_copy = true;
    }
  }
  b.convert = any_copy && !p->wbf_valid;               // bf16 weight copies, once per change of the masters
  b.part_ce = at<double>(p, y.part_ce);
  b.part_corr = at<unsigned int>(p, y.part_corr);
  gevo_status st = predict_pass<S>(p, b);
  if (st != GEVO_OK) return st;
  if (any_copy) p->wbf_valid = true;
  HIP_TRY(hipEventRecord(p->ev1, p->stream));
  p->timing_pending = true;
  p->predicted = true;
  return GEVO_OK;
}

// ---------------------------------------------------------------------------
// Static scratch of gevo_pop_predict_noalloc.  In host code `scratch` names a
// host-side stand-in, not device memory: its device address (one per GPU) is
// taken once per device with hipGetSymbolAddress and only that address is
// passed to kernels.
constexpr size_t kStaticScratchBytes = GEVO_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// device address of the current device's scratch (taken on its first use)
gevo_status static_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return GEVO_E_HIP;
  if (dev >= kMaxDevices) return GEVO_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return GEVO_E_HIP;
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return GEVO_OK;
}

// scratch bytes of a group of G variants: per hidden layer the chunk
// activations and (layers on the prediction GEMM) the bf16 weight copy, then
// the partial sums; every piece 256-byte aligned
size_t noalloc_bytes(const Layout& y, size_t G) {
  size_t n = 0;
  for (int l = 0; l + 1 < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    n += align_up(G * (size_t)kPredictChunk * q.Np * y.elt);
    if (q.pred) n += align_up(G * (size_t)q.Np * q.Kp * 2);
  }
  n += align_up(G * (size_t)y.n_chunks_test * 8) + align_up(G * (size_t)y.n_chunks_test * 4);
  return n;
}

template <typename S>
gevo_status do_predict_noalloc(gevo_pop* p) {
  const Layout& y = p->y;
  void* base = nullptr;
  gevo_status st = static_scratch(&base);
  if (st != GEVO_OK) return st;
  if (noalloc_bytes(y, 1) > kStaticScratchBytes) return GEVO_E_UNSUPPORTED;
  int gmax = 1;
  while (gmax < y.P && noalloc_bytes(y, (size_t)gmax * 2) <= kStaticScratchBytes) gmax *= 2;
  while (gmax < y.P && noalloc_bytes(y, (size_t)gmax + 1) <= kStaticScratchBytes) ++gmax;
  HIP_TRY(hipEventRecord(p->ev0, p->stream));
  HIP_TRY(launch_zero_bytes(p->ws + y.vtime, (size_t)y.P * 8, p->stream, LaunchEv{}));
  st = sync_masters(p, false);
  if (st != GEVO_OK) return st;
  // Groups run one after another on the stream and reuse the scratch; every
  // scratch byte a group reads was written earlier in that group (the
  // activations and weight copies by their producing kernels, each partial
  // sum by exactly one workgroup), so nothing needs clearing.
  for (int v0 = 0; v0 < y.P; v0 += gmax) {
    PredictBufs b;
    b.v0 = v0;
    b.G = std::min(gmax, y.P - v0);
    char* c = static_cast<char*>(base);
    size_t off = 0;
    auto take = [&](size_t bytes) { char* at_ = c + off; off += align_up(bytes); return at_; };
    for (int l = 0; l + 1 < y.L; ++l) {
      const LayerLay& q = y.lay[l];
      b.act[l] = take((size_t)b.G * kPredictChunk * q.Np * y.elt);
      if (q.pred) b.wbf[l] = reinterpret_cast<uint16_t*>(take((size_t)b.G * q.Np * q.Kp * 2));
    }
    b.part_ce = reinterpret_cast<double*>(take((size_t)b.G * y.n_chunks_test * 8));
    b.part_corr = reinterpret_cast<unsigned int*>(take((size_t)b.G * y.n_chunks_test * 4));
    if (off > kStaticScratchBytes) return GEVO_E_UNSUPPORTED;
    b.convert = true;
    b.profile = false;
    st = predict_pass<S>(p, b);
    if (st != GEVO_OK) return st;
  }
  HIP_TRY(hipEventRecord(p->ev1, p->stream));
  p->timing_pending = true;
  p->predicted = true;
  return GEVO_OK;
}

gevo_status sync_timing(gevo_pop* p) {
  HIP_TRY(hipStreamSynchronize(p->stream));
  if (p->timing_pending) {
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, p->ev0, p->ev1));
    p->last_s = (double)ms * 1e-3;
    p->timing_pending = false;
  }
  return GEVO_OK;
}

}  // namespace

extern "C" {

gevo_status gevo_pop_workspace_bytes(const gevo_pop_config* cfg, size_t* bytes) {
  if (!bytes) return GEVO_E_ARG;
  Layout y;
  gevo_status st = make_layout(cfg, &y);
  if (st != GEVO_OK) return st;
  *bytes = y.total;
  return GEVO_OK;
}

gevo_status gevo_epoch_permutation(uint64_t seed, uint32_t epoch, uint32_t n, uint32_t* out) {
  if (!out && n > 0) return GEVO_E_ARG;
  fisher_yates(seed, epoch, n, out);
  return GEVO_OK;
}

gevo_status gevo_check_bf16_rounding(void* hip_stream, uint64_t* d_counts) {
  if (!d_counts || ((uintptr_t)d_counts % 8) != 0) return GEVO_E_ARG;
  const hipStream_t s = static_cast<hipStream_t>(hip_stream);
  HIP_TRY(hipMemsetAsync(d_counts, 0, 2 * sizeof(uint64_t), s));
  HIP_TRY(launch_bf16_check(reinterpret_cast<unsigned long long*>(d_counts), s));
  HIP_TRY(hipStreamSynchronize(s));
  return GEVO_OK;
}

// weights, biases and masks of every layer from the seed (and the caller's
// base model, when given); genomes: masks from the pruning-edit lists
// bias masks of every layer: unit n of variant v trains its bias when n < N
// and, with structural edits (width[v][l], bias_keep[v][l-1]), n < the
// layer's width and its bias is kept.  Synchronous upload.
static gevo_status upload_bias_masks(gevo_pop* p, const std::vector<uint32_t>* width,
                                     const std::vector<uint32_t>* bias_keep) {
  const Layout& y = p->y;
  for (int l = 0; l < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    const int words = q.Np / 32;
    std::vector<uint32_t> bits((size_t)y.P * words, 0u);
    for (int v = 0; v < y.P; ++v) {
      int keep_n = q.N;
      if (width) keep_n = std::min<int>(keep_n, (int)(*width)[(size_t)v * (y.L + 1) + l + 1]);
      if (bias_keep && !(*bias_keep)[(size_t)v * y.L + l]) keep_n = 0;
      for (int n = 0; n < keep_n; ++n) bits[(size_t)v * words + n / 32] |= 1u << (n % 32);
    }
    HIP_TRY(hipMemcpy(p->ws + q.bmask, bits.data(), bits.size() * 4, hipMemcpyHostToDevice));
  }
  return GEVO_OK;
}

static gevo_status init_layers(gevo_pop* p, bool genomes) {
  const Layout& y = p->y;
  const gevo_pop_config* cfg = &p->cfg;
  for (int l = 0; l < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    InitArgs a{};
    a.P = y.P; a.l_index = l; a.K = q.K; a.N = q.N; a.Kp = q.Kp; a.Np = q.Np;
    a.seed = cfg->seed;
    a.init_kind = cfg->init == GEVO_INIT_BASE_NOISE ? 1 : 0;
    a.xavier_a = (float)sqrt(6.0 / ((double)q.K + (double)q.N));
    a.noise_std = cfg->noise_rel_std;
    if (p->has_base) {
      a.base_w = reinterpret_cast<const float*>(p->ws + q.base_w);
      a.base_b = reinterpret_cast<const float*>(p->ws + q.base_b);
    }
    a.thresh = reinterpret_cast<const uint32_t*>(p->ws + y.thresh);
    if (genomes) {
      a.prune_off = reinterpret_cast<const uint32_t*>(p->ws + y.prune_off);
      a.prune_id = reinterpret_cast<const uint32_t*>(p->ws + y.prune_id);
      a.prune_th = reinterpret_cast<const uint32_t*>(p->ws + y.prune_th);
      a.width_in = reinterpret_cast<const uint32_t*>(p->ws + q.win);
      a.width_out = reinterpret_cast<const uint32_t*>(p->ws + q.wout);
      a.bias_keep = reinterpret_cast<const uint32_t*>(p->ws + q.bkeep);
      a.ident = reinterpret_cast<const uint32_t*>(p->ws + q.ident);
    }
    a.Wm = reinterpret_cast<float*>(p->ws + q.Wm);
    a.bias = reinterpret_cast<float*>(p->ws + q.bias);
    a.mask = reinterpret_cast<uint32_t*>(p->ws + q.mask);
    if (q.Kp % kTile || q.Np % kTile) return GEVO_E_SHAPE;
    if (launch_init(a, p->stream, LaunchEv{}) != hipSuccess) return GEVO_E_HIP;
  }
  return GEVO_OK;
}

gevo_status gevo_pop_init(const gevo_pop_config* cfg, void* d_ws, size_t ws_bytes, const float* d_train_x,
                          const int32_t* d_train_y, const float* d_test_x, const int32_t* d_test_y,
                          void* hip_stream, gevo_pop** out) {
  if (!out) return GEVO_E_ARG;
  *out = nullptr;
  Layout y;
  gevo_status st = make_layout(cfg, &y);
  if (st != GEVO_OK) return st;
  if (!d_ws || ((uintptr_t)d_ws % kAlign) != 0 || ws_bytes < y.total) return GEVO_E_WORKSPACE;
  if (!d_test_x || !d_test_y) return GEVO_E_ARG;
  if (y.n_train > 0 && (!d_train_x || !d_train_y)) return GEVO_E_ARG;
  gevo_pop* p = new (std::nothrow) gevo_pop();
  if (!p) return GEVO_E_ARG;
  p->cfg = *cfg;
  if (cfg->n_dens_list > 0) p->dens_list.assign(cfg->dens_list, cfg->dens_list + cfg->n_dens_list);
  p->cfg.dens_list = nullptr;
  p->cfg.base_params = nullptr;
  p->y = y;
  p->ws = reinterpret_cast<char*>(d_ws);
  p->stream = reinterpret_cast<hipStream_t>(hip_stream);
  p->trX = d_train_x; p->trY = d_train_y; p->teX = d_test_x; p->teY = d_test_y;
  auto fail = [&](gevo_status s) { gevo_pop_destroy(p); return s; };
  {
    void* scr = nullptr;                         // the no-allocation prediction's scratch on this device
    if (static_scratch(&scr) != GEVO_OK) return fail(GEVO_E_HIP);
  }
  if (hipEventCreate(&p->ev0) != hipSuccess || hipEventCreate(&p->ev1) != hipSuccess ||
      hipEventCreateWithFlags(&p->perm_ev[0], hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&p->perm_ev[1], hipEventDisableTiming) != hipSuccess)
    return fail(GEVO_E_HIP);
  // per-variant learning rate, density and mask threshold (host, fp64)
  const int P = y.P;
  p->lr.resize(P); p->dens.resize(P); p->thresh.resize(P);
  for (int v = 0; v < P; ++v) {
    if (cfg->lr_lo == cfg->lr_hi) {
      p->lr[v] = cfg->lr_lo;
    } else {
      const double u = (double)(draw_word(cfg->seed, 0, 0, (uint32_t)v, kStreamLr, 0) >> 8) * (1.0 / 16777216.0);
      const double lo = log((double)cfg->lr_lo), hi = log((double)cfg->lr_hi);
      p->lr[v] = (float)exp(lo + u * (hi - lo));
    }
    float rho;
    if (!p->dens_list.empty()) {
      rho = p->dens_list[(size_t)v % p->dens_list.size()];
    } else {
      const double u = (double)(draw_word(cfg->seed, 0, 0, (uint32_t)v, kStreamDens, 0) >> 8) * (1.0 / 16777216.0);
      rho = (float)((double)cfg->dens_lo + u * ((double)cfg->dens_hi - (double)cfg->dens_lo));
    }
    p->dens[v] = rho;
    double t = floor((double)rho * 16777216.0 + 0.5);
    if (t < 0.0) t = 0.0;
    if (t > 16777216.0) t = 16777216.0;
    p->thresh[v] = (uint32_t)t;
  }
  hipStream_t s = p->stream;
  if (hipMemcpyAsync(p->ws + y.lr, p->lr.data(), (size_t)P * 4, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipMemcpyAsync(p->ws + y.thresh, p->thresh.data(), (size_t)P * 4, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(GEVO_E_HIP);
  for (int l = 0; l < y.L; ++l)                  // every layer trains at the variant's rate
    if (hipMemcpyAsync(p->ws + y.lrh + (size_t)l * P * 4, p->lr.data(), (size_t)P * 4, hipMemcpyHostToDevice, s) !=
        hipSuccess)
      return fail(GEVO_E_HIP);
  // optional base model, padded and transposed to the device layout
  std::vector<std::vector<float>> base_w(y.L), base_b(y.L);
  if (cfg->init == GEVO_INIT_BASE_NOISE && cfg->base_params) {
    size_t off = 0;
    for (int l = 0; l < y.L; ++l) {
      const LayerLay& q = y.lay[l];
      base_w[l].assign((size_t)q.Np * q.Kp, 0.0f);
      base_b[l].assign((size_t)q.Np, 0.0f);
      for (int k = 0; k < q.K; ++k)
        for (int n = 0; n < q.N; ++n) base_w[l][(size_t)n * q.Kp + k] = cfg->base_params[off + (size_t)k * q.N + n];
      off += (size_t)q.K * q.N;
      for (int n = 0; n < q.N; ++n) base_b[l][n] = cfg->base_params[off + n];
      off += (size_t)q.N;
      if (hipMemcpy(p->ws + q.base_w, base_w[l].data(), base_w[l].size() * 4, hipMemcpyHostToDevice) != hipSuccess ||
          hipMemcpy(p->ws + q.base_b, base_b[l].data(), base_b[l].size() * 4, hipMemcpyHostToDevice) != hipSuccess)
        return fail(GEVO_E_HIP);
    }
  }
  p->has_base = cfg->init == GEVO_INIT_BASE_NOISE && cfg->base_params;
  {
    gevo_status st = upload_bias_masks(p, nullptr, nullptr);
    if (st == GEVO_OK) st = init_layers(p, false);
    if (st != GEVO_OK) return fail(st);
  }
  // test split converted once to the operand type, padded to whole chunks
  GatherArgs g{};
  g.X = d_test_x; g.y = d_test_y; g.perm = nullptr; g.n = y.n_test;
  g.d0 = y.lay[0].K; g.Kp = y.lay[0].Kp; g.B = y.n_test_pad; g.Bp = y.n_test_pad; g.T = 1;
  g.rows = p->ws + y.xte; g.labels = reinterpret_cast<int32_t*>(p->ws + y.yte);
  hipError_t e = cfg->dtype == GEVO_BF16 ? launch_gather<uint16_t>(g, s, LaunchEv{}) : launch_gather<float>(g, s, LaunchEv{});
  if (e != hipSuccess) return fail(GEVO_E_HIP);
  if (launch_zero_bytes(p->ws + y.vtime, (size_t)P * 8, s, LaunchEv{}) != hipSuccess ||
      launch_zero_bytes(p->ws + y.train_ce, (size_t)P * 8, s, LaunchEv{}) != hipSuccess ||
      launch_zero_bytes(p->ws + y.train_corr, (size_t)P * 8, s, LaunchEv{}) != hipSuccess ||
      launch_zero_bytes(p->ws + y.test_ce, (size_t)P * 8, s, LaunchEv{}) != hipSuccess ||
      launch_zero_bytes(p->ws + y.test_corr, (size_t)P * 8, s, LaunchEv{}) != hipSuccess)
    return fail(GEVO_E_HIP);
  if (cfg->init == GEVO_INIT_BASE_NOISE && cfg->base_params) {
    if (hipStreamSynchronize(s) != hipSuccess) return fail(GEVO_E_HIP);   // host staging vectors die here
  }
  *out = p;
  return GEVO_OK;
}

gevo_status gevo_pop_set_genomes(gevo_pop* p, float lr_base, const uint32_t* offsets, const gevo_edit* edits,
                                 float* lr_out, double* density_out) {
  if (!p || !offsets || offsets[0] != 0) return GEVO_E_ARG;
  if (p->open_epoch >= 0) return GEVO_E_ORDER;
  const Layout& y = p->y;
  const int P = y.P;
  for (int v = 0; v < P; ++v)
    if (offsets[v + 1] < offsets[v]) return GEVO_E_ARG;
  if (offsets[P] > 0 && !edits) return GEVO_E_ARG;
  const int L = y.L;
  std::vector<float> lr(P);
  std::vector<double> dens(P);
  std::vector<uint32_t> off(P + 1, 0), ids, th;
  std::vector<uint32_t> width((size_t)P * (L + 1)), bkeep((size_t)P * L, 1u), gone((size_t)P * L, 0u);
  double total_w = 0.0;
  for (int l = 1; l <= L; ++l) total_w += (double)y.lay[l - 1].K * (double)y.lay[l - 1].N;
  for (int v = 0; v < P; ++v) {
    float r = lr_base;
    double d = 1.0;
    uint32_t np = 0;
    uint32_t* wv = width.data() + (size_t)v * (L + 1);
    wv[0] = (uint32_t)y.lay[0].K;
    for (int l = 1; l <= L; ++l) wv[l] = (uint32_t)y.lay[l - 1].N;
    for (uint32_t i = offsets[v]; i < offsets[v + 1]; ++i) {
      const gevo_edit& e = edits[i];
      if (e.kind == GEVO_EDIT_LR) {
        float f;
        memcpy(&f, &e.value, 4);
        r = r * f;                               // binary32 product, in order
      } else if (e.kind == GEVO_EDIT_PRUNE) {
        if (e.value > (1u << 24) || ++np > kMaxGenomePrunes) return GEVO_E_ARG;
        ids.push_back(e.id);
        th.push_back(e.value);
        d = d * ((double)e.value / 16777216.0);
      } else if (e.kind == GEVO_EDIT_WIDTH) {
        if (e.id < 1 || (int)e.id > L - 1 || e.value == 0) return GEVO_E_ARG;
        wv[e.id] = std::min(wv[e.id], e.value);
      } else if (e.kind == GEVO_EDIT_BIAS_OFF) {
        if (e.id < 1 || (int)e.id > L) return GEVO_E_ARG;
        bkeep[(size_t)v * L + e.id - 1] = 0u;
      } else if (e.kind == GEVO_EDIT_LAYER_OFF) {
        if (e.id < 1 || (int)e.id > L - 1) return GEVO_E_ARG;
        gone[(size_t)v * L + e.id - 1] = 1u;
      } else {
        return GEVO_E_ARG;
      }
    }
    double kept_w = 0.0;
    for (int l = 1; l <= L; ++l)
      if (!gone[(size_t)v * L + l - 1]) kept_w += (double)wv[l - 1] * (double)wv[l];
    for (int l = 1; l < L; ++l)                  // a removed layer keeps its identity biases
      if (gone[(size_t)v * L + l - 1]) bkeep[(size_t)v * L + l - 1] = 1u;
    d = d * (kept_w / total_w);
    if (!(r > 0.0f) || !std::isfinite(r)) return GEVO_E_ARG;
    lr[v] = r;
    dens[v] = d;
    off[v + 1] = (uint32_t)ids.size();
  }
  hipStream_t s = p->stream;
  HIP_TRY(hipStreamSynchronize(s));              // nothing may still read the state being replaced
  HIP_TRY(hipMemcpy(p->ws + y.lr, lr.data(), (size_t)P * 4, hipMemcpyHostToDevice));
  for (int l = 0; l < L; ++l) {                  // per-layer rates: 0 for a removed (frozen) layer
    std::vector<float> lrl(P);
    for (int v = 0; v < P; ++v) lrl[v] = gone[(size_t)v * L + l] ? 0.0f : lr[v];
    HIP_TRY(hipMemcpy(p->ws + y.lrh + (size_t)l * P * 4, lrl.data(), (size_t)P * 4, hipMemcpyHostToDevice));
  }
  HIP_TRY(hipMemcpy(p->ws + y.prune_off, off.data(), off.size() * 4, hipMemcpyHostToDevice));
  if (!ids.empty()) {
    HIP_TRY(hipMemcpy(p->ws + y.prune_id, ids.data(), ids.size() * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p->ws + y.prune_th, th.data(), th.size() * 4, hipMemcpyHostToDevice));
  }
  for (int l = 0; l < L; ++l) {                  // per-layer structural arrays of the init kernel
    std::vector<uint32_t> win(P), wout(P), bk(P), id(P);
    for (int v = 0; v < P; ++v) {
      win[v] = width[(size_t)v * (L + 1) + l];
      wout[v] = width[(size_t)v * (L + 1) + l + 1];
      bk[v] = bkeep[(size_t)v * L + l];
      id[v] = gone[(size_t)v * L + l];
    }
    HIP_TRY(hipMemcpy(p->ws + y.lay[l].ident, id.data(), (size_t)P * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p->ws + y.lay[l].win, win.data(), (size_t)P * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p->ws + y.lay[l].wout, wout.data(), (size_t)P * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p->ws + y.lay[l].bkeep, bk.data(), (size_t)P * 4, hipMemcpyHostToDevice));
  }
  {
    const gevo_status sb = upload_bias_masks(p, &width, &bkeep);
    if (sb != GEVO_OK) return sb;
  }
  const gevo_status st = init_layers(p, true);
  if (st != GEVO_OK) return st;
  // Narrowed hidden layers: training skips the workgroups of removed unit
  // tiles, which then never write their activation, gradient and operand-copy
  // slots, so those buffers start from zeros.
  bool narrowed = false;
  for (int v = 0; v < P; ++v)
    for (int l = 1; l < L; ++l) narrowed = narrowed || width[(size_t)v * (L + 1) + l] < (uint32_t)y.lay[l - 1].N;
  p->ragged = narrowed;
  if (narrowed)
    for (int l = 0; l + 1 < L; ++l) {
      const LayerLay& q = y.lay[l];
      const size_t act = (size_t)P * y.Bp * q.Np * y.elt;
      for (int bsel = 0; bsel < 2; ++bsel) {
        HIP_TRY(launch_zero_bytes(p->ws + q.arows[bsel], act, s, LaunchEv{}));
        HIP_TRY(launch_zero_bytes(p->ws + q.acols[bsel], act, s, LaunchEv{}));
      }
      HIP_TRY(launch_zero_bytes(p->ws + q.gcols, act, s, LaunchEv{}));
      if (q.grows) HIP_TRY(launch_zero_bytes(p->ws + q.grows, act, s, LaunchEv{}));
      if (q.Wt) HIP_TRY(launch_zero_bytes(p->ws + q.Wt, (size_t)P * q.Kp * q.Np * y.elt, s, LaunchEv{}));
    }
  HIP_TRY(launch_zero_bytes(p->ws + y.train_ce, (size_t)P * 8, s, LaunchEv{}));
  HIP_TRY(launch_zero_bytes(p->ws + y.train_corr, (size_t)P * 8, s, LaunchEv{}));
  HIP_TRY(launch_zero_bytes(p->ws + y.test_ce, (size_t)P * 8, s, LaunchEv{}));
  HIP_TRY(launch_zero_bytes(p->ws + y.test_corr, (size_t)P * 8, s, LaunchEv{}));
  HIP_TRY(hipStreamSynchronize(s));
  for (int v = 0; v < P; ++v) {
    p->lr[v] = lr[v];
    p->dens[v] = (float)dens[v];
    p->thresh[v] = 0;
    if (lr_out) lr_out[v] = lr[v];
    if (density_out) density_out[v] = dens[v];
  }
  p->expected_epoch = 0;
  p->open_epoch = -1;
  p->last_epoch = -1;
  p->next_step = 0;
  p->rows_done = 0;
  p->predicted = false;
  p->timing_pending = false;
  p->img_valid = false;                          // the register-image copies are stale
  p->wbf_valid = false;
  p->blk_stale = false;
  return GEVO_OK;
}

gevo_status gevo_pop_set_grad_scale(gevo_pop* p, const float* scale) {
  if (!p) return GEVO_E_ARG;
  if (p->open_epoch >= 0) return GEVO_E_ORDER;
  if (!scale) {
    p->gscale_on = false;
    return GEVO_OK;
  }
  const Layout& y = p->y;
  const int C = y.lay[y.L - 1].N;
  const size_t n = (size_t)y.P * y.B * C;
  for (size_t i = 0; i < n; ++i)
    if (!std::isfinite(scale[i])) return GEVO_E_ARG;
  std::vector<float> dev((size_t)y.P * y.Bp * 32, 0.0f);
  for (int v = 0; v < y.P; ++v)
    for (int b = 0; b < y.B; ++b)
      for (int c = 0; c < C; ++c)
        dev[((size_t)v * y.Bp + b) * 32 + c] = scale[((size_t)v * y.B + b) * C + c];
  HIP_TRY(hipStreamSynchronize(p->stream));      // no step in flight may read the old scales
  HIP_TRY(hipMemcpy(p->ws + y.gscale, dev.data(), dev.size() * 4, hipMemcpyHostToDevice));
  p->gscale_on = true;
  return GEVO_OK;
}

gevo_status gevo_pop_train_steps(gevo_pop* p, uint32_t epoch, uint32_t s0, uint32_t s1) {
  if (!p) return GEVO_E_ARG;
  return p->cfg.dtype == GEVO_BF16 ? do_train_steps<uint16_t>(p, epoch, s0, s1)
                                   : do_train_steps<float>(p, epoch, s0, s1);
}

gevo_status gevo_pop_train_epoch(gevo_pop* p, uint32_t epoch) {
  if (!p) return GEVO_E_ARG;
  if (p->y.n_train == 0) return GEVO_E_ORDER;
  return gevo_pop_train_steps(p, epoch, 0, (uint32_t)p->y.T);
}

gevo_status gevo_pop_steps_per_epoch(const gevo_pop* p, uint32_t* steps) {
  if (!p || !steps) return GEVO_E_ARG;
  *steps = (uint32_t)p->y.T;
  return GEVO_OK;
}

gevo_status gevo_pop_predict(gevo_pop* p) {
  if (!p) return GEVO_E_ARG;
  return p->cfg.dtype == GEVO_BF16 ? do_predict<uint16_t>(p) : do_predict<float>(p);
}

gevo_status gevo_pop_predict_noalloc(gevo_pop* p) {
  if (!p) return GEVO_E_ARG;
  return p->cfg.dtype == GEVO_BF16 ? do_predict_noalloc<uint16_t>(p) : do_predict_noalloc<float>(p);
}

gevo_status gevo_pop_scores(gevo_pop* p, float* train_loss, float* train_acc, float* test_loss, float* test_acc,
                            float* time_s) {
  if (!p) return GEVO_E_ARG;
  gevo_status st = sync_timing(p);
  if (st != GEVO_OK) return st;
  const Layout& y = p->y;
  const int P = y.P;
  std::vector<double> tce(P), sce(P);
  std::vector<unsigned long long> tc(P), sc(P);
  HIP_TRY(hipMemcpy(tce.data(), p->ws + y.train_ce, (size_t)P * 8, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(tc.data(), p->ws + y.train_corr, (size_t)P * 8, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(sce.data(), p->ws + y.test_ce, (size_t)P * 8, hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(sc.data(), p->ws + y.test_corr, (size_t)P * 8, hipMemcpyDeviceToHost));
  std::vector<unsigned long long> vt(P);
  HIP_TRY(hipMemcpy(vt.data(), p->ws + y.vtime, (size_t)P * 8, hipMemcpyDeviceToHost));
  double vt_sum = 0.0;
  for (int v = 0; v < P; ++v) vt_sum += (double)vt[v];
  const bool trained = p->last_epoch >= 0 && p->rows_done > 0;
  for (int v = 0; v < P; ++v) {
    if (train_loss) train_loss[v] = trained ? (float)(tce[v] / (double)p->rows_done) : NAN;
    if (train_acc) train_acc[v] = trained ? (float)((double)tc[v] / (double)p->rows_done) : NAN;
    if (test_loss) test_loss[v] = p->predicted ? (float)(sce[v] / (double)y.n_test) : NAN;
    if (test_acc) test_acc[v] = p->predicted ? (float)((double)sc[v] / (double)y.n_test) : NAN;
    // the call's wall time split in proportion to each variant's device time
    // (equal shares when no per-variant kernel ran)
    if (time_s) time_s[v] = (float)(vt_sum > 0.0 ? p->last_s * ((double)vt[v] / vt_sum) : p->last_s / (double)P);
  }
  return GEVO_OK;
}

gevo_status gevo_pop_last_time(gevo_pop* p, double* seconds) {
  if (!p || !seconds) return GEVO_E_ARG;
  gevo_status st = sync_timing(p);
  if (st != GEVO_OK) return st;
  *seconds = p->last_s;
  return GEVO_OK;
}

gevo_status gevo_pop_export(gevo_pop* p, uint32_t v, float* params_out, uint8_t* mask_out, float* lr_out,
                            float* density_out) {
  if (!p) return GEVO_E_ARG;
  const Layout& y = p->y;
  if (v >= (uint32_t)y.P) return GEVO_E_ARG;
  gevo_status stb = sync_masters(p);
  if (stb != GEVO_OK) return stb;
  HIP_TRY(hipStreamSynchronize(p->stream));
  size_t off = 0, moff = 0;
  for (int l = 0; l < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    const size_t nw = (size_t)q.Np * q.Kp, words = (size_t)q.Np * (q.Kp / 32);
    std::vector<float> W(nw), b((size_t)q.Np);
    std::vector<uint32_t> M(words);
    HIP_TRY(hipMemcpy(W.data(), p->ws + q.Wm + (size_t)v * nw * 4, nw * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(b.data(), p->ws + q.bias + (size_t)v * q.Np * 4, (size_t)q.Np * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(M.data(), p->ws + q.mask + (size_t)v * words * 4, words * 4, hipMemcpyDeviceToHost));
    for (int k = 0; k < q.K; ++k)
      for (int n = 0; n < q.N; ++n) {
        if (params_out) params_out[off + (size_t)k * q.N + n] = W[((size_t)(k / 32) * q.Np + n) * 32 + k % 32];
        if (mask_out) mask_out[moff + (size_t)k * q.N + n] = (uint8_t)((M[(size_t)n * (q.Kp / 32) + k / 32] >> (k % 32)) & 1u);
      }
    off += (size_t)q.K * q.N;
    moff += (size_t)q.K * q.N;
    for (int n = 0; n < q.N; ++n)
      if (params_out) params_out[off + n] = b[n];
    off += (size_t)q.N;
  }
  if (lr_out) *lr_out = p->lr[v];
  if (density_out) *density_out = p->dens[v];
  return GEVO_OK;
}

gevo_status gevo_pop_import(gevo_pop* p, uint32_t v, const float* params) {
  if (!p || !params) return GEVO_E_ARG;
  const Layout& y = p->y;
  if (v >= (uint32_t)y.P) return GEVO_E_ARG;
  if (p->open_epoch >= 0) return GEVO_E_ORDER;        // only between epochs
  gevo_status stb = sync_masters(p);
  if (stb != GEVO_OK) return stb;
  HIP_TRY(hipStreamSynchronize(p->stream));
  p->img_valid = false;                               // the image is rebuilt from the imported master
  p->wbf_valid = false;
  size_t off = 0;
  for (int l = 0; l < y.L; ++l) {
    const LayerLay& q = y.lay[l];
    const size_t nw = (size_t)q.Np * q.Kp, words = (size_t)q.Np * (q.Kp / 32);
    std::vector<uint32_t> M(words);
    HIP_TRY(hipMemcpy(M.data(), p->ws + q.mask + (size_t)v * words * 4, words * 4, hipMemcpyDeviceToHost));
    std::vector<float> W(nw, 0.0f), b((size_t)q.Np, 0.0f);
    for (int k = 0; k < q.K; ++k)
      for (int n = 0; n < q.N; ++n) {
        const bool keep = (M[(size_t)n * (q.Kp / 32) + k / 32] >> (k % 32)) & 1u;
        W[((size_t)(k / 32) * q.Np + n) * 32 + k % 32] = keep ? params[off + (size_t)k * q.N + n] : 0.0f;
      }
    off += (size_t)q.K * q.N;
    for (int n = 0; n < q.N; ++n) b[n] = params[off + n];
    off += (size_t)q.N;
    HIP_TRY(hipMemcpy(p->ws + q.Wm + (size_t)v * nw * 4, W.data(), nw * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(p->ws + q.bias + (size_t)v * q.Np * 4, b.data(), (size_t)q.Np * 4, hipMemcpyHostToDevice));
  }
  return GEVO_OK;
}

gevo_status gevo_pop_epoch_labels(gevo_pop* p, int32_t* labels_out, int64_t n) {
  if (!p || !labels_out) return GEVO_E_ARG;
  const Layout& y = p->y;
  if (n != y.n_train) return GEVO_E_SHAPE;
  if (p->last_epoch < 0) return GEVO_E_ORDER;
  HIP_TRY(hipStreamSynchronize(p->stream));
  std::vector<int32_t> yep((size_t)y.T * y.Bp);
  HIP_TRY(hipMemcpy(yep.data(), p->ws + y.yep, yep.size() * 4, hipMemcpyDeviceToHost));
  for (int64_t r = 0; r < n; ++r) labels_out[r] = yep[(size_t)(r / y.B) * y.Bp + (size_t)(r % y.B)];
  return GEVO_OK;
}

gevo_status gevo_pop_set_profiling(gevo_pop* p, int enable) {
  if (!p) return GEVO_E_ARG;
  if (!enable && prof_resolve(p) != hipSuccess) return GEVO_E_HIP;
  p->prof_on = enable != 0;
  return GEVO_OK;
}

gevo_status gevo_pop_kernel_stats(gevo_pop* p, int kind, double* total_ms, uint64_t* launches) {
  if (!p || kind < 0 || kind >= GEVO_KERNEL_KINDS) return GEVO_E_ARG;
  if (prof_resolve(p) != hipSuccess) return GEVO_E_HIP;
  if (total_ms) *total_ms = p->prof_ms[kind];
  if (launches) *launches = p->prof_n[kind];
  return GEVO_OK;
}

void gevo_pop_destroy(gevo_pop* p) {
  if (!p) return;
  (void)hipStreamSynchronize(p->stream);   // pending copies may still read host buffers
  if (p->ev0) (void)hipEventDestroy(p->ev0);
  if (p->ev1) (void)hipEventDestroy(p->ev1);
  if (p->perm_ev[0]) (void)hipEventDestroy(p->perm_ev[0]);
  if (p->perm_ev[1]) (void)hipEventDestroy(p->perm_ev[1]);
  for (hipEvent_t e : p->ev_all) (void)hipEventDestroy(e);
  delete p;
}

const char* gevo_status_str(gevo_status s) {
  switch (s) {
    case GEVO_OK: return "ok";
    case GEVO_E_ARG: return "invalid argument";
    case GEVO_E_SHAPE: return "inconsistent shape";
    case GEVO_E_WORKSPACE: return "workspace too small or misaligned";
    case GEVO_E_ORDER: return "call out of order";
    case GEVO_E_HIP: return "HIP runtime error";
    case GEVO_E_UNSUPPORTED: return "unsupported configuration";
  }
  return "unknown status";
}

}  // extern "C"
