// Search step of GEVO-ML over patch-list genomes (host code, declared in
// include/gevo.h): NSGA-II ranking and crowding distance (Deb, Pratap,
// Agarwal, Meyarivan, IEEE TEC 2002), elitist selection with binary
// tournaments (paper section 4.4), the initial population with drawn edits
// (section 4) and breeding by one-point messy crossover (section 4.2) and
// mutation.  Every random choice is a Philox4x32-10 draw at the counter the
// header documents.
#include <math.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "gevo.h"
#include "gevo_internal.h"

namespace {

using gevo::kStreamCross;
using gevo::kStreamMut;
using gevo::kStreamSelect;

void draw4(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2, uint32_t stream, uint32_t out[4]) {
  const uint32_t ctr[4] = {c0, c1, c2, stream};
  const uint32_t key[2] = {(uint32_t)(seed & 0xffffffffu), (uint32_t)(seed >> 32)};
  gevo::philox4x32_10_host(ctr, key, out);
}

double u24(uint32_t r) { return (double)(r >> 8) * (1.0 / 16777216.0); }

uint32_t below(uint32_t r, uint64_t n) { return (uint32_t)(((uint64_t)r * n) >> 32); }

uint32_t float_bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

// a dominates b: no objective larger, one smaller (all minimised)
bool dominates(const double* a, const double* b, uint32_t m) {
  bool smaller = false;
  for (uint32_t k = 0; k < m; ++k) {
    if (a[k] > b[k]) return false;
    if (a[k] < b[k]) smaller = true;
  }
  return smaller;
}

// shape of the nets a drawn structural edit applies to
struct NetShape {
  uint32_t L = 0;
  const uint32_t* dims = nullptr;
};

// the edit drawn from (j, gen, i, mutation stream): with probability struct_p
// a structural edit (bias removal; with hidden layers, bias removal, a width
// of a hidden layer or a removed hidden layer with equal odds), otherwise a
// learning-rate factor log-uniform on [1/2, 2] or pruning at a density
// uniform on [rho_lo, 1], with equal odds
gevo_edit random_edit(uint64_t seed, uint32_t gen, uint32_t i, uint32_t j, uint32_t id, double rho_lo,
                      double struct_p, const NetShape& net) {
  uint32_t w[4];
  draw4(seed, j, gen, i, kStreamMut, w);
  const double u = u24(w[2]), uk = u24(w[1]);
  gevo_edit e{};
  if (uk < struct_p) {
    const double us = u24(w[3]);
    if (us < 1.0 / 3.0 || net.L < 2) {
      e.kind = GEVO_EDIT_BIAS_OFF;
      e.id = 1 + below(w[0], net.L);
      e.value = 0;
    } else if (us < 2.0 / 3.0) {
      e.kind = GEVO_EDIT_WIDTH;
      e.id = 1 + below(w[0], net.L - 1);
      e.value = 1 + below(w[2], net.dims[e.id]);
    } else {
      e.kind = GEVO_EDIT_LAYER_OFF;
      e.id = 1 + below(w[0], net.L - 1);
      e.value = 0;
    }
    return e;
  }
  e.id = id;
  if (uk < struct_p + (1.0 - struct_p) * 0.5) {
    e.kind = GEVO_EDIT_LR;
    e.value = float_bits((float)exp(log(0.5) + u * log(4.0)));
  } else {
    e.kind = GEVO_EDIT_PRUNE;
    e.value = (uint32_t)nearbyint((rho_lo + u * (1.0 - rho_lo)) * 16777216.0);   // round half to even
  }
  return e;
}

bool valid_shape(double struct_p, uint32_t n_layers, const uint32_t* dims, NetShape* net) {
  if (!(struct_p >= 0.0 && struct_p <= 1.0)) return false;
  if (struct_p == 0.0) return true;
  if (n_layers < 1 || !dims) return false;
  for (uint32_t l = 0; l <= n_layers; ++l)
    if (dims[l] == 0) return false;
  net->L = n_layers;
  net->dims = dims;
  return true;
}

bool valid_offsets(uint32_t n, const uint32_t* off) {
  if (!off || off[0] != 0) return false;
  for (uint32_t i = 0; i < n; ++i)
    if (off[i + 1] < off[i]) return false;
  return true;
}

}  // namespace

extern "C" {

gevo_status gevo_nsga2_rank(uint32_t n, uint32_t m, const double* objs, uint32_t* rank, double* crowding) {
  if (n == 0) return GEVO_OK;
  if (!objs || !rank || !crowding || m == 0) return GEVO_E_ARG;
  for (size_t i = 0; i < (size_t)n * m; ++i)
    if (objs[i] != objs[i]) return GEVO_E_ARG;
  // fast non-dominated sort: who each point dominates, how many dominate it
  std::vector<std::vector<uint32_t>> dominated(n);
  std::vector<uint32_t> n_dom(n, 0);
  for (uint32_t p = 0; p < n; ++p)
    for (uint32_t q = 0; q < n; ++q) {
      if (dominates(objs + (size_t)p * m, objs + (size_t)q * m, m)) dominated[p].push_back(q);
      else if (dominates(objs + (size_t)q * m, objs + (size_t)p * m, m)) ++n_dom[p];
    }
  std::vector<uint32_t> front, next;
  for (uint32_t p = 0; p < n; ++p)
    if (n_dom[p] == 0) front.push_back(p);
  uint32_t r = 0;
  while (!front.empty()) {
    next.clear();
    for (uint32_t p : front) {
      rank[p] = r;
      for (uint32_t q : dominated[p])
        if (--n_dom[q] == 0) next.push_back(q);
    }
    front.swap(next);
    ++r;
  }
  // crowding distance per front
  for (uint32_t i = 0; i < n; ++i) crowding[i] = 0.0;
  std::vector<uint32_t> members, order;
  for (uint32_t f = 0; f < r; ++f) {
    members.clear();
    for (uint32_t i = 0; i < n; ++i)
      if (rank[i] == f) members.push_back(i);
    for (uint32_t k = 0; k < m; ++k) {
      order = members;   // ascending index, so a stable sort orders by (f_k, index)
      std::stable_sort(order.begin(), order.end(),
                       [&](uint32_t a, uint32_t b) { return objs[(size_t)a * m + k] < objs[(size_t)b * m + k]; });
      const double lo = objs[(size_t)order.front() * m + k], hi = objs[(size_t)order.back() * m + k];
      crowding[order.front()] = INFINITY;
      crowding[order.back()] = INFINITY;
      if (hi > lo)
        for (size_t j = 1; j + 1 < order.size(); ++j) {
          const uint32_t i = order[j];
          crowding[i] = crowding[i] + (objs[(size_t)order[j + 1] * m + k] - objs[(size_t)order[j - 1] * m + k]) / (hi - lo);
        }
    }
  }
  return GEVO_OK;
}

gevo_status gevo_nsga2_select(uint32_t n, const uint32_t* rank, const double* crowding, uint32_t n_elite,
                              uint32_t n_select, uint64_t seed, uint32_t gen, uint32_t* out) {
  if (n_elite > n_select || n_elite > n) return GEVO_E_ARG;
  if (n_select == 0) return GEVO_OK;
  if (n == 0 || !rank || !crowding || !out) return GEVO_E_ARG;
  auto better = [&](uint32_t a, uint32_t b) {
    if (rank[a] != rank[b]) return rank[a] < rank[b];
    if (crowding[a] != crowding[b]) return crowding[a] > crowding[b];
    return a < b;
  };
  std::vector<uint32_t> order(n);
  for (uint32_t i = 0; i < n; ++i) order[i] = i;
  std::sort(order.begin(), order.end(), better);
  for (uint32_t i = 0; i < n_elite; ++i) out[i] = order[i];
  for (uint32_t j = 0; j < n_select - n_elite; ++j) {
    uint32_t w[4];
    draw4(seed, j, gen, 0, kStreamSelect, w);
    const uint32_t a = below(w[0], n), b = below(w[1], n);
    out[n_elite + j] = (a == b || better(a, b)) ? a : b;
  }
  return GEVO_OK;
}

gevo_status gevo_genomes_initial(uint32_t n, uint32_t n_mut, uint64_t seed, double rho_lo, uint32_t id_base,
                                 double struct_p, uint32_t n_layers, const uint32_t* dims, gevo_edit* out) {
  NetShape net;
  if (!(rho_lo >= 0.0 && rho_lo <= 1.0) || !valid_shape(struct_p, n_layers, dims, &net)) return GEVO_E_ARG;
  if ((size_t)n * n_mut == 0) return GEVO_OK;
  if (!out) return GEVO_E_ARG;
  for (uint32_t i = 0; i < n; ++i)
    for (uint32_t j = 0; j < n_mut; ++j)
      out[(size_t)n_mut * i + j] = random_edit(seed, 0, i, j, id_base + n_mut * i + j, rho_lo, struct_p, net);
  return GEVO_OK;
}

gevo_status gevo_genomes_breed(uint32_t n, const uint32_t* offsets, const gevo_edit* edits, uint64_t seed,
                               uint32_t gen, double cxpb, double mutpb, double rho_lo, uint32_t id_base,
                               uint32_t max_edits, double struct_p, uint32_t n_layers, const uint32_t* dims,
                               uint32_t* out_offsets, gevo_edit* out_edits, size_t out_capacity) {
  NetShape net;
  if (gen == 0 || !valid_offsets(n, offsets) || !out_offsets || !valid_shape(struct_p, n_layers, dims, &net))
    return GEVO_E_ARG;
  if (!(cxpb >= 0.0 && cxpb <= 1.0) || !(mutpb >= 0.0 && mutpb <= 1.0) || !(rho_lo >= 0.0 && rho_lo <= 1.0))
    return GEVO_E_ARG;
  if (offsets[n] > 0 && !edits) return GEVO_E_ARG;
  if (out_capacity < (size_t)offsets[n] + n || (out_capacity > 0 && !out_edits)) return GEVO_E_ARG;
  std::vector<std::vector<gevo_edit>> kids(n);
  for (uint32_t i = 0; i < n; ++i) kids[i].assign(edits + offsets[i], edits + offsets[i + 1]);
  for (uint32_t i = 0; i + 1 < n; i += 2) {
    uint32_t w[4];
    draw4(seed, 0, gen, i, kStreamCross, w);
    if (u24(w[0]) < cxpb) {
      std::vector<gevo_edit> cat = kids[i];
      cat.insert(cat.end(), kids[i + 1].begin(), kids[i + 1].end());
      for (size_t t = cat.size(); t-- > 1;) {
        uint32_t s[4];
        draw4(seed, 1 + (uint32_t)(t / 4), gen, i, kStreamCross, s);
        std::swap(cat[t], cat[below(s[t % 4], t + 1)]);
      }
      const size_t cut = below(w[1], cat.size() + 1);
      kids[i].assign(cat.begin(), cat.begin() + std::min(cut, (size_t)max_edits));
      kids[i + 1].assign(cat.begin() + cut, cat.begin() + cut + std::min(cat.size() - cut, (size_t)max_edits));
    }
  }
  for (uint32_t i = 0; i < n; ++i) {
    uint32_t w[4];
    draw4(seed, 0, gen, i, kStreamMut, w);
    if (u24(w[0]) < mutpb && kids[i].size() < max_edits)
      kids[i].push_back(random_edit(seed, gen, i, 1, id_base + i, rho_lo, struct_p, net));
  }
  size_t off = 0;
  out_offsets[0] = 0;
  for (uint32_t i = 0; i < n; ++i) {
    for (const gevo_edit& e : kids[i]) out_edits[off++] = e;
    out_offsets[i + 1] = (uint32_t)off;
  }
  return GEVO_OK;
}

}  // extern "C"
