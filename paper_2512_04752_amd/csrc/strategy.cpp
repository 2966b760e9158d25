// Workload-aware drafting-strategy selection (RLHFSpec Section 5), host code.
//
// Objective (Section 5.1): the draft token num n that maximises
// al(n) / t_sd(n), the accepted tokens per unit of step time.
//   * al(n) (Section 5.2): the sum of the node weights w(u) = F(dl(u)) of the
//     selected nodes S(n); the caller passes w (F is fitted on the draft side).
//   * t_sd(n) (Section 5.2): a regression on the verification features, the
//     summed committed lengths N_seq and the summed draft-token counts
//     N_draft (plus the tree-token x KV-length product, the part of attention
//     that grows with both), with a bucket cache: feature values within one
//     bucket share one prediction.
// Search (Section 5.3): S(n+1) = S(n) + the heaviest unselected node, taken
// from a max-priority queue that receives the nodes of layer m when the
// search reaches layer m; the search stops once the objective has fallen
// `patience` times in a row (the sugar-water argument: once an increment's
// ratio of accepted tokens to time is below the running ratio, it only falls).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <queue>
#include <unordered_map>
#include <vector>

#include "common.h"
#include "specverify.h"

struct spec_cost_model {
  spec_cost_coeffs c;
  std::unordered_map<uint64_t, double> cache;
  int64_t hits = 0, misses = 0;
};

namespace {

int bad(int code, const char* msg) { return spec::set_error(code, msg); }

double evaluate(const spec_cost_coeffs& c, double n_seq, double n_draft, double tree_kv) {
  return c.c0 + c.c_seq * n_seq + c.c_draft * n_draft + c.c_tree * tree_kv;
}

// Bucket index of a non-negative feature: 0 for 0, else 1 + floor(log(x) /
// log(1 + ratio)); its representative is the geometric midpoint.
int64_t bucket(int64_t x, double lr) { return x <= 0 ? 0 : 1 + (int64_t)std::floor(std::log((double)x) / lr); }
double representative(int64_t b, double lr) { return b == 0 ? 0.0 : std::exp((b - 1 + 0.5) * lr); }

double predict(spec_cost_model* m, int64_t n_seq, int64_t n_draft, int64_t tree_kv) {
  if (m->c.bucket_ratio <= 0.0) return evaluate(m->c, (double)n_seq, (double)n_draft, (double)tree_kv);
  const double lr = std::log1p(m->c.bucket_ratio);
  const int64_t bs = bucket(n_seq, lr), bd = bucket(n_draft, lr), bt = bucket(tree_kv, lr);
  const uint64_t key = ((uint64_t)bs << 42) ^ ((uint64_t)bd << 21) ^ (uint64_t)bt;
  auto it = m->cache.find(key);
  if (it != m->cache.end()) {
    ++m->hits;
    return it->second;
  }
  ++m->misses;
  const double t = evaluate(m->c, representative(bs, lr), representative(bd, lr), representative(bt, lr));
  m->cache.emplace(key, t);
  return t;
}

}  // namespace

extern "C" {

__attribute__((visibility("default"))) int spec_cost_model_create(const spec_cost_coeffs* c,
                                                                  spec_cost_model** out) {
  if (!c || !out) return bad(SPEC_ERR_INVALID, "null argument");
  if (!(c->bucket_ratio >= 0.0) || c->bucket_ratio > 1.0)
    return bad(SPEC_ERR_INVALID, "bucket_ratio must be in [0, 1]");
  spec_cost_model* m = new spec_cost_model;
  m->c = *c;
  *out = m;
  return SPEC_OK;
}

__attribute__((visibility("default"))) int spec_cost_model_free(spec_cost_model* m) {
  if (!m) return bad(SPEC_ERR_INVALID, "null handle");
  delete m;
  return SPEC_OK;
}

__attribute__((visibility("default"))) double spec_cost_predict(spec_cost_model* m, int64_t n_seq,
                                                               int64_t n_draft, int64_t tree_kv) {
  if (!m || n_seq < 0 || n_draft < 0 || tree_kv < 0) return -1.0;
  return predict(m, n_seq, n_draft, tree_kv);
}

__attribute__((visibility("default"))) int spec_cost_model_stats(const spec_cost_model* m,
                                                                int64_t* hits, int64_t* misses) {
  if (!m || !hits || !misses) return bad(SPEC_ERR_INVALID, "null argument");
  *hits = m->hits;
  *misses = m->misses;
  return SPEC_OK;
}

__attribute__((visibility("default"))) int spec_select_draft_count(
    spec_cost_model* m, int32_t batch, const int32_t* seq_lens, const int32_t* tree_offsets,
    const int32_t* parents, const float* weights, int32_t n_max, int32_t patience, int32_t* n_out,
    int32_t* selected, double* objective) {
  if (!m || !seq_lens || !tree_offsets || !parents || !weights || !n_out || !selected)
    return bad(SPEC_ERR_INVALID, "null argument");
  if (batch < 1 || n_max < 1 || n_max > SPEC_MAX_TREE || patience < 1)
    return bad(SPEC_ERR_INVALID, "batch, n_max or patience out of range");
  if (tree_offsets[0] != 0) return bad(SPEC_ERR_TREE, "tree_offsets[0] must be 0");
  // Validate the candidate trees and compute node depths.
  std::vector<int> depth(tree_offsets[batch] > 0 ? tree_offsets[batch] : 0);
  for (int b = 0; b < batch; ++b) {
    const int o = tree_offsets[b], t = tree_offsets[b + 1] - o;
    if (t < 1) return bad(SPEC_ERR_TREE, "empty candidate tree");
    if (seq_lens[b] < 0) return bad(SPEC_ERR_INVALID, "negative seq_len");
    if (parents[o] != -1) return bad(SPEC_ERR_TREE, "parents[root] must be -1");
    depth[o] = 0;
    for (int i = 1; i < t; ++i) {
      const int p = parents[o + i];
      if (p < 0 || p >= i) return bad(SPEC_ERR_TREE, "parent must precede its child");
      depth[o + i] = depth[o + p] + 1;
    }
    for (int i = 0; i < t; ++i) {
      if (!(weights[o + i] >= 0.f)) return bad(SPEC_ERR_INVALID, "node weights must be >= 0");
      if (i > 0 && weights[o + i] > weights[o + parents[o + i]])
        return bad(SPEC_ERR_INVALID, "node weights must not increase from parent to child");
    }
  }
  // Per sample: S(1) = {root}; the step that forms S(k+1) first lets the
  // nodes of depth k (the tree's layer k+1) join a max-priority queue
  // (heavier first; on equal weight the shallower, then the lower index),
  // then moves the top of the queue into S.  al_b[k] = weight of S(k+1).
  struct Cand {
    float w;
    int depth, idx;
    bool operator<(const Cand& o) const {   // priority order: larger is better
      if (w != o.w) return w < o.w;
      if (depth != o.depth) return depth > o.depth;
      return idx > o.idx;
    }
  };
  std::vector<std::vector<double>> al(batch);
  std::vector<int> size_of(batch);
  for (int b = 0; b < batch; ++b) {
    const int o = tree_offsets[b], t = tree_offsets[b + 1] - o;
    const int limit = std::min(t, (int)n_max);
    int32_t* sel = selected + (size_t)b * n_max;
    for (int k = 0; k < n_max; ++k) sel[k] = -1;
    std::vector<std::vector<int>> by_layer;
    for (int i = 0; i < t; ++i) {
      const int d = depth[o + i];
      if ((int)by_layer.size() <= d) by_layer.resize(d + 1);
      by_layer[d].push_back(i);
    }
    std::priority_queue<Cand> pq;
    sel[0] = 0;
    al[b].push_back(weights[o]);
    for (int mstep = 1; mstep < limit; ++mstep) {
      if (mstep < (int)by_layer.size())
        for (int i : by_layer[mstep]) pq.push(Cand{weights[o + i], mstep, i});
      if (pq.empty()) break;
      const Cand c = pq.top();
      pq.pop();
      sel[mstep] = c.idx;
      al[b].push_back(al[b].back() + c.w);
    }
    size_of[b] = (int)al[b].size();
  }
  // Search over n with early stopping.
  double best = -1.0, prev = -1.0;
  int best_n = 1, falls = 0;
  for (int n = 1; n <= n_max; ++n) {
    double al_n = 0.0;
    int64_t n_seq = 0, n_draft = 0, tree_kv = 0;
    for (int b = 0; b < batch; ++b) {
      const int k = std::min(n, size_of[b]);
      al_n += al[b][k - 1];
      n_seq += seq_lens[b];
      n_draft += k;
      tree_kv += (int64_t)k * seq_lens[b];
    }
    const double t = predict(m, n_seq, n_draft, tree_kv);
    if (!(t > 0.0)) return bad(SPEC_ERR_INVALID, "cost model predicted a non-positive time");
    const double obj = al_n / t;
    if (objective) objective[n - 1] = obj;
    if (obj > best) {
      best = obj;
      best_n = n;
    }
    falls = (n > 1 && obj < prev) ? falls + 1 : 0;
    prev = obj;
    if (falls >= patience) {
      for (int r = n; r < n_max && objective; ++r) objective[r] = 0.0;
      break;
    }
  }
  *n_out = best_n;
  return SPEC_OK;
}

}  // extern "C"
