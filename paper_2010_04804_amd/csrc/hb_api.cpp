// hb_api.cpp -- the C-ABI of libhb: validation, canonical renumbering, the
// per-strategy tensor builders (Tables 3, 5 and 6 of Sec. 4.1), the strategy
// selector (Sec. 5.1) and device upload. The scoring itself runs only in the
// HIP kernels of hb_kernels.hip; there is no host fallback.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <map>
#include <tuple>
#include <new>
#include <string>
#include <vector>

#include "hb.h"
#include "hb_internal.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string &msg) {
  g_last_error = msg;
  return code;
}

uint32_t fbits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

// One tree renumbered breadth-first: canonical node 0 is the root and the two
// children of an internal node get consecutive ids (left, then right).
struct CanonTree {
  std::vector<int32_t> caller;  // canonical -> caller-local id
  std::vector<int32_t> feat;    // -1 at leaves
  std::vector<uint8_t> dleft;   // 1: a missing (NaN) value goes left at this node
  std::vector<int32_t> cat;     // category set of a categorical node (index into the
                                // compile's set table), -1 for a numeric node or a leaf
  std::vector<float> thr;
  std::vector<int32_t> left;    // canonical left child (right = left + 1), -1 at leaves
  std::vector<int32_t> parent;  // -1 at the root
  std::vector<int32_t> depth;
  int32_t max_depth = 0;
  int32_t n_internal = 0, n_leaves = 0;
  int32_t size() const { return (int32_t)caller.size(); }
};

// Category sets, deduplicated: trailing zero words dropped, so sets that hold
// the same categories share one entry.
struct CatSets {
  std::vector<std::vector<uint32_t>> sets;
  std::map<std::vector<uint32_t>, int32_t> index;
  int32_t add(const uint32_t *w, int64_t n) {
    while (n > 0 && w[n - 1] == 0) --n;
    std::vector<uint32_t> key(w, w + n);
    auto it = index.find(key);
    if (it != index.end()) return it->second;
    const int32_t id = (int32_t)sets.size();
    index.emplace(key, id);
    sets.push_back(std::move(key));
    return id;
  }
};

bool is_categorical(const hb_ensemble_desc *d, int64_t node) {
  return d->cat_offset && d->cat_offset[node + 1] > d->cat_offset[node];
}

int canonicalise(const hb_ensemble_desc *d, int32_t t, CanonTree *ct, CatSets *cs) {
  const int64_t base = d->tree_node_offset[t];
  const int64_t n64 = d->tree_node_offset[t + 1] - base;
  if (n64 < 1 || n64 > (int64_t)std::numeric_limits<int32_t>::max() / 2)
    return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + ": bad node count");
  const int32_t n = (int32_t)n64;
  std::vector<int32_t> canon_of(n, -1);
  ct->caller.clear();
  ct->caller.reserve(n);
  ct->caller.push_back(0);
  canon_of[0] = 0;
  for (size_t i = 0; i < ct->caller.size(); ++i) {
    const int32_t v = ct->caller[i];
    const int32_t f = d->feature[base + v];
    if (f < 0) continue;
    if (f >= d->n_features)
      return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + " node " +
                                            std::to_string(v) + ": feature out of range");
    const bool cat = is_categorical(d, base + v);  // its threshold is not read
    if (!cat && std::isnan(d->threshold[base + v]))
      return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + " node " +
                                            std::to_string(v) + ": NaN threshold");
    if (d->default_left && d->default_left[base + v] > 1)
      return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + " node " +
                                            std::to_string(v) + ": default_left must be 0 or 1");
    if (!cat && d->default_left && d->default_left[base + v] && d->threshold[base + v] == -INFINITY)
      return fail(HB_ERR_UNSUPPORTED, "tree " + std::to_string(t) + " node " + std::to_string(v) +
                                          ": a node that sends missing values left cannot have threshold -inf");
    const int32_t kids[2] = {d->left[base + v], d->right[base + v]};
    for (int32_t c : kids) {
      if (c < 0 || c >= n)
        return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + " node " +
                                              std::to_string(v) + ": child out of range");
      if (canon_of[c] >= 0)
        return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + " node " +
                                              std::to_string(c) + ": reached twice (cycle or shared node)");
      canon_of[c] = (int32_t)ct->caller.size();
      ct->caller.push_back(c);
    }
  }
  if ((int32_t)ct->caller.size() != n)
    return fail(HB_ERR_INVALID_MODEL, "tree " + std::to_string(t) + ": " +
                                          std::to_string(n - (int32_t)ct->caller.size()) +
                                          " node(s) unreachable from the root");
  ct->feat.assign(n, -1);
  ct->dleft.assign(n, 0);
  ct->cat.assign(n, -1);
  ct->thr.assign(n, 0.0f);
  ct->left.assign(n, -1);
  ct->parent.assign(n, -1);
  ct->depth.assign(n, 0);
  ct->max_depth = 0;
  ct->n_internal = ct->n_leaves = 0;
  for (int32_t c = 0; c < n; ++c) {
    const int32_t v = ct->caller[c];
    const int32_t f = d->feature[base + v];
    if (f < 0) {
      ++ct->n_leaves;
      ct->max_depth = std::max(ct->max_depth, ct->depth[c]);
      continue;
    }
    ++ct->n_internal;
    ct->feat[c] = f;
    ct->dleft[c] = d->default_left ? d->default_left[base + v] : 0;
    ct->thr[c] = d->threshold[base + v];
    if (is_categorical(d, base + v)) {
      const int64_t lo = d->cat_offset[base + v];
      ct->cat[c] = cs->add(d->cat_bits + lo, d->cat_offset[base + v + 1] - lo);
      ct->thr[c] = 0.5f;  // the node tests its 0/1 indicator column
    }
    const int32_t l = canon_of[d->left[base + v]];
    const int32_t r = canon_of[d->right[base + v]];
    if (r != l + 1) return fail(HB_ERR_INVALID_MODEL, "internal: breadth-first order broken");
    ct->left[c] = l;
    ct->parent[l] = ct->parent[r] = c;
    ct->depth[l] = ct->depth[r] = ct->depth[c] + 1;
  }
  return HB_OK;
}

}  // namespace

struct hb_handle {
  hb_info info{};
  int32_t device = -1;
  // input column of each feature-tile column (sorted features the trees test)
  std::vector<int32_t> cols;
  bool pruned = false;  // cols is not the identity
  // host copies of the compiled tensors
  std::vector<int32_t> tree_class;
  std::vector<float> base_score;
  bool has_base = false;
  // PTT
  std::vector<uint32_t> ptt_node;
  std::vector<float> ptt_leaf_value;
  std::vector<int32_t> ptt_leaf_id;
  // TT
  std::vector<uint32_t> tt_node;
  std::vector<int32_t> tt_depth, tt_dims;
  std::vector<float> tt_leaf_value;
  std::vector<int32_t> tt_leaf_id;
  int32_t tt_n_pad = 0;
  // GEMM
  std::vector<uint32_t> gemm_node;
  std::vector<int32_t> gemm_shape, gemm_bias, gemm_dims;
  std::vector<int8_t> gemm_ct;
  std::vector<float> gemm_leaf_value;
  std::vector<int32_t> gemm_leaf_id;
  int32_t gemm_k_pad = 0, gemm_l_pad = 0, gemm_n_shapes = 0;
  // packed blocks of the fast traversal kernels (device layout only)
  std::vector<uint32_t> ptt_fast, tt_fast, tt_fast_leaf;
  std::vector<float> ptt_fast_leafv;  // mode 3: [padded T][2^D] leaf values
  int32_t ptt_fast_chunks = 0, tt_fast_lg = 0, tt_fast_chunks = 0, tt_fast_mode = 1;
  int32_t ptt_fast_mode = 0, ptt_id_base = 0;
  // device
  std::vector<void *> allocations;
  hb::EnsembleDev ens{};
  hb::PttDev ptt{};
  hb::TtDev tt{};
  hb::GemmDev gemm{};
};

namespace {

// Sec. 5.1 picks GEMM for shallow trees or small batches, PTT up to depth 10
// and TT beyond. Re-measured on MI355X (the crossover sweep: 100-tree
// forests of depth 3, 7, 11 and 12, perfect and leaf-wise, over 200 and 28
// features, batch 1 to 1M, each strategy with and without a tree-split
// workspace): PTT is fastest, or within a few percent, on every near-perfect
// forest at every batch size and depth up to 12 (with narrow rows a depth-11
// or -12 PTT walk is 2x to 3x faster than TT's from 10K rows on); on
// unbalanced trees PTT's trees-across-lanes walk still wins up to a few
// hundred rows, TT from about a thousand on; GEMM is slower than PTT at every
// point (its tree split brings batch 1 of a 500-tree depth-8 forest from 305
// to 12 us, against 6 us for PTT). So AUTO takes PTT while the padded
// perfect tree stays within a small multiple of the real node count, or for
// small batches; TT otherwise; GEMM only when asked for, or when nothing else
// can hold the model.
constexpr double kAutoPttMaxBalance = 4.0;
constexpr int64_t kAutoPttSmallBatch = 256;

int select_strategy(const hb_handle *h, int64_t n_rows) {
  const hb_info &I = h->info;
  if (I.feasible[HB_STRATEGY_PTT] && (I.balance <= kAutoPttMaxBalance || n_rows <= kAutoPttSmallBatch))
    return HB_STRATEGY_PTT;
  if (I.feasible[HB_STRATEGY_TT]) return HB_STRATEGY_TT;
  if (I.feasible[HB_STRATEGY_PTT]) return HB_STRATEGY_PTT;
  return HB_STRATEGY_GEMM;
}

void build_ptt(hb_handle *h, const hb_ensemble_desc *d, const std::vector<CanonTree> &trees) {
  const int32_t D = h->info.max_depth;
  const int64_t S = int64_t(1) << D;
  const int64_t NS = std::max<int64_t>(S, 2);  // node slots per tree (slot 0 unused)
  const int32_t ld = d->leaf_dim;
  const int32_t T = d->n_trees;
  h->ptt_node.assign((size_t)(T * NS * 2), 0u);
  h->ptt_leaf_value.assign((size_t)(T * S * ld), 0.0f);
  h->ptt_leaf_id.assign((size_t)(T * S), 0);
  std::vector<int32_t> at(2 * S);  // heap position -> canonical node it descends from
  for (int32_t t = 0; t < T; ++t) {
    const CanonTree &ct = trees[t];
    const int64_t base = d->tree_node_offset[t];
    at[1] = 0;
    for (int64_t p = 1; p < S; ++p) {
      const int32_t c = at[p];
      uint32_t *rec = &h->ptt_node[(size_t)((t * NS + p) * 2)];
      if (ct.feat[c] >= 0) {
        rec[0] = fbits(ct.thr[c]);
        rec[1] = (uint32_t)ct.feat[c];
        at[2 * p] = ct.left[c];
        at[2 * p + 1] = ct.left[c] + 1;
      } else {
        // Sec. 4.1: a leaf above depth D becomes a perfect subtree whose
        // decisions are free; every leaf under it maps to the original leaf.
        rec[0] = fbits(0.0f);
        rec[1] = 0u;
        at[2 * p] = at[2 * p + 1] = c;
      }
    }
    for (int64_t s = 0; s < S; ++s) {
      const int32_t c = D == 0 ? 0 : at[S + s];
      const int32_t v = ct.caller[c];
      h->ptt_leaf_id[(size_t)(t * S + s)] = v;
      for (int32_t k = 0; k < ld; ++k)
        h->ptt_leaf_value[(size_t)((t * S + s) * ld + k)] = d->leaf_value[(base + v) * ld + k];
    }
  }
}

void build_tt(hb_handle *h, const hb_ensemble_desc *d, const std::vector<CanonTree> &trees) {
  int32_t n_pad = 2;
  for (const CanonTree &ct : trees) n_pad = std::max(n_pad, ct.size());
  n_pad += n_pad & 1;  // even, so a tree's records are a whole number of 16-byte words
  h->tt_n_pad = n_pad;
  const int32_t ld = d->leaf_dim;
  const int32_t T = d->n_trees;
  const uint32_t ninf = fbits(-std::numeric_limits<float>::infinity());
  h->tt_node.assign((size_t)T * n_pad * 2, 0u);
  h->tt_depth.assign(T, 0);
  h->tt_leaf_value.assign((size_t)T * n_pad * ld, 0.0f);
  h->tt_leaf_id.assign((size_t)T * n_pad, 0);
  for (int32_t t = 0; t < T; ++t) {
    const CanonTree &ct = trees[t];
    const int64_t base = d->tree_node_offset[t];
    h->tt_depth[t] = ct.max_depth;
    for (int32_t c = 0; c < n_pad; ++c) {
      uint32_t *rec = &h->tt_node[((size_t)t * n_pad + c) * 2];
      if (c < ct.size() && ct.feat[c] >= 0) {
        rec[0] = fbits(ct.thr[c]);
        rec[1] = (uint32_t)ct.feat[c] | ((uint32_t)(ct.left[c] + 1) << 16);
      } else {
        // Table 5 makes leaves point to themselves; here a leaf's threshold
        // is -inf so the rule always takes the stored "right" id, itself.
        rec[0] = ninf;
        rec[1] = (uint32_t)c << 16;
      }
      if (c < ct.size()) {
        const int32_t v = ct.caller[c];
        h->tt_leaf_id[(size_t)t * n_pad + c] = v;
        if (ct.feat[c] < 0)
          for (int32_t k = 0; k < ld; ++k)
            h->tt_leaf_value[((size_t)t * n_pad + c) * ld + k] = d->leaf_value[(base + v) * ld + k];
      }
    }
  }
  h->tt_dims = {n_pad};
}

// Packed blocks for the fast kernels; see hb_internal.h. A leaf record holds
// the leaf's value and caller id; with vector leaves the value field holds
// the first component and the kernels read the vector from the strategy's
// leaf-value table.
void build_fast(hb_handle *h, const hb_ensemble_desc *d, const std::vector<CanonTree> &trees) {
  const int32_t ld = d->leaf_dim;
  const int32_t T = d->n_trees;
  const int32_t D = h->info.max_depth;
  if (h->info.feasible[HB_STRATEGY_PTT] && D >= 1 && D <= hb::kFastMaxLg) {
    const size_t S = (size_t)1 << D;
    const size_t padded = (size_t)(T + hb::kFastIdGroup - 1) / hb::kFastIdGroup * hb::kFastIdGroup;
    // Mode 3 (leaf values apart, in global memory, ids formed from the leaf
    // slot): scalar leaves (one output, or one per tree class), depth <= 8
    // (slots fit a byte), every leaf's caller id its slot plus one base
    // (heap-ordered perfect trees), and the values small enough to stay in
    // an XCD's L2.
    bool affine = ld == 1 && D <= 8 && (int64_t)(padded * S * 4) <= hb::kTtLeafGlobalMax;
    const int32_t base = h->ptt_leaf_id.empty() ? 0 : h->ptt_leaf_id[0];
    for (size_t i = 0; affine && i < (size_t)T * S; ++i) affine = h->ptt_leaf_id[i] == base + (int32_t)(i % S);
    if (affine) {
      const int tb = hb::fast_tree_bytes(3, D);
      const int tc = hb::fast_tc_m(3, tb);
      h->ptt_fast.assign(padded * S * 2, 0u);
      h->ptt_fast_leafv.assign(padded * S, 0.0f);  // padding trees add zero
      for (int32_t t = 0; t < T; ++t) {
        uint32_t *blk = &h->ptt_fast[(size_t)t * S * 2];
        for (size_t p = 1; p < S; ++p) {
          blk[2 * p] = h->ptt_node[((size_t)t * S + p) * 2];
          blk[2 * p + 1] = h->ptt_node[((size_t)t * S + p) * 2 + 1];
        }
        for (size_t q = 0; q < S; ++q) h->ptt_fast_leafv[(size_t)t * S + q] = h->ptt_leaf_value[(size_t)t * S + q];
      }
      h->ptt_fast_chunks = (int)(padded / tc);
      h->ptt_fast_mode = 3;
      h->ptt_id_base = base;
    }
  }
  if (h->info.feasible[HB_STRATEGY_PTT] && D >= 1 && D <= hb::kFastMaxLg && h->ptt_fast_mode != 3) {
    const size_t S = (size_t)1 << D;
    const int tb = hb::fast_tree_bytes(0, D);
    const int tc = hb::fast_tc(tb);
    const int chunks = (T + hb::kFastIdGroup - 1) / hb::kFastIdGroup * (hb::kFastIdGroup / tc);
    const size_t words = (size_t)tb / 4;
    h->ptt_fast.assign((size_t)chunks * tc * words, 0u);
    for (int32_t t = 0; t < T; ++t) {
      uint32_t *blk = &h->ptt_fast[(size_t)t * words];
      for (size_t p = 1; p < S; ++p) {
        blk[2 * p] = h->ptt_node[((size_t)t * S + p) * 2];
        blk[2 * p + 1] = h->ptt_node[((size_t)t * S + p) * 2 + 1];
      }
      for (size_t q = 0; q < S; ++q) {
        blk[2 * (S + q)] = fbits(h->ptt_leaf_value[((size_t)t * S + q) * ld]);
        blk[2 * (S + q) + 1] = (uint32_t)h->ptt_leaf_id[(size_t)t * S + q];
      }
    }
    h->ptt_fast_chunks = chunks;
  }
  int32_t max_nodes = 1;
  for (const CanonTree &ct : trees) max_nodes = std::max(max_nodes, ct.size());
  int lg = 1;
  while ((1 << lg) < max_nodes) ++lg;
  if (h->info.feasible[HB_STRATEGY_TT] && lg <= hb::kFastMaxLg) {
    // node records and leaf records per tree, 2^lg of each; the tree count
    // is padded to a multiple of the leaf-id group (so of every chunk size)
    const size_t NP = (size_t)1 << lg;
    const size_t words = 2 * NP;
    const size_t padded = (size_t)(T + hb::kFastIdGroup - 1) / hb::kFastIdGroup * hb::kFastIdGroup;
    h->tt_fast.assign(padded * words, 0u);
    h->tt_fast_leaf.assign(padded * words, 0u);
    // padding trees: every node a leaf that loops to itself, so a walk over
    // them stays at the root
    const uint32_t ninf_pad = fbits(-std::numeric_limits<float>::infinity());
    for (size_t t = (size_t)T; t < padded; ++t)
      for (size_t c = 0; c < NP; ++c) {
        h->tt_fast[t * words + 2 * c] = ninf_pad;
        h->tt_fast[t * words + 2 * c + 1] = (8u * (uint32_t)c) << 16;
      }
    for (int32_t t = 0; t < T; ++t) {
      const CanonTree &ct = trees[t];
      const int64_t base = d->tree_node_offset[t];
      uint32_t *blk = &h->tt_fast[(size_t)t * words];
      uint32_t *leaf = &h->tt_fast_leaf[(size_t)t * words];
      const uint32_t ninf = fbits(-std::numeric_limits<float>::infinity());
      for (size_t c = 0; c < NP; ++c) {
        uint32_t *rec = blk + 2 * c;
        if (c < (size_t)ct.size() && ct.feat[c] >= 0) {
          rec[0] = fbits(ct.thr[c]);
          rec[1] = (uint32_t)ct.feat[c] | (8u * (uint32_t)(ct.left[c] + 1)) << 16;
        } else {  // leaves (and padding) stay put: no x is below -inf
          rec[0] = ninf;
          rec[1] = (8u * (uint32_t)c) << 16;
        }
        uint32_t *lr = leaf + 2 * c;
        if (c < (size_t)ct.size()) {
          const int32_t v = ct.caller[c];
          lr[0] = ct.feat[c] < 0 ? fbits(d->leaf_value[(base + v) * ld]) : 0u;
          lr[1] = (uint32_t)v;
        }
      }
    }
    h->tt_fast_mode = (int64_t)(padded * NP * 8) <= hb::kTtLeafGlobalMax ? 2 : 1;
    h->tt_fast_lg = lg;
    h->tt_fast_chunks = (int)(padded / hb::fast_tc(hb::fast_tree_bytes(h->tt_fast_mode, lg)));
  }
}

void build_gemm(hb_handle *h, const hb_ensemble_desc *d, const std::vector<CanonTree> &trees) {
  const int32_t T = d->n_trees;
  const int32_t ld = d->leaf_dim;
  int32_t max_i = 1, max_l = 1;
  for (const CanonTree &ct : trees) {
    max_i = std::max(max_i, ct.n_internal);
    max_l = std::max(max_l, ct.n_leaves);
  }
  const int32_t k_pad = (max_i + 63) / 64 * 64;
  const int32_t l_pad = (max_l + 15) / 16 * 16;
  h->gemm_k_pad = k_pad;
  h->gemm_l_pad = l_pad;
  const uint32_t ninf = fbits(-std::numeric_limits<float>::infinity());
  h->gemm_node.assign((size_t)T * k_pad * 2, 0u);
  for (size_t i = 0; i < h->gemm_node.size(); i += 2) h->gemm_node[i] = ninf;
  h->gemm_shape.assign(T, 0);
  h->gemm_leaf_value.assign((size_t)T * l_pad * ld, 0.0f);
  h->gemm_leaf_id.assign((size_t)T * l_pad, 0);
  h->gemm_ct.clear();
  h->gemm_bias.clear();
  std::map<std::vector<uint8_t>, int32_t> shapes;
  std::vector<int32_t> kidx, leaves;
  for (int32_t t = 0; t < T; ++t) {
    const CanonTree &ct = trees[t];
    const int64_t base = d->tree_node_offset[t];
    const int32_t n = ct.size();
    // k: internal nodes in breadth-first order
    kidx.assign(n, -1);
    int32_t k = 0;
    for (int32_t c = 0; c < n; ++c)
      if (ct.feat[c] >= 0) {
        kidx[c] = k;
        uint32_t *rec = &h->gemm_node[((size_t)t * k_pad + k) * 2];
        rec[0] = fbits(ct.thr[c]);
        rec[1] = (uint32_t)ct.feat[c];
        ++k;
      }
    // l: leaves left to right (depth-first, left child first)
    leaves.clear();
    std::vector<int32_t> stack{0};
    while (!stack.empty()) {
      const int32_t c = stack.back();
      stack.pop_back();
      if (ct.feat[c] < 0) {
        leaves.push_back(c);
      } else {
        stack.push_back(ct.left[c] + 1);
        stack.push_back(ct.left[c]);
      }
    }
    for (int32_t l = 0; l < (int32_t)leaves.size(); ++l) {
      const int32_t v = ct.caller[leaves[l]];
      h->gemm_leaf_id[(size_t)t * l_pad + l] = v;
      for (int32_t q = 0; q < ld; ++q)
        h->gemm_leaf_value[((size_t)t * l_pad + l) * ld + q] = d->leaf_value[(base + v) * ld + q];
    }
    // the shape: breadth-first leaf flags determine the tree's structure
    std::vector<uint8_t> key(n);
    for (int32_t c = 0; c < n; ++c) key[c] = ct.feat[c] < 0;
    auto it = shapes.find(key);
    if (it != shapes.end()) {
      h->gemm_shape[t] = it->second;
      continue;
    }
    const int32_t s = (int32_t)shapes.size();
    shapes.emplace(std::move(key), s);
    h->gemm_shape[t] = s;
    h->gemm_ct.resize((size_t)(s + 1) * l_pad * k_pad, 0);
    h->gemm_bias.resize((size_t)(s + 1) * l_pad, -(1 << 30));
    int8_t *C = &h->gemm_ct[(size_t)s * l_pad * k_pad];
    for (int32_t l = 0; l < (int32_t)leaves.size(); ++l) {
      // Table 3: C is +1 where the leaf lies in a node's left subtree and -1
      // in its right subtree; D counts the left edges on the leaf's root path.
      int32_t dl = 0;
      for (int32_t c = leaves[l]; ct.parent[c] >= 0; c = ct.parent[c]) {
        const int32_t p = ct.parent[c];
        const bool is_left = ct.left[p] == c;
        C[(size_t)l * k_pad + kidx[p]] = is_left ? 4 : -4;
        dl += is_left;
      }
      h->gemm_bias[(size_t)s * l_pad + l] = l - 256 * dl;
    }
  }
  h->gemm_n_shapes = (int32_t)shapes.size();
  h->gemm_dims = {k_pad, l_pad, h->gemm_n_shapes};
}

// Node records [T][slots] (two words each) regrouped as [ceil(T/64)][slots][64]
// for the trees-across-lanes kernel; records of padding trees stay zero and
// are never read (lanes past the last tree do not walk).
std::vector<uint32_t> interleave64(const std::vector<uint32_t> &node, int64_t T, int64_t slots) {
  const int64_t groups = (T + 63) / 64;
  std::vector<uint32_t> il((size_t)(groups * slots * 64 * 2), 0u);
  for (int64_t t = 0; t < T; ++t)
    for (int64_t p = 0; p < slots; ++p) {
      const size_t dst = (size_t)(((t / 64) * slots + p) * 64 + t % 64) * 2;
      il[dst] = node[(size_t)(t * slots + p) * 2];
      il[dst + 1] = node[(size_t)(t * slots + p) * 2 + 1];
    }
  return il;
}

// Leaf values [T * slots][ld] and caller ids [T * slots] as one record per
// leaf: ld value words, the id, zero padding to leaf_pk_words(ld).
std::vector<uint32_t> pack_leaves(const std::vector<float> &value, const std::vector<int32_t> &id, int32_t ld) {
  const size_t w = (size_t)hb::leaf_pk_words(ld);
  std::vector<uint32_t> pk(id.size() * w, 0u);
  for (size_t i = 0; i < id.size(); ++i) {
    for (int32_t k = 0; k < ld; ++k) pk[i * w + k] = fbits(value[i * ld + k]);
    pk[i * w + ld] = (uint32_t)id[i];
  }
  return pk;
}

// The PTT last decision level with its leaves, trees interleaved by 64 (the
// layout of PttDev::last_il); D >= 1 and leaf_dim <= 2.
std::vector<uint32_t> ptt_last_level(const hb_handle *h, int32_t D, int32_t ld) {
  const int64_t T = h->info.n_trees, S = int64_t(1) << D, half = S / 2;
  const int64_t groups = (T + 63) / 64;
  std::vector<uint32_t> out((size_t)(groups * half * 64 * hb::kLastWords), 0u);
  for (int64_t t = 0; t < T; ++t)
    for (int64_t q = 0; q < half; ++q) {
      uint32_t *w = &out[(size_t)(((t / 64) * half + q) * 64 + t % 64) * hb::kLastWords];
      const size_t node = (size_t)(t * S + half + q) * 2;
      w[0] = h->ptt_node[node];
      w[1] = h->ptt_node[node + 1];
      for (int side = 0; side < 2; ++side) {
        const size_t leaf = (size_t)(t * S + 2 * q + side);
        uint32_t *lw = w + 2 + side * (ld + 1);
        for (int32_t k = 0; k < ld; ++k) lw[k] = fbits(h->ptt_leaf_value[leaf * ld + k]);
        lw[ld] = (uint32_t)h->ptt_leaf_id[leaf];
      }
    }
  return out;
}

template <class T>
int upload(hb_handle *h, const std::vector<T> &src, const T **dst) {
  if (src.empty()) {
    *dst = nullptr;
    return HB_OK;
  }
  void *p = nullptr;
  const size_t bytes = src.size() * sizeof(T);
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) return fail(HB_ERR_OOM, std::string("hipMalloc: ") + hipGetErrorString(e));
  h->allocations.push_back(p);
  e = hipMemcpy(p, src.data(), bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) return fail(HB_ERR_HIP, std::string("hipMemcpy: ") + hipGetErrorString(e));
  *dst = static_cast<const T *>(p);
  return HB_OK;
}

void release(hb_handle *h) {
  if (!h) return;
  if (h->device >= 0 && !h->allocations.empty()) {
    int prev = -1;
    (void)hipGetDevice(&prev);
    (void)hipSetDevice(h->device);
    (void)hipDeviceSynchronize();
    for (void *p : h->allocations) (void)hipFree(p);
    if (prev >= 0) (void)hipSetDevice(prev);
  }
  delete h;
}

int validate_desc(const hb_ensemble_desc *d) {
  if (!d) return fail(HB_ERR_INVALID_ARG, "desc is NULL");
  if (d->n_trees < 1 || d->n_trees > HB_MAX_TREES)
    return fail(HB_ERR_INVALID_ARG, "n_trees must be in [1, " + std::to_string(HB_MAX_TREES) + "]");
  if (d->n_features < 1) return fail(HB_ERR_INVALID_ARG, "n_features must be >= 1");
  if (d->n_outputs < 1 || d->n_outputs > HB_MAX_OUTPUTS)
    return fail(HB_ERR_INVALID_ARG, "n_outputs must be in [1, " + std::to_string(HB_MAX_OUTPUTS) + "]");
  if (d->leaf_dim != 1 && d->leaf_dim != d->n_outputs)
    return fail(HB_ERR_INVALID_ARG, "leaf_dim must be 1 or n_outputs");
  if (!d->tree_node_offset || !d->feature || !d->threshold || !d->left || !d->right || !d->leaf_value)
    return fail(HB_ERR_INVALID_ARG, "a per-node array is NULL");
  if (d->aggregation != HB_AGG_SUM && d->aggregation != HB_AGG_MEAN)
    return fail(HB_ERR_INVALID_ARG, "bad aggregation");
  if (d->transform < HB_POST_NONE || d->transform > HB_POST_SOFTMAX)
    return fail(HB_ERR_INVALID_ARG, "bad transform");
  if (d->tree_node_offset[0] != 0) return fail(HB_ERR_INVALID_ARG, "tree_node_offset[0] must be 0");
  for (int32_t t = 0; t < d->n_trees; ++t)
    if (d->tree_node_offset[t + 1] <= d->tree_node_offset[t])
      return fail(HB_ERR_INVALID_ARG, "tree_node_offset must be strictly increasing");
  if (d->leaf_dim == 1 && d->tree_class)
    for (int32_t t = 0; t < d->n_trees; ++t)
      if (d->tree_class[t] < 0 || d->tree_class[t] >= d->n_outputs)
        return fail(HB_ERR_INVALID_MODEL, "tree_class out of range at tree " + std::to_string(t));
  if (d->cat_offset) {
    const int64_t n_nodes = d->tree_node_offset[d->n_trees];
    if (d->cat_offset[0] != 0) return fail(HB_ERR_INVALID_MODEL, "cat_offset[0] must be 0");
    for (int64_t i = 0; i < n_nodes; ++i) {
      const int64_t w = d->cat_offset[i + 1] - d->cat_offset[i];
      if (w < 0) return fail(HB_ERR_INVALID_MODEL, "cat_offset must not decrease (node " + std::to_string(i) + ")");
      if (w > HB_MAX_CATEGORY_WORDS)
        return fail(HB_ERR_INVALID_MODEL, "node " + std::to_string(i) + ": more than " +
                                              std::to_string(HB_MAX_CATEGORY_WORDS) + " category words");
    }
    if (d->cat_offset[n_nodes] > 0 && !d->cat_bits) return fail(HB_ERR_INVALID_ARG, "cat_bits is NULL");
  }
  return HB_OK;
}

int compile_impl(const hb_ensemble_desc *d, int hint, int device, hb_handle **out) {
  int rc = validate_desc(d);
  if (rc) return rc;
  if (hint < HB_STRATEGY_AUTO || hint > HB_STRATEGY_PTT) return fail(HB_ERR_INVALID_ARG, "bad strategy hint");
  if (device < -1) return fail(HB_ERR_INVALID_ARG, "bad device");
  const int32_t T = d->n_trees;
  std::vector<CanonTree> trees(T);
  CatSets cat_sets;
  int64_t n_nodes = 0, n_int = 0, n_leaf = 0;
  int32_t D = 0, max_nodes = 0, max_leaves = 0;
  for (int32_t t = 0; t < T; ++t) {
    rc = canonicalise(d, t, &trees[t], &cat_sets);
    if (rc) return rc;
    n_nodes += trees[t].size();
    n_int += trees[t].n_internal;
    n_leaf += trees[t].n_leaves;
    D = std::max(D, trees[t].max_depth);
    max_nodes = std::max(max_nodes, trees[t].size());
    max_leaves = std::max(max_leaves, trees[t].n_leaves);
  }
  hb_handle *h = new (std::nothrow) hb_handle();
  if (!h) return fail(HB_ERR_OOM, "out of host memory");
  // Feature selection injection for trees (Sec. 5.2): features no decision
  // node tests are pruned and the decision variables re-indexed. The kernels
  // then stage only the columns some node tests (a narrower LDS tile, so
  // wide inputs reach the faster kernels), and the tables address a column by
  // its rank among those. Missing values: a column that nodes with the
  // default-left flag test gets a second tile column that reads NaN as -inf
  // (then x < t holds for every finite or +inf threshold, so NaN goes left),
  // and those nodes test that column; every other node sees NaN, which no
  // x < t accepts, so NaN goes right. Categorical nodes: each distinct
  // (column, category set, default-left) gets a tile column holding the 0/1
  // indicator of the row going left, which the node tests against 0.5. The
  // walk itself is unchanged.
  int32_t n_cols = d->n_features;
  {
    std::vector<int32_t> rank(2 * (size_t)d->n_features, -1);  // [column][default-left]
    std::map<std::tuple<int32_t, int32_t, int32_t>, int32_t> cat_rank;  // (column, set, dl)
    for (const CanonTree &ct : trees)
      for (int32_t c = 0; c < ct.size(); ++c)
        if (ct.feat[c] >= 0) {
          if (ct.cat[c] >= 0)
            cat_rank[std::make_tuple(ct.feat[c], ct.cat[c], (int32_t)ct.dleft[c])] = 0;
          else
            rank[2 * (size_t)ct.feat[c] + ct.dleft[c]] = 0;
        }
    std::vector<int32_t> cols;
    bool variant = !cat_rank.empty();
    for (size_t k = 0; k < rank.size(); ++k)
      if (rank[k] == 0) {
        rank[k] = (int32_t)cols.size();
        cols.push_back((int32_t)(k >> 1) | ((k & 1) ? hb::kColNanLeft : 0));
        variant |= (k & 1) != 0;
      }
    for (auto &kv : cat_rank) {
      kv.second = (int32_t)cols.size();
      cols.push_back(0);  // set below, once the descriptors' offset is known
    }
    if (cols.empty()) cols.push_back(0);  // only single-leaf trees: one dummy column
    // Pruning costs the kernels a gather through the column list instead of
    // whole-row loads, so it is applied when it removes at least a quarter of
    // the columns (or when missing values or categories need their own columns).
    h->pruned = variant || (int64_t)cols.size() * 4 <= (int64_t)d->n_features * 3;
    if (h->pruned) {
      n_cols = (int32_t)cols.size();
      // category descriptors {input column, W, W words} after the columns
      std::vector<int32_t> pool;
      for (const auto &kv : cat_rank) {
        const int64_t at = (int64_t)cols.size() + (int64_t)pool.size();
        if (at > hb::kColMask) {
          delete h;
          return fail(HB_ERR_UNSUPPORTED, "category sets too large");
        }
        const std::vector<uint32_t> &set = cat_sets.sets[std::get<1>(kv.first)];
        cols[kv.second] = (int32_t)at | hb::kColCat | (std::get<2>(kv.first) ? hb::kColNanLeft : 0);
        pool.push_back(std::get<0>(kv.first));
        pool.push_back((int32_t)set.size());
        for (uint32_t w : set) pool.push_back((int32_t)w);
      }
      h->cols = cols;
      h->cols.insert(h->cols.end(), pool.begin(), pool.end());
      for (CanonTree &ct : trees)
        for (int32_t c = 0; c < ct.size(); ++c)
          if (ct.feat[c] >= 0)
            ct.feat[c] = ct.cat[c] >= 0 ? cat_rank[std::make_tuple(ct.feat[c], ct.cat[c], (int32_t)ct.dleft[c])]
                                        : rank[2 * (size_t)ct.feat[c] + ct.dleft[c]];
    } else {
      h->cols.resize(d->n_features);
      for (int32_t f = 0; f < d->n_features; ++f) h->cols[f] = f;
    }
  }
  hb_info &I = h->info;
  I.n_trees = T;
  I.n_features = d->n_features;
  I.n_outputs = d->n_outputs;
  I.leaf_dim = d->leaf_dim;
  I.max_depth = D;
  I.device = device;
  I.n_nodes = n_nodes;
  I.n_internal = n_int;
  I.n_leaves = n_leaf;
  I.balance = n_int > 0 ? (double)T * (double)((int64_t(1) << D) - 1) / (double)n_int : 1.0;
  I.default_strategy = hint;
  I.ptt_depth = D;
  I.n_used_features = n_cols;
  // The traversal kernels stage at least one tree's tables in LDS.
  const int64_t per_slot = 12 + 4 * (int64_t)d->leaf_dim;
  const int64_t ptt_tree_bytes = per_slot * std::max<int64_t>(int64_t(1) << std::min(D, 30), 2);
  const int64_t tt_tree_bytes = per_slot * (max_nodes + 1);
  I.feasible[HB_STRATEGY_PTT] = D <= HB_PTT_MAX_DEPTH && ptt_tree_bytes <= hb::kTreeLdsLimit;
  I.feasible[HB_STRATEGY_TT] = max_nodes <= HB_TT_MAX_NODES && n_cols <= HB_MAX_FEATURES &&
                               tt_tree_bytes <= hb::kTreeLdsLimit;
  I.feasible[HB_STRATEGY_GEMM] = max_leaves <= HB_GEMM_MAX_LEAVES;
  I.feasible[HB_STRATEGY_AUTO] =
      I.feasible[HB_STRATEGY_PTT] || I.feasible[HB_STRATEGY_TT] || I.feasible[HB_STRATEGY_GEMM];
  if (!I.feasible[hint]) {
    delete h;
    return fail(HB_ERR_UNSUPPORTED, "requested strategy is infeasible for this ensemble");
  }
  h->device = device;
  try {
    if (I.feasible[HB_STRATEGY_PTT]) build_ptt(h, d, trees);
    if (I.feasible[HB_STRATEGY_TT]) build_tt(h, d, trees);
    if (I.feasible[HB_STRATEGY_GEMM]) build_gemm(h, d, trees);
    build_fast(h, d, trees);
  } catch (const std::bad_alloc &) {
    delete h;
    return fail(HB_ERR_OOM, "out of host memory building tables");
  }
  I.gemm_shapes = h->gemm_n_shapes;
  I.table_bytes[HB_STRATEGY_PTT] = (int64_t)(h->ptt_node.size() * 4 + h->ptt_leaf_value.size() * 4 +
                                             h->ptt_leaf_id.size() * 4);
  I.table_bytes[HB_STRATEGY_TT] = (int64_t)(h->tt_node.size() * 4 + h->tt_depth.size() * 4 +
                                            h->tt_leaf_value.size() * 4 + h->tt_leaf_id.size() * 4);
  I.table_bytes[HB_STRATEGY_GEMM] =
      (int64_t)(h->gemm_node.size() * 4 + h->gemm_shape.size() * 4 + h->gemm_ct.size() +
                h->gemm_bias.size() * 4 + h->gemm_leaf_value.size() * 4 + h->gemm_leaf_id.size() * 4);
  h->tree_class.assign(T, 0);
  if (d->leaf_dim == 1 && d->tree_class)
    for (int32_t t = 0; t < T; ++t) h->tree_class[t] = d->tree_class[t];
  if (d->base_score) {
    h->has_base = true;
    h->base_score.assign(d->base_score, d->base_score + d->n_outputs);
  }
  hb::EnsembleDev &E = h->ens;
  E.n_trees = T;
  E.n_features = d->n_features;
  E.n_cols = n_cols;
  E.cols = nullptr;
  E.n_outputs = d->n_outputs;
  E.leaf_dim = d->leaf_dim;
  E.aggregation = d->aggregation;
  E.transform = d->transform;
  if (device >= 0) {
    int count = 0;
    if (hipGetDeviceCount(&count) != hipSuccess || device >= count) {
      delete h;
      return fail(HB_ERR_HIP, "no such HIP device");
    }
    int prev = -1;
    (void)hipGetDevice(&prev);
    if (hipSetDevice(device) != hipSuccess) {
      delete h;
      return fail(HB_ERR_HIP, "hipSetDevice failed");
    }
    const uint32_t *pn = nullptr;
    rc = upload(h, h->tree_class, &E.tree_class);
    if (!rc && h->pruned) rc = upload(h, h->cols, &E.cols);
    if (!rc && h->has_base) rc = upload(h, h->base_score, &E.base_score);
    if (!rc && I.feasible[HB_STRATEGY_PTT]) {
      rc = upload(h, h->ptt_node, &pn);
      h->ptt.node = reinterpret_cast<const uint2 *>(pn);
      if (!rc) rc = upload(h, h->ptt_leaf_value, &h->ptt.leaf_value);
      if (!rc) rc = upload(h, h->ptt_leaf_id, &h->ptt.leaf_id);
      h->ptt.depth = D;
      if (!rc) {
        const int64_t slots = (int64_t)h->ptt_node.size() / 2 / h->info.n_trees;
        rc = upload(h, interleave64(h->ptt_node, h->info.n_trees, slots), &pn);
        h->ptt.node_il = reinterpret_cast<const uint2 *>(pn);
      }
      if (!rc) rc = upload(h, pack_leaves(h->ptt_leaf_value, h->ptt_leaf_id, d->leaf_dim), &h->ptt.leaf_pk);
      if (!rc && D >= 1 && d->leaf_dim <= 2) {
        rc = upload(h, ptt_last_level(h, D, d->leaf_dim), &pn);
        h->ptt.last_il = reinterpret_cast<const uint4 *>(pn);
      }
      if (!rc && !h->ptt_fast.empty()) {
        rc = upload(h, h->ptt_fast, &pn);
        h->ptt.fast = reinterpret_cast<const uint4 *>(pn);
        h->ptt.fast_chunks = h->ptt_fast_chunks;
        h->ptt.fast_mode = h->ptt_fast_mode;
        h->ptt.id_base = h->ptt_id_base;
        if (!rc && h->ptt_fast_mode == 3) rc = upload(h, h->ptt_fast_leafv, &h->ptt.fast_leafv);
      }
    }
    if (!rc && I.feasible[HB_STRATEGY_TT]) {
      rc = upload(h, h->tt_node, &pn);
      h->tt.node = reinterpret_cast<const uint2 *>(pn);
      if (!rc) rc = upload(h, h->tt_depth, &h->tt.depth);
      if (!rc) rc = upload(h, h->tt_leaf_value, &h->tt.leaf_value);
      if (!rc) rc = upload(h, h->tt_leaf_id, &h->tt.leaf_id);
      h->tt.n_pad = h->tt_n_pad;
      h->tt.max_depth = D;
      if (!rc) {
        rc = upload(h, interleave64(h->tt_node, h->info.n_trees, h->tt_n_pad), &pn);
        h->tt.node_il = reinterpret_cast<const uint2 *>(pn);
      }
      if (!rc) rc = upload(h, pack_leaves(h->tt_leaf_value, h->tt_leaf_id, d->leaf_dim), &h->tt.leaf_pk);
      if (!rc && !h->tt_fast.empty()) {
        if (h->tt_fast_mode == 2) {  // node blocks, leaf records apart
          rc = upload(h, h->tt_fast, &pn);
          h->tt.fast = reinterpret_cast<const uint4 *>(pn);
          if (!rc) rc = upload(h, h->tt_fast_leaf, &pn);
          h->tt.fast_leaf = reinterpret_cast<const uint2 *>(pn);
        } else {  // each tree's node records, then its leaf records
          const size_t w = (size_t)2 << h->tt_fast_lg;
          std::vector<uint32_t> blocks(2 * h->tt_fast.size());
          for (size_t t = 0; t < h->tt_fast.size() / w; ++t) {
            std::copy_n(&h->tt_fast[t * w], w, &blocks[2 * t * w]);
            std::copy_n(&h->tt_fast_leaf[t * w], w, &blocks[2 * t * w + w]);
          }
          rc = upload(h, blocks, &pn);
          h->tt.fast = reinterpret_cast<const uint4 *>(pn);
          h->tt.fast_leaf = nullptr;
        }
        h->tt.fast_mode = h->tt_fast_mode;
        h->tt.fast_lg = h->tt_fast_lg;
        h->tt.fast_chunks = h->tt_fast_chunks;
      }
    }
    if (!rc && I.feasible[HB_STRATEGY_GEMM]) {
      rc = upload(h, h->gemm_node, &pn);
      h->gemm.node = reinterpret_cast<const uint2 *>(pn);
      if (!rc) rc = upload(h, h->gemm_shape, &h->gemm.shape);
      if (!rc) rc = upload(h, h->gemm_ct, &h->gemm.ct);
      if (!rc) rc = upload(h, h->gemm_bias, &h->gemm.bias);
      if (!rc) rc = upload(h, h->gemm_leaf_value, &h->gemm.leaf_value);
      if (!rc) rc = upload(h, h->gemm_leaf_id, &h->gemm.leaf_id);
      h->gemm.k_pad = h->gemm_k_pad;
      h->gemm.l_pad = h->gemm_l_pad;
      h->gemm.n_shapes = h->gemm_n_shapes;
    }
    if (prev >= 0) (void)hipSetDevice(prev);
    if (rc) {
      std::string msg = g_last_error;
      release(h);
      return fail(rc, msg);
    }
  }
  *out = h;
  return HB_OK;
}

}  // namespace

namespace hb {
int set_error(int code, const std::string &msg) { return fail(code, msg); }
int handle_device(const hb_handle *h) { return h ? h->device : -1; }
}  // namespace hb

extern "C" {

int hb_compile(const hb_ensemble_desc *desc, int strategy_hint, int device, hb_handle **out) {
  g_last_error.clear();
  if (!out) return fail(HB_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  try {
    return compile_impl(desc, strategy_hint, device, out);
  } catch (const std::bad_alloc &) {
    return fail(HB_ERR_OOM, "out of host memory");
  } catch (...) {
    return fail(HB_ERR_INVALID_ARG, "unexpected exception in hb_compile");
  }
}

int hb_select_strategy(const hb_handle *h, int64_t n_rows) {
  if (!h) return fail(HB_ERR_INVALID_ARG, "handle is NULL");
  if (h->info.default_strategy != HB_STRATEGY_AUTO) return h->info.default_strategy;
  return select_strategy(h, n_rows);
}

int64_t hb_workspace_bytes(const hb_handle *h, int64_t n_rows, int strategy) {
  if (!h) return fail(HB_ERR_INVALID_ARG, "handle is NULL");
  if (n_rows < 0) return fail(HB_ERR_INVALID_ARG, "n_rows < 0");
  if (strategy < HB_STRATEGY_AUTO || strategy > HB_STRATEGY_PTT) return fail(HB_ERR_INVALID_ARG, "bad strategy");
  if (strategy == HB_STRATEGY_AUTO) strategy = hb_select_strategy(h, n_rows);
  const bool fast = (strategy == HB_STRATEGY_PTT && !h->ptt_fast.empty()) ||
                    (strategy == HB_STRATEGY_TT && !h->tt_fast.empty());
  // GEMM splits on its 16-row tiles: every tree one shape of 256 leaves
  const bool tiles = strategy == HB_STRATEGY_GEMM && h->gemm_n_shapes == 1 && h->gemm_k_pad == 256 &&
                     h->gemm_l_pad == 256;
  if (tiles) return hb::gemm_split_workspace_bytes(n_rows, h->info.n_trees, h->info.n_outputs);
  return fast ? hb::split_workspace_bytes(n_rows, h->info.n_trees, h->info.n_outputs) : 0;
}

int hb_predict(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids,
               int strategy, void *stream) {
  return hb_predict_ws(h, X, n_rows, scores, leaf_ids, strategy, stream, nullptr, 0);
}

}  // extern "C"

namespace {

// hb_predict_ws, or with `plan` a dry run that describes the launches instead.
int predict_impl(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids, int strategy,
                 void *stream, void *workspace, int64_t workspace_bytes, std::string *plan) {
  if (!h) return fail(HB_ERR_INVALID_ARG, "handle is NULL");
  if (workspace_bytes < 0 || (workspace_bytes > 0 && !workspace))
    return fail(HB_ERR_INVALID_ARG, "workspace_bytes > 0 needs a workspace");
  if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 7))
    return fail(HB_ERR_INVALID_ARG, "workspace must be 8-byte aligned");
  if (h->device < 0) return fail(HB_ERR_INVALID_ARG, "host-only handle: compile with a device to predict");
  if (n_rows < 0) return fail(HB_ERR_INVALID_ARG, "n_rows < 0");
  if (strategy < HB_STRATEGY_AUTO || strategy > HB_STRATEGY_PTT) return fail(HB_ERR_INVALID_ARG, "bad strategy");
  if (strategy == HB_STRATEGY_AUTO) strategy = hb_select_strategy(h, n_rows);
  if (!h->info.feasible[strategy]) return fail(HB_ERR_UNSUPPORTED, "strategy infeasible for this ensemble");
  if (n_rows == 0) return HB_OK;
  if (!plan && (!X || !scores)) return fail(HB_ERR_INVALID_ARG, "X or scores is NULL");
  if (n_rows > (int64_t)std::numeric_limits<int32_t>::max())
    return fail(HB_ERR_INVALID_ARG, "n_rows above 2^31 - 1");
  int prev = -1;
  (void)hipGetDevice(&prev);
  if (prev != h->device && hipSetDevice(h->device) != hipSuccess) return fail(HB_ERR_HIP, "hipSetDevice failed");
  std::string err;
  int rc = HB_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hb::Launch ws;
  if (workspace && workspace_bytes > 0) {
    ws.ptr = workspace;
    ws.bytes = workspace_bytes;
  }
  ws.plan = plan;
  try {
    if (strategy == HB_STRATEGY_PTT)
      rc = hb::launch_ptt(h->ens, h->ptt, X, n_rows, scores, leaf_ids, ws, s, &err);
    else if (strategy == HB_STRATEGY_TT)
      rc = hb::launch_tt(h->ens, h->tt, X, n_rows, scores, leaf_ids, ws, s, &err);
    else
      rc = hb::launch_gemm(h->ens, h->gemm, X, n_rows, scores, leaf_ids, ws, s, &err);
  } catch (...) {
    rc = HB_ERR_HIP;
    err = "unexpected exception in hb_predict";
  }
  if (prev >= 0 && prev != h->device) (void)hipSetDevice(prev);
  if (rc) return fail(rc, err);
  return HB_OK;
}

}  // namespace

extern "C" {

int hb_predict_ws(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids,
                  int strategy, void *stream, void *workspace, int64_t workspace_bytes) {
  return predict_impl(h, X, n_rows, scores, leaf_ids, strategy, stream, workspace, workspace_bytes, nullptr);
}

int hb_plan(const hb_handle *h, int64_t n_rows, int strategy, int64_t workspace_bytes, char *buf, int64_t buf_bytes) {
  if (!buf || buf_bytes < 1) return fail(HB_ERR_INVALID_ARG, "buf is NULL or empty");
  buf[0] = '\0';
  if (workspace_bytes < 0) return fail(HB_ERR_INVALID_ARG, "workspace_bytes < 0");
  std::string plan;
  // the dry run reads the workspace pointer only to test it for NULL and alignment
  void *ws = workspace_bytes > 0 ? reinterpret_cast<void *>(uintptr_t(256)) : nullptr;
  const int rc = predict_impl(const_cast<hb_handle *>(h), nullptr, n_rows, nullptr, nullptr, strategy, nullptr, ws,
                              workspace_bytes, &plan);
  if (rc) return rc;
  if ((int64_t)plan.size() >= buf_bytes) return fail(HB_ERR_INVALID_ARG, "buf too small for the plan");
  std::memcpy(buf, plan.c_str(), plan.size() + 1);
  return HB_OK;
}

int hb_query(const hb_handle *h, hb_info *info) {
  if (!h || !info) return fail(HB_ERR_INVALID_ARG, "NULL argument");
  *info = h->info;
  return HB_OK;
}

int hb_table(const hb_handle *h, int strategy, const char *name, const void **data, int64_t *bytes) {
  if (!h || !name || !data || !bytes) return fail(HB_ERR_INVALID_ARG, "NULL argument");
  if (strategy < HB_STRATEGY_GEMM || strategy > HB_STRATEGY_PTT || !h->info.feasible[strategy])
    return fail(HB_ERR_INVALID_ARG, "strategy has no tables");
  const std::string n(name);
  auto give = [&](const auto &v) {
    *data = v.data();
    *bytes = (int64_t)(v.size() * sizeof(v[0]));
    return HB_OK;
  };
  if (n == "features") return give(h->cols);
  if (strategy == HB_STRATEGY_PTT) {
    if (n == "node") return give(h->ptt_node);
    if (n == "leaf_value") return give(h->ptt_leaf_value);
    if (n == "leaf_id") return give(h->ptt_leaf_id);
  } else if (strategy == HB_STRATEGY_TT) {
    if (n == "node") return give(h->tt_node);
    if (n == "depth") return give(h->tt_depth);
    if (n == "leaf_value") return give(h->tt_leaf_value);
    if (n == "leaf_id") return give(h->tt_leaf_id);
    if (n == "dims") return give(h->tt_dims);
    if (n == "fast_node") return give(h->tt_fast);
    if (n == "fast_leaf") return give(h->tt_fast_leaf);
  } else {
    if (n == "node") return give(h->gemm_node);
    if (n == "shape") return give(h->gemm_shape);
    if (n == "ct") return give(h->gemm_ct);
    if (n == "bias") return give(h->gemm_bias);
    if (n == "leaf_value") return give(h->gemm_leaf_value);
    if (n == "leaf_id") return give(h->gemm_leaf_id);
    if (n == "dims") return give(h->gemm_dims);
  }
  return fail(HB_ERR_INVALID_ARG, "unknown table name");
}

void hb_destroy(hb_handle *h) { release(h); }

const char *hb_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
