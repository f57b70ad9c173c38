/*
 * oracle.c -- TEST INFRASTRUCTURE ONLY. A plain, slow, obviously correct CPU
 * reference for batched tree-ensemble scoring. Only the test suite, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product library
 * never links, loads or calls it, and the two share no source.
 *
 * What it computes (Hummingbird, "A Tensor Compiler for Unified Machine
 * Learning Prediction Serving", Sec. 4.1 "Compiling Tree-based Models"):
 * the three compilation strategies of that section (GEMM, Algorithm 1;
 * TreeTraversal, Algorithm 2; PerfectTreeTraversal, Algorithm 3) are exact
 * reformulations of the ordinary walk from the root to a leaf: GEMM returns
 * the leaf selected by the encoded path, TreeTraversal iterates until every
 * record has reached its leaf, and the perfect-tree padding keeps the tree's
 * function unchanged. The oracle is therefore that plain definition written
 * out: for every row and every tree, start at the root and follow the
 * decision rule "x[feature] < threshold goes left" (Sec. 4.1 assumes every
 * decision node performs a strict < comparison) until a leaf is reached.
 *
 * Readings of the paper used here (each listed in the design notes):
 *  - ties x == t go right (strict <), NaN goes right (IEEE: NaN < t is false)
 *    unless the caller gives the node a default direction: the paper leaves
 *    missing values to future work (Sec. 4.1 notes they are not supported
 *    yet), and this extension follows the common per-node "missing values go
 *    left" flag of tree learners;
 *  - categorical splits (also future work in Sec. 4.1): a node may carry a
 *    category set, a bit set of 32-bit words (bit j of word w is category
 *    32 w + j); the category of a row is the integer part of a non-negative
 *    feature value below 32 times the word count, and the row goes left when
 *    the set holds it; every other value goes right, and NaN is missing as
 *    above;
 *  - the reported leaf index is the caller's local node id of the leaf;
 *  - ensemble aggregation is SUM or MEAN (the paper's ReduceMean) over
 *    trees, per output column, plus an optional base score; the paper's
 *    classification output is then optionally passed through sigmoid or a
 *    max-subtracted softmax (Table 2 lists Sigmoid and Softmax among the
 *    tensor operators used);
 *  - accumulation and transforms run in double precision.
 *
 * Parity status: leaf ids are pinned by hand-traced trees, brute-force path
 * enumeration, the GEMM closed form of Table 3 and scikit-learn's apply();
 * scores by closed forms and scikit-learn's predict/predict_proba.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_ERR_ARG -1
#define ORACLE_ERR_CYCLE -2  /* walk longer than the tree's node count */
#define ORACLE_ERR_CHILD -3  /* child id outside the tree */
#define ORACLE_ERR_FEATURE -4

#define ORACLE_AGG_SUM 0
#define ORACLE_AGG_MEAN 1
#define ORACLE_POST_NONE 0
#define ORACLE_POST_SIGMOID 1
#define ORACLE_POST_SOFTMAX 2

typedef struct {
  int32_t n_trees, n_features, n_outputs, leaf_dim;
  const int64_t *tree_node_offset; /* [n_trees + 1] */
  const int32_t *feature;          /* [nodes], < 0 marks a leaf */
  const float *threshold;          /* [nodes] */
  const int32_t *left, *right;     /* [nodes], tree-local ids */
  const float *leaf_value;         /* [nodes * leaf_dim] */
  const int32_t *tree_class;       /* [n_trees] or NULL */
  int32_t aggregation, transform;
  const float *base_score;         /* [n_outputs] or NULL */
  const uint8_t *default_left;     /* [nodes] or NULL: NaN goes left where 1 */
  const int64_t *cat_offset;       /* [nodes + 1] or NULL: node i's category set is
                                      cat_bits[cat_offset[i] .. cat_offset[i + 1]) */
  const uint32_t *cat_bits;
  const float *X;                  /* [n_rows, n_features] row-major */
  int64_t n_rows;
  double *raw;                     /* [n_rows, n_outputs] before transform */
  double *out;                     /* [n_rows, n_outputs] after transform */
  int32_t *leaf_ids;               /* [n_rows, n_trees] or NULL */
} oracle_job;

/* Walk one tree for one row; returns the local leaf id or a negative error. */
static int64_t walk(const oracle_job *J, int32_t t, const float *x) {
  const int64_t base = J->tree_node_offset[t];
  const int64_t count = J->tree_node_offset[t + 1] - base;
  int64_t v = 0; /* the root is local node 0 */
  int64_t steps = 0;
  while (J->feature[base + v] >= 0) {
    int32_t f = J->feature[base + v];
    if (f >= J->n_features) return ORACLE_ERR_FEATURE;
    if (++steps > count) return ORACLE_ERR_CYCLE;
    /* Sec. 4.1: every decision node performs a strict < comparison; a
       missing (NaN) value follows the node's default direction if given. */
    const int64_t node = base + v;
    if (J->default_left && isnan(x[f]))
      v = J->default_left[node] ? J->left[node] : J->right[node];
    else if (J->cat_offset && J->cat_offset[node + 1] > J->cat_offset[node]) {
      /* categorical node: left when the set holds the row's category */
      const int64_t words = J->cat_offset[node + 1] - J->cat_offset[node];
      int in_set = 0;
      if (x[f] >= 0.0f && (double)x[f] < 32.0 * (double)words) {
        const int64_t c = (int64_t)x[f]; /* integer part */
        in_set = (J->cat_bits[J->cat_offset[node] + c / 32] >> (c % 32)) & 1u;
      }
      v = in_set ? J->left[node] : J->right[node];
    } else if (x[f] < J->threshold[base + v])
      v = J->left[base + v];
    else
      v = J->right[base + v];
    if (v < 0 || v >= count) return ORACLE_ERR_CHILD;
  }
  return v;
}

typedef struct {
  const oracle_job *J;
  int64_t r0, r1;
  int status;
} oracle_slice;

static void *run_slice(void *arg) {
  oracle_slice *S = (oracle_slice *)arg;
  const oracle_job *J = S->J;
  const int32_t K = J->n_outputs;
  double *acc = (double *)malloc(sizeof(double) * (size_t)K);
  if (!acc) {
    S->status = ORACLE_ERR_ARG;
    return NULL;
  }
  S->status = ORACLE_OK;
  for (int64_t r = S->r0; r < S->r1; ++r) {
    const float *x = J->X + r * (int64_t)J->n_features;
    for (int32_t k = 0; k < K; ++k) acc[k] = 0.0;
    for (int32_t t = 0; t < J->n_trees; ++t) {
      int64_t leaf = walk(J, t, x);
      if (leaf < 0) {
        S->status = (int)leaf;
        free(acc);
        return NULL;
      }
      if (J->leaf_ids) J->leaf_ids[r * (int64_t)J->n_trees + t] = (int32_t)leaf;
      const int64_t node = J->tree_node_offset[t] + leaf;
      if (J->leaf_dim == 1) {
        int32_t c = J->tree_class ? J->tree_class[t] : 0;
        acc[c] += (double)J->leaf_value[node];
      } else {
        for (int32_t k = 0; k < K; ++k)
          acc[k] += (double)J->leaf_value[node * J->leaf_dim + k];
      }
    }
    double *raw = J->raw + r * (int64_t)K;
    double *out = J->out + r * (int64_t)K;
    for (int32_t k = 0; k < K; ++k) {
      double s = acc[k];
      if (J->aggregation == ORACLE_AGG_MEAN) s /= (double)J->n_trees;
      if (J->base_score) s += (double)J->base_score[k];
      raw[k] = s;
    }
    if (J->transform == ORACLE_POST_SIGMOID) {
      for (int32_t k = 0; k < K; ++k) out[k] = 1.0 / (1.0 + exp(-raw[k]));
    } else if (J->transform == ORACLE_POST_SOFTMAX) {
      double m = raw[0];
      for (int32_t k = 1; k < K; ++k)
        if (raw[k] > m) m = raw[k];
      double z = 0.0;
      for (int32_t k = 0; k < K; ++k) {
        out[k] = exp(raw[k] - m);
        z += out[k];
      }
      for (int32_t k = 0; k < K; ++k) out[k] /= z;
    } else {
      for (int32_t k = 0; k < K; ++k) out[k] = raw[k];
    }
  }
  free(acc);
  return NULL;
}

/*
 * Score n_rows rows against every tree. Returns 0, or a negative code for an
 * invalid argument or an ill-formed tree met during a walk. n_threads <= 0
 * uses one thread.
 */
int oracle_predict(int32_t n_trees, int32_t n_features, int32_t n_outputs,
                   int32_t leaf_dim, const int64_t *tree_node_offset,
                   const int32_t *feature, const float *threshold,
                   const int32_t *left, const int32_t *right,
                   const float *leaf_value, const int32_t *tree_class,
                   int32_t aggregation, int32_t transform,
                   const float *base_score, const uint8_t *default_left,
                   const int64_t *cat_offset, const uint32_t *cat_bits,
                   const float *X, int64_t n_rows,
                   double *raw, double *out, int32_t *leaf_ids,
                   int32_t n_threads) {
  if (n_trees < 1 || n_features < 1 || n_outputs < 1 || n_rows < 0) return ORACLE_ERR_ARG;
  if (leaf_dim != 1 && leaf_dim != n_outputs) return ORACLE_ERR_ARG;
  if (!tree_node_offset || !feature || !threshold || !left || !right || !leaf_value)
    return ORACLE_ERR_ARG;
  if (n_rows > 0 && (!X || !raw || !out)) return ORACLE_ERR_ARG;
  if (aggregation != ORACLE_AGG_SUM && aggregation != ORACLE_AGG_MEAN) return ORACLE_ERR_ARG;
  if (transform < ORACLE_POST_NONE || transform > ORACLE_POST_SOFTMAX) return ORACLE_ERR_ARG;
  for (int32_t t = 0; t < n_trees; ++t)
    if (tree_node_offset[t + 1] <= tree_node_offset[t]) return ORACLE_ERR_ARG;
  if (cat_offset) {
    const int64_t n_nodes = tree_node_offset[n_trees];
    if (cat_offset[0] < 0 || (!cat_bits && cat_offset[n_nodes] > 0)) return ORACLE_ERR_ARG;
    for (int64_t i = 0; i < n_nodes; ++i)
      if (cat_offset[i + 1] < cat_offset[i]) return ORACLE_ERR_ARG;
  }
  if (leaf_dim == 1 && tree_class) {
    for (int32_t t = 0; t < n_trees; ++t)
      if (tree_class[t] < 0 || tree_class[t] >= n_outputs) return ORACLE_ERR_ARG;
  }
  if (n_rows == 0) return ORACLE_OK;

  oracle_job J = {n_trees, n_features, n_outputs, leaf_dim, tree_node_offset,
                  feature, threshold, left, right, leaf_value, tree_class,
                  aggregation, transform, base_score, default_left, cat_offset, cat_bits, X, n_rows,
                  raw, out, leaf_ids};
  if (n_threads < 1) n_threads = 1;
  if ((int64_t)n_threads > n_rows) n_threads = (int32_t)n_rows;
  oracle_slice *slices = (oracle_slice *)calloc((size_t)n_threads, sizeof(oracle_slice));
  pthread_t *tids = (pthread_t *)calloc((size_t)n_threads, sizeof(pthread_t));
  char *spawned = (char *)calloc((size_t)n_threads, 1);
  if (!slices || !tids || !spawned) {
    free(slices);
    free(tids);
    free(spawned);
    return ORACLE_ERR_ARG;
  }
  const int64_t per = (n_rows + n_threads - 1) / n_threads;
  for (int32_t i = 0; i < n_threads; ++i) {
    slices[i].J = &J;
    slices[i].r0 = (int64_t)i * per;
    slices[i].r1 = slices[i].r0 + per < n_rows ? slices[i].r0 + per : n_rows;
    slices[i].status = ORACLE_OK;
    if (slices[i].r0 >= slices[i].r1) continue;
    if (i > 0 && pthread_create(&tids[i], NULL, run_slice, &slices[i]) == 0) spawned[i] = 1;
  }
  /* slice 0, and any slice whose thread could not be spawned, runs here */
  for (int32_t i = 0; i < n_threads; ++i)
    if (!spawned[i] && slices[i].r0 < slices[i].r1) run_slice(&slices[i]);
  for (int32_t i = 0; i < n_threads; ++i)
    if (spawned[i]) pthread_join(tids[i], NULL);
  int status = ORACLE_OK;
  for (int32_t i = 0; i < n_threads; ++i)
    if (slices[i].status != ORACLE_OK) status = slices[i].status;
  free(slices);
  free(tids);
  free(spawned);
  return status;
}
