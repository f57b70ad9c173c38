/*
 * hb.h -- batched tree-ensemble inference on AMD Instinct MI355X (gfx950).
 *
 * A trained ensemble of binary decision trees (gradient-boosted trees or a
 * random forest) is compiled once into device-resident tensors and then
 * scores batches of rows, every row against every tree. This follows the
 * problem statement of Sec. 4.1 ("Compiling Tree-based Models") of
 * Nakandala et al., "A Tensor Compiler for Unified Machine Learning
 * Prediction Serving" (OSDI 2020): input records X in R^{n x |F|}, one
 * prediction per record; trees over numerical features whose decision nodes
 * all perform x[f] < threshold (true goes to the left child). Three
 * compilation strategies are provided, each an exact reformulation of the
 * plain root-to-leaf walk:
 *
 *   HB_STRATEGY_GEMM  Algorithm 1 with the tensors of Table 3: all decision
 *                     nodes evaluated, the path encoded by a 0/+-1 matrix
 *                     product (int8 matrix cores) and matched against D.
 *   HB_STRATEGY_TT    Algorithm 2 (TreeTraversal) with the tensors of Table 5:
 *                     level-synchronous descent through child arrays.
 *   HB_STRATEGY_PTT   Algorithm 3 (PerfectTreeTraversal) with the tensors of
 *                     Table 6: trees padded to perfect trees, children found
 *                     by heap arithmetic.
 *   HB_STRATEGY_AUTO  the selector of Sec. 5.1 re-derived for this device,
 *                     keyed on depth, balance and batch size.
 *
 * All functions are thread-safe except that a handle must not be destroyed
 * while another call uses it. No C++ exception crosses this interface. Every
 * non-zero return leaves a message for hb_last_error() on the calling thread.
 */
#ifndef HB_H_
#define HB_H_

#include <stdint.h>

/* The library is built with hidden visibility; only these entry points are
 * exported. */
#define HB_API __attribute__((visibility("default")))

#ifdef __cplusplus
extern "C" {
#endif

/* ---- return codes ------------------------------------------------------- */
#define HB_OK 0
#define HB_ERR_INVALID_ARG (-1)   /* NULL pointer, bad size, bad enum value */
#define HB_ERR_INVALID_MODEL (-2) /* not a tree: cycle, shared or unreachable
                                     node, child/feature out of range, NaN
                                     threshold, bad class id */
#define HB_ERR_UNSUPPORTED (-3)   /* strategy infeasible for this ensemble
                                     (depth or size limits below) */
#define HB_ERR_OOM (-4)           /* host or device allocation failed */
#define HB_ERR_HIP (-5)           /* a HIP runtime call or launch failed */

/* ---- enums -------------------------------------------------------------- */
enum hb_strategy {
  HB_STRATEGY_AUTO = 0,
  HB_STRATEGY_GEMM = 1,
  HB_STRATEGY_TT = 2,
  HB_STRATEGY_PTT = 3
};
/* Ensemble aggregation over trees, per output column: SUM, or MEAN (the
 * paper's ReduceMean over the batched tree dimension, Sec. 4.1). */
enum hb_aggregation { HB_AGG_SUM = 0, HB_AGG_MEAN = 1 };
/* Post-transform of the aggregated margin (Table 2 lists Sigmoid and
 * Softmax among the tensor operators used). Softmax subtracts the row max. */
enum hb_transform { HB_POST_NONE = 0, HB_POST_SIGMOID = 1, HB_POST_SOFTMAX = 2 };

/* ---- limits ------------------------------------------------------------- */
#define HB_MAX_OUTPUTS 16          /* n_outputs (columns of the score)      */
#define HB_PTT_MAX_DEPTH 12        /* PTT tables grow as 2^depth per tree   */
#define HB_TT_MAX_NODES 65535      /* nodes per tree for TT (16-bit ids)    */
#define HB_MAX_FEATURES 65535      /* features (16-bit ids in TT records)   */
#define HB_MAX_CATEGORY_WORDS 65536 /* words of one node's category set      */
#define HB_GEMM_MAX_LEAVES 256     /* leaves per tree for GEMM              */
#define HB_MAX_TREES (1 << 24)     /* n_trees (kernels index eight rows of
                                      leaf ids with 32-bit offsets)          */

/*
 * The ensemble, in host memory, owned by the caller and only read (copied)
 * by hb_compile. Tree t owns nodes [tree_node_offset[t], tree_node_offset[t+1])
 * of every per-node array; node ids inside a tree are local (0 .. count-1)
 * and local node 0 is the root. A node is a leaf iff feature < 0.
 */
typedef struct hb_ensemble_desc {
  int32_t n_trees;                 /* 1 .. HB_MAX_TREES                      */
  int32_t n_features;              /* >= 1, columns of X                     */
  int32_t n_outputs;               /* K: 1 .. HB_MAX_OUTPUTS                 */
  int32_t leaf_dim;                /* 1 (scalar leaves) or n_outputs         */
  const int64_t *tree_node_offset; /* [n_trees + 1], strictly increasing, [0] == 0 */
  const int32_t *feature;          /* [nodes] in [0, n_features), -1 at leaves */
  const float *threshold;          /* [nodes]; read at internal nodes only   */
  const int32_t *left;             /* [nodes] local child id, -1 at leaves   */
  const int32_t *right;            /* [nodes] local child id, -1 at leaves   */
  const float *leaf_value;         /* [nodes * leaf_dim]; read at leaves only */
  const int32_t *tree_class;       /* [n_trees] output column of each tree when
                                      leaf_dim == 1; NULL means column 0     */
  int32_t aggregation;             /* enum hb_aggregation                    */
  int32_t transform;               /* enum hb_transform                      */
  const float *base_score;         /* [n_outputs] added after aggregation, or NULL */
  const uint8_t *default_left;     /* [nodes] or NULL; read at internal nodes only.
                                      Missing values: a NaN feature value goes to
                                      the left child where this is 1 and to the
                                      right child where it is 0 (NULL: right
                                      everywhere, which is also what x < t gives
                                      for NaN). Values other than 0/1 are
                                      HB_ERR_INVALID_MODEL; a 1 on a node whose
                                      threshold is -inf is HB_ERR_UNSUPPORTED.
                                      The paper leaves missing values to future
                                      work (Sec. 4.1); this is the per-node
                                      default direction of common tree learners. */
  const int64_t *cat_offset;       /* [nodes + 1] or NULL. Categorical splits: the
                                      category set of internal node i is the bit set
                                      cat_bits[cat_offset[i] .. cat_offset[i + 1])
                                      (bit j of word w is category 32 w + j); an
                                      empty range makes the node numeric (x < t).
                                      A row's category is the integer part of a
                                      non-negative feature value below 32 times the
                                      word count; it goes left when the set holds
                                      that category and right otherwise (negative
                                      values, +inf and values past the bit set go
                                      right); NaN follows default_left as for a
                                      numeric node. The threshold of a categorical
                                      node is not read. Offsets must start at 0 and
                                      not decrease, and a node may hold at most
                                      HB_MAX_CATEGORY_WORDS words
                                      (HB_ERR_INVALID_MODEL otherwise). The paper
                                      leaves categorical values to future work
                                      (Sec. 4.1); this is the category-set split of
                                      common tree learners. */
  const uint32_t *cat_bits;        /* [cat_offset[nodes]] words, or NULL when
                                      cat_offset is NULL                       */
} hb_ensemble_desc;

typedef struct hb_handle hb_handle;

typedef struct hb_info {
  int32_t n_trees, n_features, n_outputs, leaf_dim;
  int32_t max_depth;               /* max internal nodes on a root-leaf path */
  int32_t device;                  /* HIP device id, or -1 for a host-only handle */
  int64_t n_nodes, n_internal, n_leaves;
  double balance;                  /* sum_t (2^D - 1) / sum_t internal_t, D = max_depth */
  int32_t default_strategy;        /* hint given to hb_compile               */
  int32_t feasible[4];             /* indexed by enum hb_strategy (AUTO = 1) */
  int64_t table_bytes[4];          /* bytes of compiled tensors per strategy */
  int32_t gemm_shapes;             /* distinct tree shapes (C/D matrices)    */
  int32_t ptt_depth;               /* D used by PTT (= max_depth)            */
  int32_t n_used_features;         /* feature columns the kernels stage: the
                                      input columns some decision node tests,
                                      one more for each column that nodes with
                                      default_left = 1 test, one for each
                                      distinct (column, category set,
                                      default_left) of categorical nodes;
                                      n_features (all columns, in order) when
                                      no node is categorical or sends missing
                                      values left and pruning would drop less
                                      than a quarter of them */
} hb_info;

/*
 * Compile an ensemble. Validates the trees, renumbers each breadth-first
 * (children adjacent), builds the tensors of every feasible strategy
 * (Tables 3, 5 and 6) and, for device >= 0, uploads them to that HIP device
 * with synchronous copies. device == -1 builds a host-only handle whose
 * tensors can be inspected with hb_table() but which hb_predict rejects.
 * strategy_hint becomes the handle's default strategy (AUTO allowed); a
 * forced hint that is infeasible returns HB_ERR_UNSUPPORTED.
 * On success *out owns all device memory; release it with hb_destroy.
 */
HB_API int hb_compile(const hb_ensemble_desc *desc, int strategy_hint, int device, hb_handle **out);

/*
 * Score n_rows rows. X, scores and leaf_ids are device pointers on the
 * handle's device:
 *   X        float32 [n_rows, n_features], row-major, contiguous, read only;
 *   scores   float32 [n_rows, n_outputs], row-major: the aggregated margin
 *            after the transform;
 *   leaf_ids int32 [n_rows, n_trees], row-major, or NULL to skip: the
 *            caller's local node id of the leaf each row reaches in each tree
 *            (the same for every strategy).
 * strategy: HB_STRATEGY_AUTO uses the handle's default, or the selector when
 * that is AUTO too. The work is enqueued on `stream` (a hipStream_t; NULL is
 * the default stream) without any host synchronisation; launch errors are
 * reported, execution errors surface on the stream. n_rows == 0 returns
 * HB_OK and enqueues nothing. Concurrent calls on one handle are allowed:
 * the compiled tensors are read only and no scratch memory is shared.
 */
HB_API int hb_predict(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids,
               int strategy, void *stream);

/*
 * hb_predict with an optional device workspace (8-byte aligned, on the
 * handle's device, owned by the caller, not shared with any call that may
 * run concurrently). With a workspace of at least
 * hb_workspace_bytes(h, n_rows, strategy) bytes, batches of up to 65,536
 * rows on PTT or TT divide the trees of each row tile among several
 * workgroups (the walk of a small batch otherwise occupies few compute
 * units) and add the partial sums in a fixed order in a second kernel, so
 * results are reproducible run to run. A NULL workspace (or 0 bytes) is
 * exactly hb_predict; a smaller one is used only where it suffices. The
 * workspace holds nothing between calls. Errors as hb_predict, plus
 * HB_ERR_INVALID_ARG for workspace_bytes < 0, a NULL workspace with
 * workspace_bytes > 0, or a misaligned workspace.
 */
HB_API int hb_predict_ws(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids,
                  int strategy, void *stream, void *workspace, int64_t workspace_bytes);

/*
 * hb_predict_ws for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the workspace is the library's own static device scratch of
 * HB_SCRATCH_BYTES bytes, one copy per GPU, held from the first such call on
 * a device until the process ends. scratch_bytes (0 .. HB_SCRATCH_BYTES) is
 * how much of it the call may use, as workspace_bytes in hb_predict_ws (e.g.
 * hb_workspace_bytes(), capped at HB_SCRATCH_BYTES; the split then uses the
 * most parts whose partial sums fit). Allocates nothing: no hipMalloc, no
 * hipFree. Every call on a GPU shares that GPU's scratch, so calls that may
 * overlap on one device (other streams, other threads) race and must be
 * serialised by the caller; the scratch keeps the last call's partial sums,
 * which a call overwrites before reading. Errors as hb_predict_ws, plus
 * HB_ERR_INVALID_ARG for scratch_bytes outside [0, HB_SCRATCH_BYTES], and
 * HB_ERR_HIP if the scratch's device address cannot be obtained.
 */
#define HB_SCRATCH_BYTES ((int64_t)32 << 20)
HB_API int hb_predict_scratch(hb_handle *h, const float *X, int64_t n_rows, float *scores, int32_t *leaf_ids,
                              int strategy, void *stream, int64_t scratch_bytes);

/* Workspace bytes that let hb_predict_ws split the trees of a batch of
 * n_rows rows under `strategy` (AUTO: the selector's choice); 0 when that
 * batch never splits. A negative value is an error code. The split serves
 * the small batches of request-response serving, for which the paper
 * measures latency per batch size (Sec. 6, batch-size and request-response
 * experiments); the paper's own kernels have no such scratch. */
HB_API int64_t hb_workspace_bytes(const hb_handle *h, int64_t n_rows, int strategy);

/* The strategy hb_predict would run for this batch size under AUTO: the
 * selector of Sec. 5.1 ("Execution Strategy Selection"), which picks among
 * GEMM, TreeTraversal and PerfectTreeTraversal by tree depth and batch
 * size, re-measured on this device: PTT while it holds the trees (depth up
 * to HB_PTT_MAX_DEPTH) and they are near-perfect (balance <= 4) or the
 * batch is small (<= 256 rows), TT otherwise; GEMM only when forced or when
 * nothing else holds the model. Returns the enum value, or a negative error
 * code for a NULL handle. */
HB_API int hb_select_strategy(const hb_handle *h, int64_t n_rows);

/* Shape statistics, feasibility and table sizes of a compiled handle: the
 * quantities Table 4 states the strategies' costs in (trees, depth, internal
 * and leaf node counts, the perfect-tree padding that PTT's O(2^D) memory
 * implies) and the bytes each strategy's tensors take. Returns HB_OK or
 * HB_ERR_INVALID_ARG for a NULL argument. */
HB_API int hb_query(const hb_handle *h, hb_info *info);

/*
 * Host copy of one compiled tensor (the tensors of Table 3 for GEMM, Table 5
 * for TT and Table 6 for PTT, in the layouts below), for inspection and
 * testing: *data points
 * into memory owned by the handle (valid until hb_destroy), *bytes is its
 * size. Names per strategy:
 *   PTT : "node" (uint32 pairs {threshold bits, feature} per tree, max(2^D, 2)
 *         heap slots, slot 0 unused), "leaf_value" (float [T][2^D][leaf_dim]),
 *         "leaf_id" (int32 [T][2^D])
 *   TT  : "node" (uint32 pairs {threshold bits, feature | right << 16} per
 *         tree, n_pad slots, n_pad even; a leaf holds {-inf, own id << 16}),
 *         "depth" (int32 [T]), "leaf_value"
 *         (float [T][n_pad][leaf_dim]), "leaf_id" (int32 [T][n_pad]),
 *         "dims" (int32 {n_pad}), and the row-parallel kernels' packed form:
 *         "fast_node" (uint32 pairs per tree, trees padded to a multiple of
 *         32, 2^lg records each: {threshold bits, feature | 8 * right << 16};
 *         leaves and padding trees hold {-inf, 8 * own index << 16}),
 *         "fast_leaf" (uint32 pairs {value bits, caller id} per record of
 *         "fast_node"); empty when the model has vector leaves or lg > 11.
 *         On the device the leaf records stay a separate array while they
 *         take at most 4 MB, and follow each tree's node records otherwise
 *   GEMM: "node" (uint32 pairs {threshold bits, feature} [T][k_pad]),
 *         "shape" (int32 [T]), "ct" (int8 [S][l_pad][k_pad], 4*C^T),
 *         "bias" (int32 [S][l_pad]), "leaf_value" (float [T][l_pad][leaf_dim]),
 *         "leaf_id" (int32 [T][l_pad]), "dims" (int32 {k_pad, l_pad, S})
 *   any : "features" (int32: n_used_features entries, one per feature index
 *         the tables above use: the input column in bits 0-28; bit 30 set
 *         means a NaN input goes left (a numeric index reads it as -inf);
 *         bit 29 set means the index is the 0/1 indicator of a category set
 *         (0 where the row goes left; its nodes test it against 0.5) and bits
 *         0-28 are the offset, in entries from the start of this array, of
 *         its descriptor {input column, word count W, W words of the set};
 *         the descriptors follow the n_used_features entries. Unless this is
 *         the identity, the tables hold these indices instead of input
 *         columns)
 * Returns HB_ERR_INVALID_ARG for an unknown name or an infeasible strategy.
 */
HB_API int hb_table(const hb_handle *h, int strategy, const char *name, const void **data, int64_t *bytes);

/*
 * Dry run of hb_predict_ws: writes into buf (NUL-terminated, at most
 * buf_bytes bytes including the NUL) the kernels a call with this batch size,
 * strategy and workspace size would launch, in launch order, separated by
 * "; ", each as "name grid=(x,y) block=b lds=bytes" with name the kernel
 * template instantiation as a profiler prints it. Launches nothing and needs
 * no buffers; the handle must be a device handle. Errors: those of
 * hb_predict_ws, HB_ERR_INVALID_ARG for a NULL or too small buf. This
 * reports the launch plan behind the selector of Sec. 5.1.
 */
HB_API int hb_plan(const hb_handle *h, int64_t n_rows, int strategy, int64_t workspace_bytes, char *buf,
                   int64_t buf_bytes);

/* Synchronise the handle's device and free everything it owns. NULL is a no-op. */
HB_API void hb_destroy(hb_handle *h);

/* Message for the last non-zero return on this thread ("" if none). */
HB_API const char *hb_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HB_H_ */
