// hb_internal.h -- shared between the host compiler (hb_api.cpp) and the
// device kernels (hb_kernels.hip): device views of the compiled tensors and
// the launcher entry points. Not part of the public C-ABI.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "hb.h"

namespace hb {

// Largest per-tree table the traversal kernels can stage: the 160 KiB of LDS
// of a gfx950 CU less the leaf-id staging buffer.
constexpr int64_t kTreeLdsLimit = 160 * 1024 - 4 * 1024;

// Packed per-tree blocks for the fast traversal kernels (scalar leaves).
// Node and leaf records are 8 bytes; a leaf record is {value bits, caller id}.
//   PTT (mode 0, lg = D): the block holds 2^D node records followed by 2^D
//     leaf records: node record p = {threshold bits, feature} for heap index
//     p in [1, 2^D) (slot 0 unused); the leaf record of heap index a in
//     [2^D, 2^(D+1)) sits at byte 8a of the block.
//   TT (2^lg >= nodes): node record c = {threshold bits, feature | 8 * right
//     child << 16} (children adjacent: left = right - 1; a leaf holds
//     threshold -inf and points to itself), leaf record c for node c.
//     Mode 1: the block holds the 2^lg node records followed by the 2^lg
//     leaf records, all staged through LDS. Mode 2: the block holds the node
//     records only, and the leaf records live in a separate array
//     [trees][2^lg] read from global memory once per walk, so a chunk holds
//     twice the trees; used while that array fits in an XCD's L2.
//   PTT mode 3 (lg = D <= 8; scalar leaves whose caller ids are the leaf slot
//     plus one base, as in heap-ordered perfect trees): the block holds the
//     node records only; the leaf values live in a float array [trees][2^D]
//     read from global memory once per walk, and the ids are formed from
//     the slots.
// Blocks are grouped in chunks of fast_tc() trees staged through LDS, either
// double-buffered (the next chunk is stored while nobody reads its buffer) or
// single-buffered with twice as many trees per chunk (more independent walks
// per wave, one extra barrier per chunk), whichever fits more trees in the
// kernel's table budget (64 or 32 KiB). Leaf ids are held for the last
// kFastIdGroup trees, and the tree count is padded with zero blocks to a
// multiple of kFastIdGroup (so every chunk size divides it).
constexpr int kFastTableLds = 64 * 1024;
constexpr int kFastIdGroup = 32;
// The fast kernels hold and stage leaf ids as 16-bit halves (mode 3: byte
// slots, half the staging): every caller id they report is a local node id
// of a tree with at most 2^(kFastMaxLg + 1) nodes. Each wave stages up to 16
// of its 64 rows at a time (the 32 ids of one 128-byte output line per row,
// for two lines), so the staging costs 16 bytes per row of a workgroup.
constexpr int kFastIdStageBytes = 2 * 8 * kFastIdGroup * 2 / 64;
constexpr int fast_node_bytes(int mode) { return (void)mode, 8; }
// modes 2 (TT) and 3 (PTT) keep the leaves apart, in global memory
constexpr int fast_tree_bytes(int mode, int lg) { return (1 << lg) * (fast_node_bytes(mode) + (mode >= 2 ? 0 : 8)); }
// TT leaf records up to this size stay in global memory (mode 2); measured
// on 1M rows: leaf-wise 500 trees (2 MB) 5.1 -> 3.9 ms, 3500 depth-8 trees
// (14 MB, L2 misses on every leaf read) 16.6 -> 21.6 ms.
constexpr int64_t kTtLeafGlobalMax = (int64_t)4 << 20;
constexpr int fast_pow2_fit(int budget, int tree_bytes) {
  int t = 16;
  while (t > 1 && t * tree_bytes > budget) t >>= 1;
  return t;
}
constexpr bool fast_single(int tree_bytes, int budget = kFastTableLds) {
  return fast_pow2_fit(budget, tree_bytes) > fast_pow2_fit(budget / 2, tree_bytes);
}
constexpr int fast_bufs(int tree_bytes, int budget = kFastTableLds) { return fast_single(tree_bytes, budget) ? 1 : 2; }
constexpr int fast_tc(int tree_bytes, int budget = kFastTableLds) {
  return fast_pow2_fit(budget / fast_bufs(tree_bytes, budget), tree_bytes);
}
// PTT with the leaves in global memory (mode 3) always double-buffers: its
// blocks are half the size, so the same budget holds two chunks of the
// trees a mode-0 chunk holds, and a chunk needs one barrier instead of two.
constexpr int fast_bufs_m(int mode, int tree_bytes, int budget = kFastTableLds) {
  return mode == 3 ? 2 : fast_bufs(tree_bytes, budget);
}
constexpr int fast_tc_m(int mode, int tree_bytes, int budget = kFastTableLds) {
  return mode == 3 ? fast_pow2_fit(budget / 2, tree_bytes) : fast_tc(tree_bytes, budget);
}
// Kernels with the half budget trade chunk size for occupancy: wider
// workgroups, or wider feature tiles, leave room for half the chunk. Blocks
// are contiguous per tree, so a kernel with a smaller chunk walks the same
// packed buffer (the padded tree count is a multiple of every chunk size).
constexpr int kFastTableSmall = kFastTableLds / 2;
constexpr int kFastMaxLg = 12;
static_assert(kFastMaxLg < 15, "fast-kernel leaf ids must fit in 16 bits");

// Ensemble-wide parameters every kernel needs.
// Feature-tile column flags (in EnsembleDev::cols): kColNanLeft: a NaN input
// value goes left (a numeric column reads it as -inf); kColCat: the column is
// the 0/1 category-set indicator of categorical nodes (0 when the row goes
// left), and the low bits are the int offset, from the start of cols, of its
// descriptor {input column, word count W, W words of the set}, which follow
// the n_cols column entries. Otherwise the low bits are the input column.
constexpr int32_t kColNanLeft = 1 << 30;
constexpr int32_t kColCat = 1 << 29;
constexpr int32_t kColMask = kColCat - 1;

struct EnsembleDev {
  int32_t n_trees, n_features, n_outputs, leaf_dim;
  // Feature tile: the kernels stage n_cols columns per row; column i is input
  // column cols[i] & kColMask, read with NaN -> -inf when kColNanLeft is set,
  // or a category-set indicator when kColCat is set (cols == nullptr: the
  // identity, n_cols == n_features). n_features stays the row stride of X.
  int32_t n_cols;
  const int32_t *cols;
  int32_t aggregation, transform;
  const int32_t *tree_class;  // [T] device; output column of a scalar-leaf tree
  const float *base_score;    // [K] device, or nullptr
};

// Interleaved node records (node_il) serve the trees-across-lanes kernel, in
// which lane l of a wave walks tree 64 g + l: slot p of the 64 trees of group
// g is 64 consecutive records, so lanes at the same slot share cache lines
// (the paper batches the trees' tensors level by level in the same spirit).
// The same kernel reads a leaf through one packed record (leaf_pk):
// [T][leaf slots][leaf_pk_words(leaf_dim)] 32-bit words, the leaf_dim values
// then the caller id, padded to a power of two so a record never straddles a
// 128-byte line.
// For perfect trees with leaf_dim <= 2 the last decision level and the two
// leaves under each of its nodes form one 32-byte record (last_il), so the
// final step and the leaf read are one access:
// [ceil(T/64)][2^(D-1)][64][8 words] = {threshold bits, feature, left leaf,
// right leaf}, a leaf being {value, caller id} (leaf_dim 1, then two zero
// words) or {value 0, value 1, caller id} (leaf_dim 2).
constexpr int kLastWords = 8;
constexpr int leaf_pk_words(int leaf_dim) {
  int w = 2;
  while (w < leaf_dim + 1) w *= 2;
  return w;
}

// PerfectTreeTraversal tensors (Table 6, Algorithm 3), 1-based heap per tree:
// slot p in [1, 2^D) is a decision node, the children of p are 2p and 2p+1,
// and after D steps the index lies in [2^D, 2^(D+1)); leaf slot = index - 2^D.
struct PttDev {
  const uint2 *node;        // [T][2^D] {threshold bits, feature}; slot 0 unused
  const float *leaf_value;  // [T][2^D][leaf_dim]
  const int32_t *leaf_id;   // [T][2^D] caller-local node id
  int32_t depth;            // D
  const uint2 *node_il;     // [ceil(T/64)][2^D][64]: the node records of 64
                            // consecutive trees interleaved slot by slot
  const uint32_t *leaf_pk;  // [T][2^D][leaf_pk_words]: values, then caller id
  const uint4 *last_il;     // D >= 1 and leaf_dim <= 2: the last level with its leaves, else nullptr
  const uint4 *fast;        // packed blocks (mode 0 or 3, lg = D), or nullptr
  const float *fast_leafv;  // mode 3: [padded T][2^D] leaf values; else nullptr
  int32_t fast_mode;        // 0: each block holds its leaf records; 3: leaf values apart, ids = slot + id_base
  int32_t fast_chunks;      // padded trees / fast_tc_m(fast_mode, block bytes)
  int32_t id_base;          // mode 3: caller id of leaf slot 0 in every tree
};

// TreeTraversal tensors (Table 5, Algorithm 2), breadth-first per tree with
// siblings adjacent (left = right - 1). Leaves loop to themselves: threshold
// -inf (no x is below it, NaN included) and right = the leaf's own id.
struct TtDev {
  const uint2 *node;        // [T][n_pad] {threshold bits, feature | right << 16}
  const int32_t *depth;     // [T] levels to descend per tree
  const float *leaf_value;  // [T][n_pad][leaf_dim], indexed by node id
  const int32_t *leaf_id;   // [T][n_pad] caller-local node id
  int32_t n_pad;
  int32_t max_depth;
  const uint2 *node_il;     // [ceil(T/64)][n_pad][64], as PttDev::node_il
  const uint32_t *leaf_pk;  // [T][n_pad][leaf_pk_words], as PttDev::leaf_pk
  const uint4 *fast;        // packed blocks (mode 1 or 2), or nullptr
  const uint2 *fast_leaf;   // mode 2: [padded T][2^fast_lg] leaf records; else nullptr
  int32_t fast_mode;
  int32_t fast_lg;
  int32_t fast_chunks;
};

// GEMM tensors (Table 3, Algorithm 1). Internal nodes in breadth-first order
// give the reduction index k; leaves in left-to-right order give column l.
// ct holds 4*C^T so that, with predicates encoded as 0/64, one product term
// is +-256 and the accumulator started at bias[l] = l - 256*D[l] ends at
// 256*((T.C)_l - D_l) + l: non-negative exactly at the selected leaf.
struct GemmDev {
  const uint2 *node;        // [T][k_pad] {threshold bits, feature}; padding: -inf
  const int32_t *shape;     // [T] index into ct / bias
  const int8_t *ct;         // [S][l_pad][k_pad]
  const int32_t *bias;      // [S][l_pad]; padded columns hold a large negative
  const float *leaf_value;  // [T][l_pad][leaf_dim]
  const int32_t *leaf_id;   // [T][l_pad]
  int32_t k_pad, l_pad, n_shapes;
};

// How a launcher is called: the caller-provided device scratch for the tree
// split of small batches, and, for a dry run, a string that receives a
// description of the kernels the call would launch (name as the compiler
// prints the instantiation, grid, block, dynamic LDS) instead of launching.
struct Launch {
  void *ptr = nullptr;
  int64_t bytes = 0;
  std::string *plan = nullptr;
};

// GEMM tree split: batches up to kGemmSplitMaxRows rows may divide their
// trees, in groups of kGemmSplitGroup, among the 16-row tile workgroups.
constexpr int64_t kGemmSplitMaxRows = 4096;
constexpr int kGemmSplitGroup = 4;
inline int64_t gemm_split_workspace_bytes(int64_t n_rows, int32_t n_trees, int32_t n_outputs) {
  if (n_rows < 1 || n_rows > kGemmSplitMaxRows) return 0;
  const int64_t groups = (n_trees + kGemmSplitGroup - 1) / kGemmSplitGroup;
  return groups < 2 ? 0 : groups * n_rows * n_outputs * 8;
}

// The error message hb_last_error() returns on this thread; returns code.
int set_error(int code, const std::string &msg);
// The HIP device of a compiled handle (-1: host-only handle or NULL).
int handle_device(const hb_handle *h);

// Tree split: batches up to kSplitMaxRows rows may have their trees divided
// among up to one workgroup per 32-tree group of each row tile, so that a
// small batch still fills the chip; the workgroups leave double partial sums
// (split x rows x outputs) that a second kernel adds in a fixed order.
constexpr int64_t kSplitMaxRows = 65536;
// Largest workspace a split of n_rows rows can use (0: never split).
inline int64_t split_workspace_bytes(int64_t n_rows, int32_t n_trees, int32_t n_outputs) {
  if (n_rows < 1 || n_rows > kSplitMaxRows) return 0;
  const int64_t groups = (n_trees + kFastIdGroup - 1) / kFastIdGroup;
  return groups < 2 ? 0 : groups * n_rows * n_outputs * 8;
}

// Each launcher checks its arguments against what the kernel and its grid
// assume, enqueues on `stream`, and returns HB_OK or an error code with a
// message in *err.
int launch_ptt(const EnsembleDev &e, const PttDev &t, const float *X, int64_t n_rows,
               float *scores, int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err);
int launch_tt(const EnsembleDev &e, const TtDev &t, const float *X, int64_t n_rows,
              float *scores, int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err);
int launch_gemm(const EnsembleDev &e, const GemmDev &t, const float *X, int64_t n_rows,
                float *scores, int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err);

// One line of a dry run's plan: "name grid=(x,y) block=b lds=bytes".
inline void plan_line(std::string *plan, const std::string &name, int64_t gx, int64_t gy, int block, size_t lds) {
  if (!plan->empty()) *plan += "; ";
  *plan += name + " grid=(" + std::to_string(gx) + "," + std::to_string(gy) + ") block=" + std::to_string(block) +
           " lds=" + std::to_string(lds);
}

}  // namespace hb
