// hb_device.h -- device helpers shared by the kernel sources.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "hb_internal.h"

namespace hb {

__device__ __forceinline__ float as_float(uint32_t u) { return __uint_as_float(u); }

// Where and how a row's aggregated margins become scores.
struct OutArgs {
  float *scores;      // [n, K]
  int32_t T, K, aggregation, transform;
  const float *base_score;  // [K] or nullptr
};

// Aggregated margin -> transformed score, in double precision: MEAN divides
// by the tree count, the base score is added, then sigmoid or a
// max-subtracted softmax is applied.
template <int KMAX>
__device__ __forceinline__ void finish_row(const OutArgs &a, const double (&acc)[KMAX], int64_t row) {
  double s[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    double v = acc[k];
    if (a.aggregation == HB_AGG_MEAN) v /= (double)a.T;
    if (a.base_score && k < a.K) v += (double)a.base_score[k];
    s[k] = v;
  }
  if (a.transform == HB_POST_SIGMOID) {
#pragma unroll
    for (int k = 0; k < KMAX; ++k) s[k] = 1.0 / (1.0 + exp(-s[k]));
  } else if (a.transform == HB_POST_SOFTMAX) {
    double m = s[0];
#pragma unroll
    for (int k = 1; k < KMAX; ++k)
      if (k < a.K) m = fmax(m, s[k]);
    double z = 0.0;
#pragma unroll
    for (int k = 0; k < KMAX; ++k)
      if (k < a.K) {
        s[k] = exp(s[k] - m);
        z += s[k];
      }
#pragma unroll
    for (int k = 0; k < KMAX; ++k) s[k] /= z;
  }
#pragma unroll
  for (int k = 0; k < KMAX; ++k)
    if (k < a.K) a.scores[row * a.K + k] = (float)s[k];
}

// Writes the leaf ids of G consecutive trees (held in registers, one row per
// lane) as whole row segments: each wave passes its rows through a
// 16-row LDS staging area (16-byte blocks XOR-swizzled by row to spread
// banks) so that every store instruction writes G*4-byte segments of 64*16/G
// rows instead of one 16-byte piece of 64 rows. The four 16-row passes are
// split in two halves (flush_stage: lanes of the pass write their rows to the
// staging area; flush_store: the wave reads them back as row segments and
// stores them) so that a caller can put other work between the two.
// Leaf ids of a group, one row per lane, either as G scalars or as G/4
// native 4-vectors (whole VGPR quads, which a 16-byte LDS write takes as is).
typedef int i32x4 __attribute__((ext_vector_type(4)));
template <int G>
__device__ __forceinline__ i32x4 id_block(const int32_t (&ids)[G], int b) {
  return i32x4{ids[4 * b], ids[4 * b + 1], ids[4 * b + 2], ids[4 * b + 3]};
}
template <int NB>
__device__ __forceinline__ i32x4 id_block(const i32x4 (&ids)[NB], int b) {
  return ids[b];
}
template <int G>
__device__ __forceinline__ int id_at(const int32_t (&ids)[G], int g) {
  return ids[g];
}
template <int NB>
__device__ __forceinline__ int id_at(const i32x4 (&ids)[NB], int g) {
  return ids[g >> 2][g & 3];
}

template <int G, class IDS>
__device__ __forceinline__ void flush_stage(int4 *stage, const IDS &ids, int p) {
  constexpr int NB = G / 4;  // 16-byte blocks per row segment
  const int lane = threadIdx.x & 63;
  if ((lane >> 4) == p) {
    const int r = lane & 15;
    i32x4 *st = reinterpret_cast<i32x4 *>(stage);
#pragma unroll
    for (int b = 0; b < NB; ++b) st[r * NB + (b ^ (r & (NB - 1)))] = id_block(ids, b);
  }
}

template <int G>
__device__ __forceinline__ void flush_store(int32_t *leaf_ids, int64_t n_rows, int T, bool ids_nt,
                                            const int4 *stage, int64_t r0w, int t0, int p) {
  constexpr int NB = G / 4;
  const int lane = threadIdx.x & 63;
  const int ntrees = min(G, T - t0);
#pragma unroll
  for (int i = 0; i < (16 * NB + 63) / 64; ++i) {
    const int q = i * 64 + lane;
    const int r = q / NB;
    const int b = q % NB;
    const int64_t grow = r0w + 16 * p + r;
    if (q < 16 * NB && grow < n_rows && 4 * b < ntrees) {
      const int4 v = stage[r * NB + (b ^ (r & (NB - 1)))];
      int32_t *dst = leaf_ids + grow * T + t0 + 4 * b;
      if (ids_nt) {  // streaming: two 8-byte stores that do not allocate in L2
        typedef int i32x2 __attribute__((ext_vector_type(2)));
        __builtin_nontemporal_store(i32x2{v.x, v.y}, reinterpret_cast<i32x2 *>(dst));
        __builtin_nontemporal_store(i32x2{v.z, v.w}, reinterpret_cast<i32x2 *>(dst + 2));
      } else {
        *reinterpret_cast<int4 *>(dst) = v;
      }
    }
  }
}

template <int G, class IDS>
__device__ __forceinline__ void flush_ids(int32_t *leaf_ids, int64_t n_rows, int T, bool ids_vec, bool ids_nt,
                                          int4 *stage, const IDS &ids, int64_t r0w, int t0) {
  const int lane = threadIdx.x & 63;
  if (ids_vec) {
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      flush_stage<G>(stage, ids, p);
      __builtin_amdgcn_wave_barrier();
      flush_store<G>(leaf_ids, n_rows, T, ids_nt, stage, r0w, t0, p);
      __builtin_amdgcn_wave_barrier();
    }
  } else {
    const int ntrees = min(G, T - t0);
    const int64_t row = r0w + lane;
    if (row < n_rows) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (g < ntrees) leaf_ids[row * T + t0 + g] = id_at(ids, g);
    }
  }
}

// ---- fast traversal kernels (instantiated in hb_fast_ptt.hip / hb_fast_tt.hip)

// Rows (= threads) per workgroup: 128, 256, 512, 768 or 1024, with a 64 or 32 KiB
// tree-chunk budget; the launcher takes the shape that puts the most waves on
// a CU within the LDS (the row tile grows with the feature count). The LDS
// stride of one feature column of the row tile is exactly the row count, so a
// lane's gather x[f] hits bank (lane mod 32) whatever feature each lane needs.

// Category-set indicator of a feature-tile column (kColCat): 0 when the row
// goes left (its category, the integer part of a non-negative value below
// 32 W, is in the set; or the value is NaN and the column's nodes send
// missing values left), else 1. The nodes test it against 0.5.
__device__ __noinline__ float xcat(const float *row, const int32_t *cols, int c) {
  const uint32_t *d = reinterpret_cast<const uint32_t *>(cols) + (c & kColMask);
  const float v = row[d[0]];
  if (__builtin_isnan(v)) return (c & kColNanLeft) ? 0.0f : 1.0f;
  if (v >= 0.0f && v < 32.0f * (float)d[1]) {
    const uint32_t k = (uint32_t)v;  // integer part
    return ((d[2 + (k >> 5)] >> (k & 31u)) & 1u) ? 0.0f : 1.0f;
  }
  return 1.0f;
}

// Feature-tile column f of an input row: the identity when cols is null, else
// input column cols[f] & kColMask, with a NaN read as -inf when the column
// serves nodes that send missing values left, or a category-set indicator.
__device__ __forceinline__ float xval(const float *row, const int32_t *cols, int f) {
  if (!cols) return row[f];
  const int c = cols[f];
  if (c & kColCat) return xcat(row, cols, c);
  const float v = row[c & kColMask];
  return ((c & kColNanLeft) && __builtin_isnan(v)) ? -__builtin_inff() : v;
}

// xval for reads straight from an input row inside a hot loop: COLS is a
// compile-time choice, so a model without a column list pays nothing.
template <bool COLS>
__device__ __forceinline__ float xget(const float *row, const int32_t *cols, int f) {
  if constexpr (COLS)
    return xval(row, cols, f);
  else
    return row[f];
}

struct FastArgs {
  const float *X;
  int64_t n_rows;
  int32_t F;                  // feature-tile columns
  int32_t Fs;                 // row stride of X (input columns)
  const int32_t *cols;        // tile column -> input column, or nullptr
  int32_t *leaf_ids;
  OutArgs out;
  const int32_t *tree_class;
  const uint4 *blocks;        // [chunks * TC][tree bytes / 16]
  const uint2 *leaf;          // TT mode 2: [chunks * TC][2^lg] leaf records (global memory)
  const float *leafv;         // PTT mode 3: [chunks * TC][2^lg] leaf values (global memory)
  int32_t id_base;            // PTT mode 3: caller id of leaf slot 0
  const int32_t *tree_depth;  // TT: [T]
  int32_t n_chunks;
  // Tree split (small batches): workgroup (x, y) walks chunks [y * split,
  // min((y + 1) * split, n_chunks)) of row tile x and stores its raw sums in
  // partial[y][row][K]; 0 = one workgroup walks every tree and finishes rows.
  int32_t split;
  double *partial;
  int32_t ids_vec;            // leaf_ids rows start 16-byte aligned (T % 4 == 0, aligned base)
  // vector leaves: [T][vec_stride][LD] leaf values, indexed by the tree and
  // the leaf's slot (PTT) or node (TT); nullptr for scalar leaves
  const float *vec;
  int32_t vec_stride;
  int32_t LD;
  // with ids_vec: byte k = the residues r mod 8 of the rows whose 128-byte
  // lines of leaf ids begin at trees congruent to 4k mod 32
  uint64_t id_phase;
};

using FastFn = void (*)(FastArgs);

// Adds the partial sums of a tree split ([split][n_rows][K] doubles) in a
// fixed order and finishes the rows; with plan, describes the launch instead.
int split_finish(const double *partial, int split, int64_t n_rows, const OutArgs &out, std::string *plan,
                 hipStream_t stream, std::string *err);

// Accumulators per row of a fast kernel: 1 (one output), 2 (two outputs,
// e.g. binary classifiers with probability-vector leaves) or HB_MAX_OUTPUTS.

// The kernel for (mode, lg, multi-output) or nullptr; lg in [1, kFastMaxLg].
FastFn fast_ptt_kernel_128(int lg, int km);
FastFn fast_ptt_kernel_256(int lg, int km);
FastFn fast_ptt_kernel_256s(int lg, int km);
FastFn fast_ptt_kernel_512(int lg, int km);
FastFn fast_ptt_kernel_512s(int lg, int km);
FastFn fast_ptt_kernel_768(int lg, int km);
FastFn fast_ptt_kernel_1024(int lg, int km);
// PTT with the leaf values in global memory and 8-bit slot ids (mode 3):
// scalar leaves, one output (km 1) or one per tree class (km 2, or 16 below
// 1024-row workgroups), lg <= 8, 32 KiB of double-buffered chunks.
FastFn fast_pttg_kernel_1024(int lg, int km);
FastFn fast_pttg_kernel_512(int lg, int km);
FastFn fast_pttg_kernel_256(int lg, int km);
FastFn fast_pttg_kernel_128(int lg, int km);
FastFn fast_tt_kernel_1024(int lg, int km);
FastFn fast_tt_kernel_256(int lg, int km);
FastFn fast_tt_kernel_512(int lg, int km);
FastFn fast_tt_kernel_512s(int lg, int km);
FastFn fast_tt_kernel_256s(int lg, int km);
FastFn fast_tt_kernel_128(int lg, int km);
// TT with leaf records in global memory (mode 2)
FastFn fast_ttg_kernel_1024(int lg, int km);
FastFn fast_ttg_kernel_256(int lg, int km);
FastFn fast_ttg_kernel_512(int lg, int km);
FastFn fast_ttg_kernel_512s(int lg, int km);
FastFn fast_ttg_kernel_256s(int lg, int km);
FastFn fast_ttg_kernel_128(int lg, int km);

}  // namespace hb
