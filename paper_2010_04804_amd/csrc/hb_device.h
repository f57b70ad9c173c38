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

// ---- fast traversal kernels (instantiated in hb_fast_ptt.hip / hb_fast_tt.hip)

// Rows (= threads) per workgroup: 512 when the row tile fits next to the
// tree chunks (eight waves share each staged chunk), else 256. The LDS stride
// of one feature column of the row tile is exactly the row count, so a lane's
// gather x[f] hits bank (lane mod 32) whatever feature each lane needs.

struct FastArgs {
  const float *X;
  int64_t n_rows;
  int32_t F;
  int32_t *leaf_ids;
  OutArgs out;
  const int32_t *tree_class;
  const uint4 *blocks;        // [chunks * TC][tree bytes / 16]
  const int32_t *tree_depth;  // TT: [T]
  int32_t n_chunks;
  int32_t ids_vec;            // leaf_ids rows start 16-byte aligned (T % 4 == 0, aligned base)
};

using FastFn = void (*)(FastArgs);

// The kernel for (mode, lg, multi-output) or nullptr; lg in [1, kFastMaxLg].
FastFn fast_ptt_kernel_256(int lg, bool multi);
FastFn fast_ptt_kernel_512(int lg, bool multi);
FastFn fast_tt_kernel_256(int lg, bool multi);
FastFn fast_tt_kernel_512(int lg, bool multi);

}  // namespace hb
