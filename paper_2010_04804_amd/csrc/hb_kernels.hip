// hb_kernels.hip -- gfx950 kernels for batched tree-ensemble scoring.
//
// Traversal kernels (PerfectTreeTraversal, Algorithm 3; TreeTraversal,
// Algorithm 2 of Sec. 4.1). One lane owns one row; a workgroup owns
// kRows = 256 consecutive rows and walks them through every tree:
//   * the rows' features are copied once into LDS, feature-major with an odd
//     row stride, so the per-visit gather x[f] of 64 lanes (64 rows, any f)
//     hits 64 different banks;
//   * the trees are staged through LDS in chunks of a power-of-two number of
//     trees; all lanes of a wave visit the same tree, so node records at one
//     level come from a small contiguous range (broadcast-friendly);
//   * each wave advances G trees at once (independent index chains) so LDS
//     latency overlaps;
//   * leaf ids are staged in LDS and written out row-contiguously;
//   * aggregation is per lane in double precision, in tree order, with no
//     atomics, so results are bitwise reproducible.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>

#include "hb_device.h"

namespace hb {
namespace {

constexpr int kRows = 256;             // rows (= threads) per workgroup
constexpr int kXStride = kRows + 1;    // LDS row stride of the feature tile
constexpr int kGroup = 4;              // trees advanced together per wave

// LDS bytes of the feature tile, rounded up so the tables after it stay
// 16-byte aligned for the vector copies.
constexpr size_t xtile_bytes(int F) { return ((size_t)F * kXStride * 4 + 15) / 16 * 16; }

struct TravArgs {
  const float *X;
  int64_t n_rows;
  int32_t F;                  // feature-tile columns
  int32_t Fs;                 // row stride of X (input columns)
  const int32_t *cols;        // tile column -> input column, or nullptr
  float *scores;
  int32_t *leaf_ids;
  int32_t T, K, LD, aggregation, transform;
  const int32_t *tree_class;
  const float *base_score;
  const uint2 *node;          // [T][slots]
  const uint2 *node_il;       // [ceil(T/64)][slots][64] (trees-across-lanes kernel)
  const uint32_t *leaf_pk;    // [T][leaf_slots][leaf_pk_words(LD)] (trees-across-lanes kernel)
  const uint4 *last_il;       // PTT: last level with its leaves (PttDev::last_il), or nullptr
  const float *leaf_value;    // [T][leaf_slots][LD]
  const int32_t *leaf_id;     // [T][leaf_slots]
  const int32_t *tree_depth;  // TT: [T]
  int32_t slots;              // node records per tree
  int32_t leaf_slots;         // leaf entries per tree
  int32_t depth;              // PTT: D
  int32_t lg_tc;              // log2 of trees per LDS chunk
  int32_t x_in_lds;           // informational; the template decides
};

template <bool PERFECT, bool X_LDS, int KMAX, bool LEAF_VEC, bool COLS = false>
__global__ __launch_bounds__(kRows) void traverse_kernel(TravArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * kRows;
  const int64_t row = r0 + tid;
  const bool valid = row < a.n_rows;
  const int nblk = (int)min((int64_t)kRows, a.n_rows - r0);
  const int tc_full = 1 << a.lg_tc;
  const int LD = LEAF_VEC ? a.LD : 1;

  size_t off = 0;
  float *xs = reinterpret_cast<float *>(smem);
  if (X_LDS) off += xtile_bytes(a.F);
  uint2 *nodes = reinterpret_cast<uint2 *>(smem + off);
  off += (size_t)tc_full * a.slots * 8;
  float *lvals = reinterpret_cast<float *>(smem + off);
  off += (size_t)tc_full * a.leaf_slots * LD * 4;
  int32_t *lids = reinterpret_cast<int32_t *>(smem + off);
  off += (size_t)tc_full * a.leaf_slots * 4;
  int32_t *stage = reinterpret_cast<int32_t *>(smem + off);
  const int stage_stride = tc_full + ((tc_full & 1) ? 0 : 1);

  if (X_LDS) {
    const float *src = a.X + r0 * a.Fs;
    const int total = kRows * a.F;
    for (int i = tid; i < total; i += kRows) {
      const int r = i / a.F;
      const int f = i - r * a.F;
      xs[f * kXStride + r] = r < nblk ? xval(src + (size_t)r * a.Fs, a.cols, f) : 0.0f;
    }
  }
  // rows past the end read row n-1 (in bounds) and are never written
  const float *xrow = a.X + (valid ? row : a.n_rows - 1) * a.Fs;

  double acc[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) acc[k] = 0.0;

  for (int t0 = 0; t0 < a.T; t0 += tc_full) {
    const int tc = min(tc_full, a.T - t0);
    __syncthreads();
    {  // stage this chunk's tables (contiguous in global memory)
      const uint4 *src = reinterpret_cast<const uint4 *>(a.node + (size_t)t0 * a.slots);
      uint4 *dst = reinterpret_cast<uint4 *>(nodes);
      const int n16 = tc * a.slots / 2;  // slots is even
      for (int i = tid; i < n16; i += kRows) dst[i] = src[i];
      const float *sv = a.leaf_value + (size_t)t0 * a.leaf_slots * LD;
      const int nv = tc * a.leaf_slots * LD;
      for (int i = tid; i < nv; i += kRows) lvals[i] = sv[i];
      const int32_t *si = a.leaf_id + (size_t)t0 * a.leaf_slots;
      const int ni = tc * a.leaf_slots;
      for (int i = tid; i < ni; i += kRows) lids[i] = si[i];
    }
    __syncthreads();

    for (int j = 0; j < tc; j += kGroup) {
      uint32_t idx[kGroup];
      int jj[kGroup];
#pragma unroll
      for (int g = 0; g < kGroup; ++g) {
        jj[g] = min(j + g, tc - 1);  // a short tail repeats the last tree, unused
        idx[g] = PERFECT ? 1u : 0u;
      }
      int levels;
      if (PERFECT) {
        levels = a.depth;
      } else {
        levels = 0;
#pragma unroll
        for (int g = 0; g < kGroup; ++g) levels = max(levels, a.tree_depth[t0 + jj[g]]);
      }
      for (int lvl = 0; lvl < levels; ++lvl) {
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
          const uint2 rec = nodes[jj[g] * a.slots + idx[g]];
          const uint32_t f = PERFECT ? rec.y : (rec.y & 0xffffu);
          const float x = X_LDS ? xs[f * kXStride + tid] : xget<COLS>(xrow, a.cols, f);
          const bool go_left = x < as_float(rec.x);
          if (PERFECT)
            idx[g] = 2u * idx[g] + (go_left ? 0u : 1u);  // Algorithm 3's heap step
          else
            idx[g] = (rec.y >> 16) - (go_left ? 1u : 0u);  // left = right - 1
        }
      }
#pragma unroll
      for (int g = 0; g < kGroup; ++g) {
        if (j + g >= tc) break;  // uniform
        const uint32_t slot = PERFECT ? idx[g] - (uint32_t)a.leaf_slots : idx[g];
        const int lrec = jj[g] * a.leaf_slots + (int)slot;
        if (LEAF_VEC) {
#pragma unroll
          for (int k = 0; k < KMAX; ++k)
            if (k < LD) acc[k] += (double)lvals[lrec * LD + k];
        } else if (KMAX == 1) {
          acc[0] += (double)lvals[lrec];
        } else {
          const int c = __builtin_amdgcn_readfirstlane(a.tree_class[t0 + j + g]);
          const double v = (double)lvals[lrec];
#pragma unroll
          for (int k = 0; k < KMAX; ++k)
            if (k == c) acc[k] += v;
        }
        if (a.leaf_ids) stage[tid * stage_stride + j + g] = lids[lrec];
      }
    }
    if (a.leaf_ids) {
      __syncthreads();
      const int total = nblk << a.lg_tc;
      for (int i = tid; i < total; i += kRows) {
        const int r = i >> a.lg_tc;
        const int jt = i & (tc_full - 1);
        if (jt < tc) a.leaf_ids[(r0 + r) * a.T + t0 + jt] = stage[r * stage_stride + jt];
      }
    }
  }
  if (valid) finish_row<KMAX>(OutArgs{a.scores, a.T, a.K, a.aggregation, a.transform, a.base_score}, acc, row);
  (void)xrow;
}


using KernelFn = void (*)(TravArgs);

template <bool PERFECT, bool X_LDS, bool COLS = false>
KernelFn pick_k(int kmax, bool vec) {
  if (vec) {
    switch (kmax) {
      case 2: return traverse_kernel<PERFECT, X_LDS, 2, true, COLS>;
      case 8: return traverse_kernel<PERFECT, X_LDS, 8, true, COLS>;
      default: return traverse_kernel<PERFECT, X_LDS, 16, true, COLS>;
    }
  }
  switch (kmax) {
    case 1: return traverse_kernel<PERFECT, X_LDS, 1, false, COLS>;
    case 2: return traverse_kernel<PERFECT, X_LDS, 2, false, COLS>;
    case 8: return traverse_kernel<PERFECT, X_LDS, 8, false, COLS>;
    default: return traverse_kernel<PERFECT, X_LDS, 16, false, COLS>;
  }
}

int kmax_for(int K) { return K <= 1 ? 1 : K <= 2 ? 2 : K <= 8 ? 8 : 16; }

int max_dynamic_lds(std::string *err) {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) {
    *err = "hipDeviceGetAttribute(MaxSharedMemoryPerBlock) failed";
    return -1;
  }
  return v;
}

// Chooses the feature-tile placement and the chunk size, then launches.
// LDS bytes of traverse_kernel with or without the feature tile and tc trees
// per chunk.
size_t traverse_lds(const TravArgs &a, bool xl, int tc) {
  const size_t per_tree = (size_t)a.slots * 8 + (size_t)a.leaf_slots * a.LD * 4 + (size_t)a.leaf_slots * 4;
  const int stride = tc + ((tc & 1) ? 0 : 1);
  return (xl ? xtile_bytes(a.F) : 0) + (size_t)tc * per_tree + (size_t)kRows * stride * 4;
}

// Picks traverse_kernel's chunk size and feature-tile placement: two
// workgroups per CU (half the LDS) with at least kGroup trees per chunk if
// possible, else the whole LDS; the feature tile stays in LDS when it fits.
// Returns the trees per chunk, 0 if even one tree does not fit.
int traverse_plan(const TravArgs &a, int lds_max, bool *x_lds) {
  const size_t half = (size_t)lds_max / 2;
  for (int pass = 0; pass < 4; ++pass) {
    const bool xl = pass < 2 && xtile_bytes(a.F) <= (size_t)lds_max / 4 * 3;
    const size_t budget = (pass % 2 == 0) ? half : (size_t)lds_max;
    for (int c = 16; c >= (pass % 2 == 0 ? kGroup : 1); c >>= 1)
      if (traverse_lds(a, xl, c) <= budget) {
        *x_lds = xl;
        return c;
      }
  }
  return 0;
}

const char *tf(bool b) { return b ? "true" : "false"; }

int launch_traverse(bool perfect, TravArgs a, const Launch &L, hipStream_t stream, std::string *err) {
  if (a.n_rows <= 0) return HB_OK;
  const int lds_max = max_dynamic_lds(err);
  if (lds_max <= 0) return HB_ERR_HIP;
  const int LD = a.LD;
  bool x_lds = false;
  const int tc = traverse_plan(a, lds_max, &x_lds);
  if (tc == 0) {
    *err = "tree tables too large for LDS staging";
    return HB_ERR_UNSUPPORTED;
  }
  a.lg_tc = __builtin_ctz((unsigned)tc);
  a.x_in_lds = x_lds;
  const size_t lds = traverse_lds(a, x_lds, tc);
  const bool vec = LD > 1;
  const int kmax = kmax_for(vec ? LD : a.K);
  const bool cols = a.cols != nullptr;  // only the global-memory reads need the column list per visit
  KernelFn fn = perfect ? (x_lds ? pick_k<true, true>(kmax, vec)
                                 : cols ? pick_k<true, false, true>(kmax, vec) : pick_k<true, false>(kmax, vec))
                        : (x_lds ? pick_k<false, true>(kmax, vec)
                                 : cols ? pick_k<false, false, true>(kmax, vec) : pick_k<false, false>(kmax, vec));
  const int64_t blocks = (a.n_rows + kRows - 1) / kRows;
  if (L.plan) {
    const int km = vec ? (kmax <= 2 ? 2 : kmax <= 8 ? 8 : 16) : kmax;
    plan_line(L.plan,
              std::string("traverse_kernel<") + tf(perfect) + ", " + tf(x_lds) + ", " + std::to_string(km) + ", " +
                  tf(vec) + ", " + tf(!x_lds && cols) + ">",
              blocks, 1, kRows, lds);
    return HB_OK;
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) {
    *err = std::string("hipFuncSetAttribute: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kRows), lds, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  return HB_OK;
}

// ---------------------------------------------------------------------------
// Trees across lanes (small batches and wide rows). A workgroup owns R rows,
// copies them to LDS once, and lane t walks trees t, t + 256, ... for each of
// its rows (node records from the L1/L2 copy of the tables, reused across the
// R rows). Leaf ids come out contiguous per row; the per-lane partial sums are
// combined in a fixed order: a butterfly within each wave, then the four wave
// totals in wave order, so results are reproducible run to run.
constexpr int kLaneThreads = 256;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

template <bool PERFECT, int KMAX, bool LEAF_VEC, int R>
__global__ __launch_bounds__(kLaneThreads) void lanes_kernel(TravArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  float *xs = reinterpret_cast<float *>(smem);  // [R][F]
  double *red = reinterpret_cast<double *>(smem + (((size_t)R * a.F * 4 + 15) / 16 * 16));  // [4][R][KMAX]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t r0 = (int64_t)blockIdx.x * R;
  const int nr = (int)min((int64_t)R, a.n_rows - r0);
  for (int i = tid; i < R * a.F; i += kLaneThreads) {
    const int r = i / a.F;
    xs[i] = r < nr ? xval(a.X + (r0 + r) * a.Fs, a.cols, i - r * a.F) : 0.0f;
  }
  __syncthreads();
  const int LD = LEAF_VEC ? a.LD : 1;
  double acc[R][KMAX];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int k = 0; k < KMAX; ++k) acc[r][k] = 0.0;
  for (int t = tid; t < a.T; t += kLaneThreads) {
    // the wave's 64 trees are interleaved slot by slot: this lane's tree
    // has slot p at record 64 p of its group
    const uint2 *node = a.node_il + (size_t)(t >> 6) * a.slots * 64 + (t & 63);
    const int levels = PERFECT ? a.depth : a.tree_depth[t];
    const int cls = (!LEAF_VEC && KMAX > 1) ? a.tree_class[t] : 0;
    // the R walks of a tree are independent: advance them level by level
    // together so that R node reads are in flight at once
    uint32_t idx[R];
#pragma unroll
    for (int r = 0; r < R; ++r) idx[r] = PERFECT ? 1u : 0u;
    // perfect trees with at most two leaf values take their last level and
    // the leaf from one 32-byte record (LAST is uniform)
    const bool LAST = PERFECT && (LEAF_VEC ? KMAX == 2 : true) && a.last_il != nullptr;
    const int node_levels = LAST ? levels - 1 : levels;
    for (int lvl = 0; lvl < node_levels; ++lvl) {
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint2 rec = node[idx[r] * 64u];
        const uint32_t f = PERFECT ? rec.y : (rec.y & 0xffffu);
        const bool go_left = xs[r * a.F + f] < as_float(rec.x);
        idx[r] = PERFECT ? 2u * idx[r] + (go_left ? 0u : 1u) : (rec.y >> 16) - (go_left ? 1u : 0u);
      }
    }
    if (LAST) {
      const uint32_t half = (uint32_t)a.leaf_slots >> 1;
      const uint4 *last = a.last_il + ((size_t)(t >> 6) * half * 64 + (t & 63)) * 2;
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint4 q0 = last[(idx[r] - half) * 128u];      // {threshold, feature, leaf words}
        const uint4 q1 = last[(idx[r] - half) * 128u + 1];  // more leaf words
        const bool go_left = xs[r * a.F + q0.y] < as_float(q0.x);
        uint32_t id;
        if (!LEAF_VEC) {  // {value, id} left, then right
          const double d = (double)as_float(go_left ? q0.z : q1.x);
#pragma unroll
          for (int k = 0; k < KMAX; ++k) acc[r][k] += (k == cls) ? d : 0.0;
          id = go_left ? q0.w : q1.y;
        } else {  // {value 0, value 1, id} left, then right
          acc[r][0] += (double)as_float(go_left ? q0.z : q1.y);
          acc[r][1] += (double)as_float(go_left ? q0.w : q1.z);
          id = go_left ? q1.x : q1.w;
        }
        if (a.leaf_ids && r < nr) a.leaf_ids[(r0 + r) * a.T + t] = (int32_t)id;
      }
      continue;
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const uint32_t slot = PERFECT ? idx[r] - (uint32_t)a.leaf_slots : idx[r];
      // one packed record per leaf: the values, then the caller id
      const uint32_t *lrec = a.leaf_pk + ((size_t)t * a.leaf_slots + slot) * leaf_pk_words(LD);
      uint32_t id;
      if (!LEAF_VEC) {
        const uint2 v = *reinterpret_cast<const uint2 *>(lrec);
        const double d = (double)as_float(v.x);
#pragma unroll
        for (int k = 0; k < KMAX; ++k) acc[r][k] += (k == cls) ? d : 0.0;
        id = v.y;
      } else if (KMAX == 2) {  // leaf_dim 2: {v0, v1, id, 0}
        const uint4 v = *reinterpret_cast<const uint4 *>(lrec);
        acc[r][0] += (double)as_float(v.x);
        acc[r][1] += (double)as_float(v.y);
        id = v.z;
      } else {
#pragma unroll
        for (int k = 0; k < KMAX; ++k)
          if (k < LD) acc[r][k] += (double)as_float(lrec[k]);
        id = lrec[LD];
      }
      if (a.leaf_ids && r < nr) a.leaf_ids[(r0 + r) * a.T + t] = (int32_t)id;
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      const double w = wave_sum(acc[r][k]);
      if (lane == 0) red[(wave * R + r) * KMAX + k] = w;
    }
  __syncthreads();
  if (tid < nr) {
    double tot[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) {
      double v = 0.0;
#pragma unroll
      for (int w = 0; w < kLaneThreads / 64; ++w) v += red[(w * R + tid) * KMAX + k];
      tot[k] = v;
    }
    finish_row<KMAX>(OutArgs{a.scores, a.T, a.K, a.aggregation, a.transform, a.base_score}, tot, r0 + tid);
  }
}

using LanesFn = void (*)(TravArgs);

template <bool PERFECT, int R>
LanesFn pick_lanes_r(int kmax, bool vec) {
  if (vec) {
    switch (kmax) {
      case 2: return lanes_kernel<PERFECT, 2, true, R>;
      case 8: return lanes_kernel<PERFECT, 8, true, R>;
      default: return lanes_kernel<PERFECT, 16, true, R>;
    }
  }
  switch (kmax) {
    case 1: return lanes_kernel<PERFECT, 1, false, R>;
    case 2: return lanes_kernel<PERFECT, 2, false, R>;
    case 8: return lanes_kernel<PERFECT, 8, false, R>;
    default: return lanes_kernel<PERFECT, 16, false, R>;
  }
}

// Batch sizes up to which the trees-across-lanes kernel beats the
// row-parallel ones. The row-parallel kernels cost a near-constant time until
// the batch fills the chip (one workgroup walks every tree in sequence), the
// tree-parallel one a time proportional to the batch; both scale with
// trees x depth, so the crossing is a batch size. Measured (scores only):
// 500 perfect depth-8 trees cross at about 16K rows, 7 x 500 such trees with
// seven outputs at 12K-14K, and the leaf-wise depth-12 trees (TT, whose
// row-parallel walk is slower) at about 20K.
// Rows across lanes, for inputs too wide for the row-parallel tile: a
// workgroup stages RW whole rows in LDS and each wave walks TPW = 64 / RW
// trees for all RW rows at once (lane = tree slot q, row r), so the RW
// lanes of one tree read its nodes and leaves together and share the
// cache lines: a level-L read of a wave touches at most min(RW, 2^L) lines
// of each of its trees, against up to one line per lane when every lane
// walks its own tree. Trees come from the per-tree tables (node [T][slots]
// and leaf_pk), which stay in L2. Each lane walks ILP consecutive trees
// together (ILP node reads in flight: the walk waits on L2 latency), adds
// their values for its row in tree order and stores their ids as 16-byte
// pieces; the per-lane sums
// of a row are added in a fixed order (the wave's tree slots, then the
// waves) before finish_row, so results are reproducible run to run.
constexpr int kRowsThreads = 1024;
constexpr int kRowsIlp = 4;
// The rows of one tile in registers, between their global load (issued
// before the previous tile is walked) and their LDS store (after it): lane i
// holds 16-byte pieces i, i + 1024, ... of the tile's RW x F floats, which
// are contiguous in X when the tile is the whole rows (no column map).
template <int RW>
struct RowsPrefetch {
  static constexpr int PER = (RW * 2000 / 4 + kRowsThreads - 1) / kRowsThreads;  // up to 2000 features at RW rows
  i32x4 v[PER];
  __device__ __forceinline__ void load(const float *X, int64_t r0, int nr, int F) {
    const int n4 = nr * F / 4;
    const i32x4 *src = reinterpret_cast<const i32x4 *>(X + r0 * F);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = i * kRowsThreads + (int)threadIdx.x;
      // rows are read once: non-temporal, so they pass through L2 without
      // displacing the tree tables every walk reads
      v[i] = e < n4 ? __builtin_nontemporal_load(src + e) : i32x4{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(float *xs, int nr, int F) const {
    const int n4 = RW * F / 4;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int e = i * kRowsThreads + (int)threadIdx.x;
      if (e < n4) reinterpret_cast<i32x4 *>(xs)[e] = v[i];  // rows past nr hold zeros
    }
  }
};

// CONTIG: the tiles are whole contiguous rows in 16-byte pieces (no column
// list), loaded ahead with the contiguous prefetch; otherwise they are staged
// through the column list when needed (a gather ahead of the walk was slower:
// its loads queue in front of the walk's node reads).
template <bool PERFECT, int KMAX, bool LEAF_VEC, int RW, bool CONTIG>
__global__ __launch_bounds__(kRowsThreads) void rows_kernel(TravArgs a) {
  constexpr int TPW = 64 / RW;                    // trees of one wave-level read
  constexpr int WAVES = kRowsThreads / 64;
  constexpr int PASS = WAVES * TPW * kRowsIlp;  // trees per pass of the workgroup
  extern __shared__ __align__(16) unsigned char smem[];
  float *xs = reinterpret_cast<float *>(smem);  // [RW][F]
  // per-lane sums after the walk, apart from the rows (the next tile's rows
  // are stored while the sums are read): [WAVES][TPW][RW][KMAX]
  double *red = reinterpret_cast<double *>(smem + ((size_t)RW * a.F * 4 + 15) / 16 * 16);
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int r = lane & (RW - 1), q = lane / RW;
  const int64_t n_tiles = (a.n_rows + RW - 1) / RW;
  // a workgroup walks tiles blockIdx.x, + gridDim.x, ...; the next tile's
  // rows arrive in registers during the walk
  constexpr bool pf = CONTIG;
  RowsPrefetch<RW> next;
  auto stage_rows = [&](int64_t tile) {  // load and store at once (no prefetch)
    const int64_t r0 = tile * RW;
    const int nr = (int)min((int64_t)RW, a.n_rows - r0);
    for (int i = tid; i < RW * a.F; i += kRowsThreads) {
      const int rr = i / a.F, c = i - rr * a.F;
      xs[rr * a.F + c] = rr < nr ? xval(a.X + (r0 + rr) * a.Fs, a.cols, c) : 0.0f;
    }
  };
  int64_t tile = blockIdx.x;
  if (pf) {
    next.load(a.X, tile * RW, (int)min((int64_t)RW, a.n_rows - tile * RW), a.F);
    next.store(xs, RW, a.F);
  } else {
    stage_rows(tile);
  }
  __syncthreads();
  const int LD = LEAF_VEC ? a.LD : 1;
  const int pkw = leaf_pk_words(LD);
  const bool ids_vec = a.leaf_ids != nullptr && (a.T & 3) == 0 && (reinterpret_cast<uintptr_t>(a.leaf_ids) & 15) == 0;
  for (; tile < n_tiles; tile += gridDim.x) {
    const int64_t r0 = tile * RW;
    const int nr = (int)min((int64_t)RW, a.n_rows - r0);
    const int64_t nt = tile + gridDim.x;
    if (pf && nt < n_tiles) next.load(a.X, nt * RW, (int)min((int64_t)RW, a.n_rows - nt * RW), a.F);
    const float *xrow = xs + r * a.F;
    double acc[KMAX];
#pragma unroll
    for (int k = 0; k < KMAX; ++k) acc[k] = 0.0;
    for (int P = 0; P < a.T; P += PASS) {
      const int t0 = P + wave * (TPW * kRowsIlp) + q * kRowsIlp;  // this lane's first tree
      if (t0 >= a.T) continue;
      uint32_t idx[kRowsIlp];  // record index within the node table (32 bits: tables below 32 GB)
      int levels = PERFECT ? a.depth : 0;
#pragma unroll
      for (int j = 0; j < kRowsIlp; ++j) {
        const int t = min(t0 + j, a.T - 1);  // past the last tree: walk it again, discard
        idx[j] = (uint32_t)t * (uint32_t)a.slots + (PERFECT ? 1u : 0u);
        if (!PERFECT) levels = max(levels, a.tree_depth[t]);
      }
      for (int lvl = 0; lvl < levels; ++lvl) {
        uint2 rec[kRowsIlp];
#pragma unroll
        for (int j = 0; j < kRowsIlp; ++j) rec[j] = a.node[idx[j]];
#pragma unroll
        for (int j = 0; j < kRowsIlp; ++j) {
          const uint32_t f = PERFECT ? rec[j].y : (rec[j].y & 0xffffu);
          const bool go_left = xrow[f] < as_float(rec[j].x);
          // PTT: heap index h of tree t at record t S + h, so 2 h + b is at 2 (t S + h) - t S + b
          const uint32_t tb = (uint32_t)min(t0 + j, a.T - 1) * (uint32_t)a.slots;
          idx[j] = PERFECT ? 2u * idx[j] - tb + (go_left ? 0u : 1u) : tb + (rec[j].y >> 16) - (go_left ? 1u : 0u);
        }
      }
      uint32_t id[kRowsIlp];
#pragma unroll
      for (int j = 0; j < kRowsIlp; ++j) {
        const int t = min(t0 + j, a.T - 1);
        const uint32_t h = idx[j] - (uint32_t)t * (uint32_t)a.slots;  // heap index (PTT) or node (TT)
        const uint32_t slot = PERFECT ? h - (uint32_t)a.leaf_slots : h;
        const uint32_t *lrec = a.leaf_pk + ((size_t)t * a.leaf_slots + slot) * pkw;
        const bool live = t0 + j < a.T;
        if (!LEAF_VEC) {
          const uint2 v = *reinterpret_cast<const uint2 *>(lrec);
          if (live) {
            if (KMAX == 1) {
              acc[0] += (double)as_float(v.x);
            } else {
              const int cls = a.tree_class ? a.tree_class[t] : 0;
#pragma unroll
              for (int k = 0; k < KMAX; ++k) acc[k] += k == cls ? (double)as_float(v.x) : 0.0;
            }
          }
          id[j] = v.y;
        } else {  // KMAX == 2: {v0, v1, id, 0}
          const uint4 v = *reinterpret_cast<const uint4 *>(lrec);
          if (live) {
            acc[0] += (double)as_float(v.x);
            acc[1] += (double)as_float(v.y);
          }
          id[j] = v.z;
        }
      }
      if (a.leaf_ids && r < nr) {
        int32_t *dst = a.leaf_ids + (r0 + r) * a.T + t0;
        if (ids_vec && t0 + kRowsIlp <= a.T) {
#pragma unroll
          for (int j = 0; j < kRowsIlp; j += 4)
            __builtin_nontemporal_store(i32x4{(int)id[j], (int)id[j + 1], (int)id[j + 2], (int)id[j + 3]},
                                        reinterpret_cast<i32x4 *>(dst + j));
        } else {
#pragma unroll
          for (int j = 0; j < kRowsIlp; ++j)
            if (t0 + j < a.T) dst[j] = (int32_t)id[j];
        }
      }
    }
    // per-row totals in a fixed order: over the wave's tree slots, then the waves
#pragma unroll
    for (int k = 0; k < KMAX; ++k) red[((wave * TPW + q) * RW + r) * KMAX + k] = acc[k];
    __syncthreads();  // every wave is done with this tile's rows and sums
    if (nt < n_tiles) {
      if (pf)
        next.store(xs, RW, a.F);
      else
        stage_rows(nt);
    }
    if (tid < nr) {
      double tot[KMAX];
#pragma unroll
      for (int k = 0; k < KMAX; ++k) {
        double v = 0.0;
#pragma unroll 1
        for (int w = 0; w < WAVES * TPW; ++w) v += red[(w * RW + tid) * KMAX + k];
        tot[k] = v;
      }
      finish_row<KMAX>(OutArgs{a.scores, a.T, a.K, a.aggregation, a.transform, a.base_score}, tot, r0 + tid);
    }
    __syncthreads();  // the next tile's rows are in place; its sums may overwrite these
  }
}

// Bytes of LDS rows_kernel needs: the RW rows and the per-lane sums.
inline size_t rows_lds(int F, int RW, int kmax) {
  return ((size_t)RW * (size_t)F * 4 + 15) / 16 * 16 + (size_t)kRowsThreads * kmax * 8;
}

constexpr int64_t kLanesMaxRowsPtt = 12288;
constexpr int64_t kLanesMaxRowsTt = 16384;
// With a workspace the tree-split row-parallel kernel takes over from here
// (measured: the split wins from 1,500 to 2,000 rows on the single-output
// models, while the seven-output model gains from splitting at any size
// measured, 512 rows up).
constexpr int64_t kLanesMaxRowsSplit = 1024;

constexpr int kNotApplicable = 1;
constexpr int kPreferLanes = 2;  // launch_fast: the trees-across-lanes kernel is the better fit

// Adds the split workgroups' partial sums of each row, then applies the
// aggregation and transform. A workgroup takes 64 rows; wave j adds parts
// j, j + J, j + 2J, ... in turn (J waves keep J loads of every row in
// flight), and the first wave adds the J sums in wave order: a fixed order,
// so the result does not vary from run to run.
template <int KMAX, int J>
__global__ __launch_bounds__(64 * J) void split_finish_kernel(const double *partial, int split, int64_t n_rows,
                                                              OutArgs out) {
  extern __shared__ double red[];  // [J][K][64]
  const int lane = threadIdx.x & 63, j = threadIdx.x >> 6;
  const int64_t row = (int64_t)blockIdx.x * 64 + lane;
  const bool valid = row < n_rows;
  double tot[KMAX];
#pragma unroll
  for (int k = 0; k < KMAX; ++k) tot[k] = 0.0;
  if (valid) {
#pragma unroll 4
    for (int s = j; s < split; s += J) {
      const double *p = partial + ((size_t)s * n_rows + row) * out.K;
#pragma unroll
      for (int k = 0; k < KMAX; ++k)
        if (k < out.K) tot[k] += p[k];
    }
  }
#pragma unroll
  for (int k = 0; k < KMAX; ++k)
    if (k < out.K) red[(j * out.K + k) * 64 + lane] = tot[k];
  __syncthreads();
  if (j != 0 || !valid) return;
#pragma unroll
  for (int k = 0; k < KMAX; ++k) {
    tot[k] = 0.0;
    if (k < out.K)
      for (int w = 0; w < J; ++w) tot[k] += red[(w * out.K + k) * 64 + lane];
  }
  finish_row<KMAX>(out, tot, row);
}

// Adds the partial sums of a tree split ([split][n_rows][K] doubles) in a
// fixed order and finishes the rows (or, with plan, describes that launch).
int launch_split_finish(const double *partial, int split, int64_t n_rows, const OutArgs &out, std::string *plan,
                        hipStream_t stream, std::string *err) {
  const unsigned fin_rows = (unsigned)((n_rows + 63) / 64);
  const bool multi = out.K > 1;
  // 16 waves per 64 rows for scalar outputs, 8 for several (their sums take
  // K times the LDS: at most 64 KiB)
  if (plan) {
    if (multi)
      plan_line(plan, "split_finish_kernel<16, 8>", fin_rows, 1, 64 * 8, (size_t)8 * out.K * 64 * 8);
    else
      plan_line(plan, "split_finish_kernel<1, 16>", fin_rows, 1, 64 * 16, (size_t)16 * 64 * 8);
    return HB_OK;
  }
  if (multi)
    hipLaunchKernelGGL((split_finish_kernel<HB_MAX_OUTPUTS, 8>), dim3(fin_rows), dim3(64 * 8),
                       (size_t)8 * out.K * 64 * sizeof(double), stream, partial, split, n_rows, out);
  else
    hipLaunchKernelGGL((split_finish_kernel<1, 16>), dim3(fin_rows), dim3(64 * 16), (size_t)16 * 64 * sizeof(double),
                       stream, partial, split, n_rows, out);
  const hipError_t rc = hipGetLastError();
  if (rc != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(rc);
    return HB_ERR_HIP;
  }
  return HB_OK;
}

// Launches the fast kernel when its layout exists and its LDS fits; returns
// kNotApplicable to fall back to traverse_kernel.
// vec, vec_stride: vector leaves' values [T][vec_stride][leaf_dim] (the
// strategy's leaf-value table), or nullptr for scalar leaves.
int launch_fast(int mode, int lg, const uint4 *blocks, const void *leaf, int chunks, const int32_t *depth,
                const float *vec, int vec_stride, int id_base, const EnsembleDev &e, const float *X, int64_t n_rows,
                float *scores, int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err) {
  if (!blocks || (mode >= 2 && !leaf) || lg < 1 || lg > kFastMaxLg) return kNotApplicable;
  if (mode == 3 && (e.leaf_dim != 1 || lg > 8)) return kNotApplicable;
  if (e.leaf_dim != 1 && (!vec || e.leaf_dim != e.n_outputs || e.leaf_dim > HB_MAX_OUTPUTS)) return kNotApplicable;
  const int lds_max = max_dynamic_lds(err);
  if (lds_max <= 0) return HB_ERR_HIP;
  const int tb = fast_tree_bytes(mode, lg);
  const int km = e.n_outputs == 1 ? 1 : e.n_outputs == 2 ? 2 : HB_MAX_OUTPUTS;
  // Workgroup shapes (rows, chunk budget); the one with the most waves per CU
  // that fits in LDS wins (the walk is bound by the latency of its dependent
  // LDS reads), the larger chunk on a tie (fewer hand-overs). Wide workgroups
  // only when the batch gives every CU several of them.
  struct Shape {
    int rows, budget;
    FastFn (*get)(int, int);
  };
  static const Shape kPtt[] = {{1024, kFastTableSmall, fast_ptt_kernel_1024},
                               {768, kFastTableSmall, fast_ptt_kernel_768},
                               {512, kFastTableLds, fast_ptt_kernel_512},
                               {512, kFastTableSmall, fast_ptt_kernel_512s},
                               {256, kFastTableLds, fast_ptt_kernel_256},
                               {256, kFastTableSmall, fast_ptt_kernel_256s},
                               {128, kFastTableSmall, fast_ptt_kernel_128}};
  static const Shape kTt[] = {{1024, kFastTableSmall, fast_tt_kernel_1024},
                              {512, kFastTableLds, fast_tt_kernel_512},
                              {512, kFastTableSmall, fast_tt_kernel_512s},
                              {256, kFastTableLds, fast_tt_kernel_256},
                              {256, kFastTableSmall, fast_tt_kernel_256s},
                              {128, kFastTableSmall, fast_tt_kernel_128}};
  static const Shape kTtg[] = {{1024, kFastTableSmall, fast_ttg_kernel_1024},
                               {512, kFastTableLds, fast_ttg_kernel_512},
                               {512, kFastTableSmall, fast_ttg_kernel_512s},
                               {256, kFastTableLds, fast_ttg_kernel_256},
                               {256, kFastTableSmall, fast_ttg_kernel_256s},
                               {128, kFastTableSmall, fast_ttg_kernel_128}};
  static const Shape kPttg[] = {{1024, kFastTableSmall, fast_pttg_kernel_1024},
                                {512, kFastTableSmall, fast_pttg_kernel_512},
                                {256, kFastTableSmall, fast_pttg_kernel_256},
                                {128, kFastTableSmall, fast_pttg_kernel_128}};
  const Shape *shapes = mode == 0 ? kPtt : mode == 1 ? kTt : mode == 2 ? kTtg : kPttg;
  const int n_shapes = mode == 0 ? 7 : mode == 3 ? 4 : 6;
  // static LDS: the chunk buffer(s) and the leaf-id staging (16-bit ids of a
  // 32-tree group per row); dynamic LDS: the feature tile (F x rows floats)
  auto lds_of = [&](const Shape &sh) {
    const size_t table = (size_t)fast_bufs_m(mode, tb, sh.budget) * fast_tc_m(mode, tb, sh.budget) * tb;
    return table + (size_t)sh.rows * kFastIdStageBytes + (size_t)e.n_cols * sh.rows * 4;
  };
  int best = -1;
  long best_waves = 0;
  for (int i = 0; i < n_shapes; ++i) {
    const Shape &sh = shapes[i];
    const size_t lds = lds_of(sh);
    if (lds > (size_t)lds_max || !sh.get(lg, km)) continue;
    if (sh.rows > 256 && n_rows < 64 * (int64_t)sh.rows) continue;
    const long waves = (long)(sh.rows / 64) * (long)((size_t)lds_max / lds);
    if (waves > best_waves) {
      best = i;
      best_waves = waves;
    }
  }
  if (best < 0) return kNotApplicable;
  // Below four waves per CU the row-parallel walk is latency-bound; the
  // trees-across-lanes kernel then wins when the node tables are small
  // enough to stay in L1 (depth-3 forests: 0.9 vs 1.5 ms at 1M rows).
  const int64_t table_bytes =
      (int64_t)chunks * fast_tc_m(mode, tb) * (tb + (mode == 2 ? (8 << lg) : mode == 3 ? (4 << lg) : 0));
  if (best_waves < 4 && table_bytes <= (int64_t)64 << 10) return kPreferLanes;
  const int rows = shapes[best].rows;
  const size_t xbytes = (size_t)e.n_cols * rows * 4;
  FastFn fn = shapes[best].get(lg, km);
  if (!fn) return kNotApplicable;
  FastArgs a{};
  a.X = X;
  a.n_rows = n_rows;
  a.F = e.n_cols;
  a.Fs = e.n_features;
  a.cols = e.cols;
  a.leaf_ids = leaf_ids;
  a.out = OutArgs{scores, e.n_trees, e.n_outputs, e.aggregation, e.transform, e.base_score};
  a.tree_class = e.tree_class;
  if (e.leaf_dim != 1) {
    a.vec = vec;
    a.vec_stride = vec_stride;
    a.LD = e.leaf_dim;
  }
  a.blocks = blocks;
  a.leaf = mode == 2 ? static_cast<const uint2 *>(leaf) : nullptr;
  a.leafv = mode == 3 ? static_cast<const float *>(leaf) : nullptr;
  a.id_base = id_base;
  a.tree_depth = depth;
  a.n_chunks = (int)((int64_t)chunks * fast_tc_m(mode, tb) / fast_tc_m(mode, tb, shapes[best].budget));
  a.ids_vec = (e.n_trees % 4 == 0) && ((reinterpret_cast<uintptr_t>(leaf_ids) & 15) == 0);
  if (a.ids_vec) {
    // row r's ids begin at int b + r T of a line (b the output's offset in
    // its line), so its lines begin at trees -(b + r T) mod 32: a multiple
    // of 4 that depends on r mod 8
    const int64_t b = (int64_t)((reinterpret_cast<uintptr_t>(leaf_ids) >> 2) & 31);
    for (int rho = 0; rho < 8; ++rho) {
      const int phi = (int)((32 - (b + (int64_t)e.n_trees * rho) % 32) % 32);
      a.id_phase |= (uint64_t)1 << (8 * (phi / 4) + rho);
    }
  }
  const int64_t blocks_n = (n_rows + rows - 1) / rows;
  // Small batch with a workspace: divide the 32-tree groups among `parts`
  // workgroups per row tile. With `resident` workgroups of this shape running
  // at once, the walk takes about ceil(parts * tiles / resident) rounds of
  // `per` groups each plus a fixed cost per workgroup (feature tile, partial
  // sums) worth about kSplitOverheadGroups groups; take the fewest parts that
  // reach the least such time (no split when that is the unsplit launch).
  // Measured against forced part counts on the 500-tree depth-8, leaf-wise
  // depth-12 and 7-class models from 10K to 64K rows, this picks the fastest
  // count or one within 3% of it.
  int split = 1;
  const int cpf = kFastIdGroup / fast_tc_m(mode, tb, shapes[best].budget);  // chunks per 32 trees
  const int64_t groups = a.n_chunks / cpf;
  if (ws.ptr && n_rows <= kSplitMaxRows && groups >= 2) {
    int cus = 0, dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
      *err = "hipDeviceGetAttribute(MultiprocessorCount) failed";
      return HB_ERR_HIP;
    }
    const int64_t resident = (int64_t)cus * (int64_t)((size_t)lds_max / lds_of(shapes[best]));
    const int64_t row_bytes = n_rows * e.n_outputs * 8;
    constexpr int64_t kSplitOverheadGroups = 4;
    int64_t best_cost = (blocks_n + resident - 1) / resident * (groups + kSplitOverheadGroups), best_per = groups;
    for (int64_t p = 2; p <= groups; ++p) {
      const int64_t per = (groups + p - 1) / p, parts = (groups + per - 1) / per;
      if (parts * row_bytes > ws.bytes) break;
      const int64_t cost = (parts * blocks_n + resident - 1) / resident * (per + kSplitOverheadGroups);
      if (cost < best_cost) {
        best_cost = cost;
        best_per = per;
      }
    }
    if (best_per < groups) {
      split = (int)((groups + best_per - 1) / best_per);
      a.split = (int)best_per * cpf;
      a.partial = static_cast<double *>(ws.ptr);
    }
  }
  const unsigned fin_rows = (unsigned)((n_rows + 63) / 64);
  if (ws.plan) {
    plan_line(ws.plan,
              "fast_kernel<" + std::to_string(mode) + ", " + std::to_string(lg) + ", " + std::to_string(km) + ", " +
                  std::to_string(rows) + ", " + std::to_string(shapes[best].budget) + ">",
              blocks_n, split, rows, xbytes);
    if (split > 1) {
      if (km > 1)
        plan_line(ws.plan, "split_finish_kernel<16, 8>", fin_rows, 1, 64 * 8, (size_t)8 * e.n_outputs * 64 * 8);
      else
        plan_line(ws.plan, "split_finish_kernel<1, 16>", fin_rows, 1, 64 * 16, (size_t)16 * 64 * 8);
    }
    return HB_OK;
  }
  hipError_t rc = hipFuncSetAttribute(reinterpret_cast<const void *>(fn),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)xbytes);
  if (rc != hipSuccess) {
    *err = std::string("hipFuncSetAttribute: ") + hipGetErrorString(rc);
    return HB_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)blocks_n, (unsigned)split), dim3(rows), xbytes, stream, a);
  rc = hipGetLastError();
  if (rc == hipSuccess && split > 1) {
    // 16 waves per 64 rows for scalar outputs, 8 for several (their sums
    // take K times the LDS: at most 64 KiB)
    if (km > 1)
      hipLaunchKernelGGL((split_finish_kernel<HB_MAX_OUTPUTS, 8>), dim3(fin_rows), dim3(64 * 8),
                         (size_t)8 * e.n_outputs * 64 * sizeof(double), stream, a.partial, split, n_rows, a.out);
    else
      hipLaunchKernelGGL((split_finish_kernel<1, 16>), dim3(fin_rows), dim3(64 * 16),
                         (size_t)16 * 64 * sizeof(double), stream, a.partial, split, n_rows, a.out);
    rc = hipGetLastError();
  }
  if (rc != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(rc);
    return HB_ERR_HIP;
  }
  return HB_OK;
}

using RowsFn = void (*)(TravArgs);
template <bool PERFECT, int RW, bool CONTIG>
RowsFn pick_rows(int kmax, bool vec) {
  if (vec) return kmax == 2 ? rows_kernel<PERFECT, 2, true, RW, CONTIG> : nullptr;
  return kmax == 1   ? rows_kernel<PERFECT, 1, false, RW, CONTIG>
         : kmax == 2 ? rows_kernel<PERFECT, 2, false, RW, CONTIG>
                     : nullptr;
}

// Launches rows_kernel for batches whose rows are too wide for the
// row-parallel tile: 16 rows per workgroup (8 when 16 do not fit in LDS),
// one or two outputs, and enough rows for a workgroup per CU; returns
// kNotApplicable otherwise (the trees-across-lanes kernel then runs).
constexpr int64_t kRowsMinRows = 4096;
int launch_rows(bool perfect, const TravArgs &a, const Launch &L, hipStream_t stream, std::string *err) {
  if (a.n_rows < kRowsMinRows) return kNotApplicable;
  const bool vec = a.LD > 1;
  const int kmax = kmax_for(vec ? a.LD : a.K);
  if (kmax > 2 || (vec && a.LD != 2)) return kNotApplicable;
  const int lds_max = max_dynamic_lds(err);
  if (lds_max <= 0) return HB_ERR_HIP;
  int RW = 16;
  if (rows_lds(a.F, RW, kmax) > (size_t)lds_max) RW = 8;
  if (rows_lds(a.F, RW, kmax) > (size_t)lds_max) return kNotApplicable;
  // whole rows in 16-byte pieces go through the contiguous prefetch; its
  // 2,000-feature cap always leaves room for 16 rows per workgroup, so the
  // 8-row kernels stage through the column list only
  const bool contig = RW == 16 && a.cols == nullptr && a.Fs == a.F && (a.F & 3) == 0 && a.F <= 2000 &&
                      (reinterpret_cast<uintptr_t>(a.X) & 15) == 0;
  RowsFn fn = perfect ? (RW == 16 ? (contig ? pick_rows<true, 16, true>(kmax, vec) : pick_rows<true, 16, false>(kmax, vec))
                                  : pick_rows<true, 8, false>(kmax, vec))
                      : (RW == 16 ? (contig ? pick_rows<false, 16, true>(kmax, vec) : pick_rows<false, 16, false>(kmax, vec))
                                  : pick_rows<false, 8, false>(kmax, vec));
  if (!fn) return kNotApplicable;
  const size_t lds = rows_lds(a.F, RW, kmax);
  // persistent: as many workgroups as run at once (the row tiles are dealt
  // out round-robin), so each loads the next tile's rows during its walk
  int cus = 0, dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1) {
    *err = "hipDeviceGetAttribute(MultiprocessorCount) failed";
    return HB_ERR_HIP;
  }
  const int64_t tiles = (a.n_rows + RW - 1) / RW;
  const int64_t blocks = std::min(tiles, (int64_t)cus * (int64_t)std::max<size_t>(1, (size_t)lds_max / lds));
  if (L.plan) {
    plan_line(L.plan,
              std::string("rows_kernel<") + tf(perfect) + ", " + std::to_string(kmax) + ", " + tf(vec) + ", " +
                  std::to_string(RW) + ", " + tf(contig) + ">",
              blocks, 1, kRowsThreads, lds);
    return HB_OK;
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) {
    *err = std::string("hipFuncSetAttribute: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kRowsThreads), lds, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  return HB_OK;
}

// True when traverse_kernel would have to read the features from global
// memory (rows too wide for its LDS tile) or cannot stage a single tree:
// lanes_kernel is then the better choice at any batch size, since it stages a
// few whole rows per workgroup and reads node records through the caches.
bool rows_too_wide(const TravArgs &a, std::string *err) {
  const int lds_max = max_dynamic_lds(err);
  bool x_lds = false;
  return lds_max > 0 && (traverse_plan(a, lds_max, &x_lds) == 0 || !x_lds);
}

// Launches lanes_kernel; returns kNotApplicable if R rows of the input do not
// fit in LDS.
int launch_lanes(bool perfect, const TravArgs &a, const Launch &L, hipStream_t stream, std::string *err) {
  const int lds_max = max_dynamic_lds(err);
  if (lds_max <= 0) return HB_ERR_HIP;
  const bool vec = a.LD > 1;
  const int kmax = kmax_for(vec ? a.LD : a.K);
  // four rows per workgroup (four walks in flight per lane) when the batch is
  // large enough and the 4 x kmax double sums fit in registers
  int R = (a.n_rows > 4 * 256 && kmax <= 8) ? 4 : 1;
  auto need = [&](int r) { return ((size_t)r * a.F * 4 + 15) / 16 * 16 + (size_t)4 * r * kmax * 8; };
  if (need(R) > (size_t)lds_max) R = 1;
  if (need(R) > (size_t)lds_max) return kNotApplicable;
  LanesFn fn = perfect ? (R == 4 ? pick_lanes_r<true, 4>(kmax, vec) : pick_lanes_r<true, 1>(kmax, vec))
                       : (R == 4 ? pick_lanes_r<false, 4>(kmax, vec) : pick_lanes_r<false, 1>(kmax, vec));
  const size_t lds = need(R);
  const int64_t blocks = (a.n_rows + R - 1) / R;
  if (L.plan) {
    const int km = vec ? (kmax <= 2 ? 2 : kmax <= 8 ? 8 : 16) : kmax;
    plan_line(L.plan,
              std::string("lanes_kernel<") + tf(perfect) + ", " + std::to_string(km) + ", " + tf(vec) + ", " +
                  std::to_string(R) + ">",
              blocks, 1, kLaneThreads, lds);
    return HB_OK;
  }
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(fn), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds);
  if (e != hipSuccess) {
    *err = std::string("hipFuncSetAttribute: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)blocks), dim3(kLaneThreads), lds, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) {
    *err = std::string("kernel launch: ") + hipGetErrorString(e);
    return HB_ERR_HIP;
  }
  return HB_OK;
}

TravArgs common_args(const EnsembleDev &e, const float *X, int64_t n, float *scores, int32_t *ids) {
  TravArgs a{};
  a.X = X;
  a.n_rows = n;
  a.F = e.n_cols;
  a.Fs = e.n_features;
  a.cols = e.cols;
  a.scores = scores;
  a.leaf_ids = ids;
  a.T = e.n_trees;
  a.K = e.n_outputs;
  a.LD = e.leaf_dim;
  a.aggregation = e.aggregation;
  a.transform = e.transform;
  a.tree_class = e.tree_class;
  a.base_score = e.base_score;
  return a;
}

}  // namespace

int split_finish(const double *partial, int split, int64_t n_rows, const OutArgs &out, std::string *plan,
                 hipStream_t stream, std::string *err) {
  return launch_split_finish(partial, split, n_rows, out, plan, stream, err);
}

int launch_ptt(const EnsembleDev &e, const PttDev &t, const float *X, int64_t n_rows, float *scores,
               int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err) {
  if (!t.node || !t.node_il || !t.leaf_pk || !t.leaf_value || !t.leaf_id || t.depth < 0 || t.depth > HB_PTT_MAX_DEPTH) {
    *err = "PTT tables missing";
    return HB_ERR_INVALID_ARG;
  }
  if (n_rows <= 0) return HB_OK;
  TravArgs a = common_args(e, X, n_rows, scores, leaf_ids);
  a.node = t.node;
  a.node_il = t.node_il;
  a.leaf_pk = t.leaf_pk;
  a.last_il = t.last_il;
  a.leaf_value = t.leaf_value;
  a.leaf_id = t.leaf_id;
  a.depth = t.depth;
  a.slots = 1 << t.depth;
  a.leaf_slots = 1 << t.depth;
  if (a.slots < 2) a.slots = 2;  // depth 0 still stores two (unused) records per tree
  int rc = kNotApplicable;
  // rows too wide for the row-parallel tile: rows across lanes from a
  // workgroup per CU up, else (and for smaller batches) trees across lanes
  const bool wide = rows_too_wide(a, err);
  if (wide) rc = launch_rows(true, a, ws, stream, err);
  if (rc == kNotApplicable && n_rows <= (ws.ptr ? kLanesMaxRowsSplit : kLanesMaxRowsPtt)) rc = launch_lanes(true, a, ws, stream, err);
  if (rc == kNotApplicable)
    rc = launch_fast(t.fast_mode, t.depth, t.fast, t.fast_leafv, t.fast_chunks, nullptr, t.leaf_value, 1 << t.depth,
                     t.id_base, e, X, n_rows, scores, leaf_ids, ws, stream, err);
  if (rc == kPreferLanes || (rc == kNotApplicable && wide)) rc = launch_lanes(true, a, ws, stream, err);
  if (rc != kNotApplicable) return rc;
  return launch_traverse(true, a, ws, stream, err);
}

int launch_tt(const EnsembleDev &e, const TtDev &t, const float *X, int64_t n_rows, float *scores,
              int32_t *leaf_ids, const Launch &ws, hipStream_t stream, std::string *err) {
  if (!t.node || !t.node_il || !t.leaf_pk || !t.leaf_value || !t.leaf_id || !t.depth || t.n_pad < 1) {
    *err = "TT tables missing";
    return HB_ERR_INVALID_ARG;
  }
  if (t.n_pad % 2) {
    *err = "TT node slots must be even";
    return HB_ERR_INVALID_ARG;
  }
  if (n_rows <= 0) return HB_OK;
  TravArgs a = common_args(e, X, n_rows, scores, leaf_ids);
  a.node = t.node;
  a.node_il = t.node_il;
  a.leaf_pk = t.leaf_pk;
  a.leaf_value = t.leaf_value;
  a.leaf_id = t.leaf_id;
  a.tree_depth = t.depth;
  a.slots = t.n_pad;
  a.leaf_slots = t.n_pad;
  int rc = kNotApplicable;
  // rows too wide for the row-parallel tile: rows across lanes from a
  // workgroup per CU up, else (and for smaller batches) trees across lanes
  const bool wide = rows_too_wide(a, err);
  if (wide) rc = launch_rows(false, a, ws, stream, err);
  if (rc == kNotApplicable && n_rows <= (ws.ptr ? kLanesMaxRowsSplit : kLanesMaxRowsTt)) rc = launch_lanes(false, a, ws, stream, err);
  if (rc == kNotApplicable)
    rc = launch_fast(t.fast_mode, t.fast_lg, t.fast, t.fast_leaf, t.fast_chunks, t.depth, t.leaf_value, t.n_pad, 0, e, X,
                     n_rows, scores, leaf_ids, ws, stream, err);
  if (rc == kPreferLanes || (rc == kNotApplicable && wide)) rc = launch_lanes(false, a, ws, stream, err);
  if (rc != kNotApplicable) return rc;
  return launch_traverse(false, a, ws, stream, err);
}


}  // namespace hb
